"""Host-side pieces of bench.py: the byte counts behind roofline.achieved, the
source digest that decides whether stored HBM counters still apply, and the
refusal to run on more than one GPU."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_plain_step_bytes():
    # 12A + 20 per step for fp32 logits and gradients (both logit rows, four
    # [T,B] scalars in, d_logits and d_values out), plus 4 B of bootstrap per lane
    total, per_step = bench.algorithmic_bytes(1000, 16384, 18, 4)
    assert per_step == 12 * 18 + 20 == 236
    assert total == 1000 * 16384 * 236 + 4 * 16384
    assert bench.algorithmic_bytes(5, 4, 9, 2)[1] == 8 * 9 + 20       # bf16 logits
    assert bench.algorithmic_bytes(5, 4, 18, 4, log_probs=True)[1] == 18 * 4 + 4 + 16 + 18 * 4 + 4
    assert bench.algorithmic_bytes(5, 4, 18, 4, grad_bytes=2)[1] == 18 * 8 + 16 + 18 * 2 + 4
    assert bench.algorithmic_bytes(5, 4, 18, 4, uses_mu=False)[1] == 18 * 4 + 16 + 18 * 4 + 4


def test_head_call_bytes():
    total, per_step = bench.head_algorithmic_bytes(1000, 16384, 18, 256, 4)
    assert per_step == 2 * 256 + 4 * 18 + 12 + 4 * 256 == 1620
    assert bench.head_algorithmic_bytes(10, 3, 18, 256, 2)[1] == 1108
    per_call = 4 * 3 + (2 * 256 * 19 + 4 * 19) + (4 * 256 * 19 + 4 * 19 + 16)
    assert bench.head_algorithmic_bytes(10, 3, 18, 256, 2)[0] == 10 * 3 * 1108 + per_call
    # log mu(a_t|x_t) [T,B] in place of mu's logit row
    assert bench.head_algorithmic_bytes(10, 3, 18, 256, 4, log_probs=True)[1] == 1620 - 4 * 18 + 4


def test_digest_follows_the_kernel_sources(tmp_path, monkeypatch):
    d_plain = bench.kernel_source_digest()
    d_head = bench.kernel_source_digest(bench.HEAD_SOURCES)
    assert len(d_plain) == 16 and d_plain != d_head
    # counters stored under another digest are not used
    f = tmp_path / "c.json"
    f.write_text(json.dumps({"kernel_source_digest": "0" * 16, "hbm_bytes_per_launch": 1e9}))
    assert bench.stored_traffic(1.0, str(f)) == (None, None)
    f.write_text(json.dumps({"kernel_source_digest": d_plain, "hbm_bytes_per_launch": 2e9}))
    gbs, nbytes = bench.stored_traffic(0.5, str(f))
    assert nbytes == 2e9 and abs(gbs - 4000.0) < 1e-9
    assert bench.stored_traffic(1.0, str(tmp_path / "missing.json")) == (None, None)


def test_digest_ignores_comments_not_code(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_1802_01561_amd" / "csrc"
    csrc.mkdir(parents=True)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    src = csrc / "k.hip"

    def digest(text):
        src.write_text(text)
        return bench.kernel_source_digest(("k.hip",))

    base = digest('int f() { return 1; }  // one\nconst char* s = "a // b";\n')
    assert digest('/* doc */ int f()  {\n  return 1;  // the value one\n}\nconst char* s = "a // b";') == base
    assert digest('int f() { return 2; }  // one\nconst char* s = "a // b";\n') != base
    assert digest('int f() { return 1; }  // one\nconst char* s = "a // c";\n') != base


def test_committed_counters_are_well_formed():
    for name in ("loss_grad_stress_counters.json", "head_stress_counters.json"):
        c = json.load(open(os.path.join(ROOT, "profiles", name)))
        assert c["hbm_bytes_per_launch"] == pytest.approx(
            c["hbm_read_bytes_per_launch"] + c["hbm_write_bytes_per_launch"])
        assert 0.9 < c["traffic_over_algorithmic"] < 1.5
        assert len(c["kernel_source_digest"]) == 16 and c["commands"]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cpu_baseline_runs_on_one_thread():
    # the oracle's timing must be single-threaded (its BLAS calls included),
    # and the JSON records the host it ran on
    from threadpoolctl import threadpool_info
    with bench.one_thread():
        pools = threadpool_info()
        assert all(p["num_threads"] == 1 for p in pools)
    info = bench.host_info()
    assert info["oracle_threads"] == 1 and info["host_cpus"] >= info["host_cpus_available"] >= 1
    assert isinstance(info["cpu_model"], str)
