"""GPU parity of the correction variants (Sec. 5.2.3) and the baseline Q
estimate (App. E.3) against the oracle, through the _ex entry points."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_1802_01561_amd as vt
from gpu_util import assert_close, call_params, f32, log_case, np_out, oracle_args, require_gpu, to_device
from synth import Params, make_config, make_random

pytestmark = pytest.mark.gpu

CORRECTIONS = ["vtrace", "none", "epsilon", "one_step_is"]
Q_ESTIMATES = ["vtrace", "baseline"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def check_variant(tr, p, correction, q_estimate, epsilon=1e-6):
    dev = to_device(tr)
    out = vt.vtrace_loss_grad(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                              baseline_cost=p.baseline_cost, entropy_cost=p.entropy_cost,
                              with_vs=True, with_pg_advantages=True, with_lane_losses=True,
                              correction=correction, q_estimate=q_estimate, epsilon=epsilon)
    vs, pg = vt.vtrace_targets(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                               correction=correction, q_estimate=q_estimate, epsilon=epsilon)
    torch.cuda.synchronize()
    q = call_params(p)
    o = oracle.loss_and_grads(*oracle_args(tr), q.rho_bar, q.c_bar, q.lam, q.baseline_cost,
                              q.entropy_cost, correction=correction, q_estimate=q_estimate,
                              epsilon=f32(epsilon))
    tag = f"{correction}/{q_estimate}"
    assert_close(f"{tag} vs", np_out(out.vs), o.vs)
    assert_close(f"{tag} pg_advantages", np_out(out.pg_advantages), o.pg_advantages)
    assert_close(f"{tag} d_values", np_out(out.d_values), o.d_values)
    assert_close(f"{tag} d_logits", np_out(out.d_logits), o.d_logits)
    assert_close(f"{tag} lane_losses", np_out(out.lane_losses), o.lane_losses)
    assert_close(f"{tag} losses", np_out(out.losses), o.losses)
    assert_close(f"{tag} targets.vs", np_out(vs), o.vs)
    assert_close(f"{tag} targets.pg_advantages", np_out(pg), o.pg_advantages)


@pytest.mark.parametrize("kernel", ["tiled", "wide"])
@pytest.mark.parametrize("correction", CORRECTIONS)
@pytest.mark.parametrize("q_estimate", Q_ESTIMATES)
@pytest.mark.parametrize("cfg", [1, 2])
def test_variants_on_configs(cfg, correction, q_estimate, kernel, monkeypatch):
    monkeypatch.setenv("VTRACE_KERNEL", kernel)
    tr = make_config(cfg)
    for p in (Params(1.0, 1.0, 1.0), Params(2.0, 1.0, 0.9), Params(math.inf, math.inf, 1.0)):
        log_case(f"config {cfg} {correction}/{q_estimate} kernel={kernel} {p.label()}")
        check_variant(tr, p, correction, q_estimate)


@pytest.mark.parametrize("correction", CORRECTIONS)
@pytest.mark.parametrize("shape", [(37, 45, 18), (33, 70, 9), (12, 10, 7)])
@pytest.mark.parametrize("bf16", [False, True])
def test_variants_ragged_and_generic(correction, shape, bf16):
    T, B, A = shape
    tr = make_random(T, B, A, 90 + T + B + A, noise_std=1.0, bf16=bf16)
    log_case(f"variant {correction} T={T} B={B} A={A} bf16={bf16}")
    check_variant(tr, Params(1.0, 0.5, 0.95), correction, "baseline")
    check_variant(tr, Params(1.0, 1.0, 1.0), correction, "vtrace")


def test_epsilon_correction_with_unlikely_actions():
    """Taken actions with pi(a) near epsilon, where the correction changes the result."""
    tr = make_random(40, 64, 18, 5, noise_std=1.5)
    tr.target_logits[..., 3] -= np.float32(13.0)
    tr.actions[::3] = 3
    for eps in (1e-6, 1e-3):
        log_case(f"epsilon-correction eps={eps}")
        check_variant(tr, Params(1.0, 1.0, 1.0), "epsilon", "vtrace", epsilon=eps)
    # the correction is visible: the gradient differs from no-correction's
    dev = to_device(tr)
    a = vt.vtrace_loss_grad(**dev, correction="epsilon", epsilon=1e-3)
    b = vt.vtrace_loss_grad(**dev, correction="none")
    torch.cuda.synchronize()
    assert not np.allclose(np_out(a.d_logits), np_out(b.d_logits))


def test_variant_kernels_agree(monkeypatch):
    tr = make_random(64, 300, 9, 17, noise_std=1.0)
    dev = to_device(tr)
    for correction in CORRECTIONS:
        log_case(f"kernel agreement {correction}")
        kw = dict(rho_bar=2.0, c_bar=1.0, lam=0.9, correction=correction, q_estimate="baseline",
                  with_vs=True, with_pg_advantages=True)
        a = vt.vtrace_loss_grad(**dev, **kw)
        monkeypatch.setenv("VTRACE_KERNEL", "lane_serial")
        b = vt.vtrace_loss_grad(**dev, **kw)
        monkeypatch.delenv("VTRACE_KERNEL")
        torch.cuda.synchronize()
        for name in ("vs", "pg_advantages", "d_values", "d_logits"):
            assert_close(f"{correction} {name}", np_out(getattr(a, name)), np_out(getattr(b, name)),
                         rtol=2e-5, atol=2e-6)


# --------------------------------------------------------------------------------------
# Input/output variants: behaviour log-probabilities, reward preprocessing, bf16 grads
# --------------------------------------------------------------------------------------

# bfloat16 gradients: the float32 result (within 1e-5 + 1e-4|o| of the oracle) is
# rounded to nearest-even bfloat16 (8 significant bits), adding at most 2^-8 of
# its magnitude, so
# |g - o| <= 1e-5 + 1e-4|o| + 2^-8 (1 + 1e-4)|o| + 2^-8 * 1e-5 < 1.1e-5 + 4.1e-3|o|.
BF16_GRAD_ATOL, BF16_GRAD_RTOL = 1.1e-5, 4.1e-3


def behaviour_log_probs(tr):
    """log mu(a_t|x_t) as float32, from the behaviour logits (host, float64)."""
    import scipy.special
    lp = scipy.special.log_softmax(tr.behaviour_logits.astype(np.float64), axis=-1)
    return np.take_along_axis(lp, tr.actions[..., None].astype(np.int64), -1)[..., 0].astype(np.float32)


def check_io_variant(tr, p, *, log_probs=False, reward_transform=None, grad_bf16=False,
                     correction="vtrace", lanes=None, q_estimate="vtrace"):
    dev = to_device(tr)
    otr_args = list(oracle_args(tr))
    behaviour = "logits"
    if log_probs:
        lmu = behaviour_log_probs(tr)
        dev["behaviour_logits"] = torch.from_numpy(lmu).cuda()
        otr_args[1] = lmu
        behaviour = "log_probs"
    gd = torch.bfloat16 if grad_bf16 else torch.float32
    out = vt.vtrace_loss_grad(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                              baseline_cost=p.baseline_cost, entropy_cost=p.entropy_cost,
                              with_vs=True, with_pg_advantages=True, with_lane_losses=True,
                              correction=correction, q_estimate=q_estimate, behaviour=behaviour,
                              reward_transform=reward_transform, grad_dtype=gd)
    vs, pg = vt.vtrace_targets(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                               correction=correction, q_estimate=q_estimate, behaviour=behaviour,
                               reward_transform=reward_transform)
    torch.cuda.synchronize()
    if lanes is not None:
        idx = np.asarray(lanes)
        otr_args = [x[:, idx] if i != 6 else x[idx] for i, x in enumerate(otr_args)]
    q = call_params(p)
    o = oracle.loss_and_grads(*otr_args, q.rho_bar, q.c_bar, q.lam, q.baseline_cost,
                              q.entropy_cost, correction=correction, q_estimate=q_estimate,
                              behaviour=behaviour, reward_transform=reward_transform, epsilon=f32(1e-6))
    pick = (lambda x: x) if lanes is None else (lambda x: x[:, lanes])
    tag = f"lp={log_probs} r={reward_transform} bf16={grad_bf16} {correction}/{q_estimate}"
    assert_close(f"{tag} vs", pick(np_out(out.vs)), o.vs)
    assert_close(f"{tag} pg_advantages", pick(np_out(out.pg_advantages)), o.pg_advantages)
    assert_close(f"{tag} d_values", pick(np_out(out.d_values)), o.d_values)
    dl_kw = dict(rtol=BF16_GRAD_RTOL, atol=BF16_GRAD_ATOL) if grad_bf16 else {}
    assert out.d_logits.dtype == gd
    assert_close(f"{tag} d_logits", pick(np_out(out.d_logits)), o.d_logits, **dl_kw)
    lane = np_out(out.lane_losses)
    assert_close(f"{tag} lane_losses", lane if lanes is None else lane[lanes], o.lane_losses)
    if lanes is None:
        assert_close(f"{tag} losses", np_out(out.losses), o.losses)
        assert_close(f"{tag} targets.vs", np_out(vs), o.vs)
        assert_close(f"{tag} targets.pg_advantages", np_out(pg), o.pg_advantages)


@pytest.mark.parametrize("kernel", ["tiled", "wide"])
@pytest.mark.parametrize("log_probs", [False, True])
@pytest.mark.parametrize("reward_transform", [None, "clip", "asymmetric"])
@pytest.mark.parametrize("grad_bf16", [False, True])
def test_io_variants_configs(log_probs, reward_transform, grad_bf16, kernel, monkeypatch):
    monkeypatch.setenv("VTRACE_KERNEL", kernel)
    for cfg in (1, 2):
        tr = make_config(cfg)
        tr.rewards = (tr.rewards * 3.0 - 0.5).astype(np.float32)  # exercise the clipping
        for p in (Params(1.0, 1.0, 1.0), Params(math.inf, math.inf, 1.0)):
            log_case(f"config {cfg} io lp={log_probs} r={reward_transform} bf16={grad_bf16} {p.label()}")
            check_io_variant(tr, p, log_probs=log_probs, reward_transform=reward_transform,
                             grad_bf16=grad_bf16)


@pytest.mark.parametrize("shape", [(37, 45, 18), (33, 70, 9), (12, 10, 7), (20, 64, 18)])
@pytest.mark.parametrize("bf16_logits", [False, True])
def test_io_variants_shapes(shape, bf16_logits):
    T, B, A = shape
    tr = make_random(T, B, A, 300 + T + A, noise_std=1.0, bf16=bf16_logits)
    tr.rewards = (tr.rewards * 2.5).astype(np.float32)
    for correction in ("vtrace", "one_step_is", "epsilon"):
        log_case(f"io variants T={T} B={B} A={A} bf16-logits={bf16_logits} {correction}")
        check_io_variant(tr, Params(1.0, 0.5, 0.95), log_probs=True, reward_transform="asymmetric",
                         grad_bf16=True, correction=correction)
        check_io_variant(tr, Params(2.0, 1.0, 1.0), log_probs=False, reward_transform="clip",
                         grad_bf16=True, correction=correction)


def test_io_variants_stress_subset():
    from synth.trajectories import STRESS_SUBSET
    tr = make_config(4)
    for p in (Params(1.0, 1.0, 1.0), Params(math.inf, math.inf, 1.0)):
        log_case(f"stress, behaviour log-probabilities + bf16 grads, {p.label()}")
        check_io_variant(tr, p, log_probs=True, grad_bf16=True, lanes=STRESS_SUBSET)


@pytest.mark.parametrize("A,bf16,transform,log_probs,grad_bf16,lanes_per_cu",
                         [(18, False, "clip", False, False, 64), (18, True, "asymmetric", False, False, 64),
                          (9, False, "asymmetric", False, False, 64), (9, True, "clip", False, False, 128),
                          (18, False, None, True, False, 64), (18, True, "clip", True, False, 64),
                          (9, False, "asymmetric", True, False, 128), (18, False, None, False, True, 64),
                          (18, False, "asymmetric", False, True, 64), (9, True, "clip", True, True, 128)])
def test_plain_kernels_on_long_tiles(A, bf16, transform, log_probs, grad_bf16, lanes_per_cu, monkeypatch):
    """Plain V-trace calls with a reward transform (Atari's clipping, DMLab's
    asymmetric transform), bfloat16 gradients or behaviour log-probabilities
    (what the paper's actors send) on batches that take the long-run loss
    tiles run plain loss kernels with those as their only switches: sampled
    lanes against the oracle, and every output against the general kernel of
    the 16-step tiles (VTRACE_KERNEL=tiled_short) within the tolerance."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    T, B = 37, lanes_per_cu * cus
    tr = make_random(T, B, A, 6100 + A + lanes_per_cu, noise_std=1.0, end_prob=0.03, bf16=bf16)
    tr.rewards = (tr.rewards * 2.5).astype(np.float32)  # exercise the transform
    p = Params(1.0, 1.0, 1.0)
    lanes = [0, 1, 31, 32, 63, 64, B // 2, B - 33, B - 1]
    log_case(f"plain kernel on long tiles, rewards {transform} log-probs {log_probs} bf16 grads {grad_bf16} "
             f"T={T} B={B} A={A} bf16={bf16}")
    monkeypatch.delenv("VTRACE_KERNEL", raising=False)
    check_io_variant(tr, p, reward_transform=transform, log_probs=log_probs, grad_bf16=grad_bf16, lanes=lanes)
    dev = to_device(tr)
    kw = dict(rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam, with_vs=True, with_pg_advantages=True,
              with_lane_losses=True, reward_transform=transform,
              grad_dtype=torch.bfloat16 if grad_bf16 else torch.float32)
    if log_probs:
        dev["behaviour_logits"] = torch.from_numpy(behaviour_log_probs(tr)).cuda()
        kw["behaviour"] = "log_probs"
    a = vt.vtrace_loss_grad(**dev, **kw)
    monkeypatch.setenv("VTRACE_KERNEL", "tiled_short")
    b = vt.vtrace_loss_grad(**dev, **kw)
    monkeypatch.delenv("VTRACE_KERNEL")
    torch.cuda.synchronize()
    for name in ("vs", "pg_advantages", "d_values", "d_logits"):
        assert_close(f"long-run plain vs 16-step general {name}", np_out(getattr(a, name)),
                     np_out(getattr(b, name)), rtol=2e-5, atol=2e-6)
    for name in ("lane_losses", "losses"):
        assert_close(f"long-run plain vs 16-step general {name}", np_out(getattr(a, name)),
                     np_out(getattr(b, name)))


def _sweep_cases():
    """Seeded random draws over every axis the entry points take."""
    rng = np.random.default_rng(20261202)
    cases = []
    for _ in range(24):
        cases.append(dict(
            T=int(rng.choice([1, 5, 16, 17, 33, 64, 100, 130])),
            B=int(rng.choice([1, 3, 16, 33, 64, 200, 512, 1000])),
            A=int(rng.choice([9, 18, 9, 18, 5])),
            bf16=bool(rng.random() < 0.3),
            p=Params(float(rng.choice([1.0, 2.0, math.inf, 0.5])), float(rng.choice([1.0, 0.5, math.inf])),
                     float(rng.choice([1.0, 0.95, 0.5]))),
            correction=str(rng.choice(CORRECTIONS)), q_estimate=str(rng.choice(Q_ESTIMATES)),
            log_probs=bool(rng.random() < 0.3), reward_transform=rng.choice([None, "clip", "asymmetric"]),
            grad_bf16=bool(rng.random() < 0.3), lanes=None))
    # whole multiples of the resident workgroups (multi-tile walk), on a lane subset
    for A, bf16, lp, gb in [(18, False, False, False), (18, False, True, True), (9, False, False, True),
                            (9, True, True, False)]:
        cases.append(dict(T=20, B=24576, A=A, bf16=bf16, p=Params(1.0, 1.0, 1.0), correction="vtrace",
                          q_estimate="vtrace", log_probs=lp, reward_transform="clip", grad_bf16=gb,
                          lanes=[0, 1, 17, 4095, 12288, 24575]))
    cases.append(dict(T=20, B=24576, A=18, bf16=False, p=Params(1.0, 0.5, 0.95), correction="one_step_is",
                      q_estimate="baseline", log_probs=False, reward_transform=None, grad_bf16=False,
                      lanes=[3, 777, 24560, 24575]))
    # 64 lanes per CU on a 256-CU part: the long-run tile shapes (loss calls:
    # 32 x 8 for A = 9 and 18), with ragged T, on a lane subset
    for A, bf16, lp, gb, corr, qe, rt in [(18, False, True, True, "one_step_is", "vtrace", "asymmetric"),
                                          (9, False, False, True, "epsilon", "baseline", "clip"),
                                          (18, True, True, False, "none", "vtrace", None),
                                          (9, True, False, True, "vtrace", "baseline", "asymmetric")]:
        cases.append(dict(T=37, B=16384, A=A, bf16=bf16, p=Params(1.0, 0.5, 0.95), correction=corr,
                          q_estimate=qe, log_probs=lp, reward_transform=rt, grad_bf16=gb,
                          lanes=[0, 1, 31, 32, 63, 64, 8191, 16320, 16383]))
    # around the crossover between the time-parallel and the tiled kernel
    # (T from 17 to 256, B from 8 to 1024) and with lambda = 0.95, whose
    # float32 value the call receives
    for _ in range(12):
        cases.append(dict(
            T=int(rng.choice([17, 20, 48, 100, 129, 200, 256])),
            B=int(rng.choice([8, 15, 100, 512, 700, 1024])),
            A=int(rng.choice([9, 18])),
            bf16=bool(rng.random() < 0.3),
            p=Params(float(rng.choice([1.0, math.inf])), float(rng.choice([1.0, 0.5, math.inf])), 0.95),
            correction=str(rng.choice(["vtrace", "vtrace", "none", "one_step_is"])),
            q_estimate=str(rng.choice(Q_ESTIMATES)), log_probs=bool(rng.random() < 0.4),
            reward_transform=rng.choice([None, "clip", "asymmetric"]), grad_bf16=bool(rng.random() < 0.3),
            lanes=None))
    # 128 lanes per CU: loss calls with A = 9 take 64 x 4 tiles
    for bf16, lp, gb, corr, qe in [(False, True, False, "epsilon", "vtrace"), (True, False, True, "one_step_is", "baseline")]:
        cases.append(dict(T=21, B=32768, A=9, bf16=bf16, p=Params(2.0, 1.0, 0.9), correction=corr,
                          q_estimate=qe, log_probs=lp, reward_transform="clip", grad_bf16=gb,
                          lanes=[0, 1, 63, 64, 127, 16383, 16384, 32704, 32767]))
    return cases


@pytest.mark.parametrize("i", range(len(_sweep_cases())))
def test_random_sweep(i):
    """Seeded draws mixing shapes (ragged T and B, A = 5, 9, 18), logit types,
    corrections, Q estimates, behaviour log-probabilities, reward transforms,
    bfloat16 gradients and clipping levels, each against the oracle; then
    batches of 24576 lanes, whole multiples of the workgroups the chip holds at
    once, which take the tiled kernel's multi-tile walk (bf16 logits with
    A = 9: the 32 x 8 long-run tiles, which fill the chip once there), of
    16384 lanes, which take the long-run tile shapes, and of 32768 lanes with
    A = 9, whose loss calls take 64 x 4 tiles; and draws around the crossover
    between the time-parallel and the tiled kernel with lambda = 0.95."""
    c = _sweep_cases()[i]
    tr = make_random(c["T"], c["B"], c["A"], 900 + i, noise_std=1.0, end_prob=0.03, bf16=c["bf16"])
    tr.rewards = (tr.rewards * 2.5).astype(np.float32)  # exercise the clipping
    log_case(f"sweep {i}: " + ", ".join(f"{k}={v}" for k, v in c.items() if k != "lanes"))
    check_io_variant(tr, c["p"], log_probs=c["log_probs"], reward_transform=c["reward_transform"],
                     grad_bf16=c["grad_bf16"], correction=c["correction"], q_estimate=c["q_estimate"],
                     lanes=c["lanes"])
