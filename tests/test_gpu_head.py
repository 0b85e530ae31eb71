"""GPU parity of the fused output layer + V-trace entry point
(vtrace_head_loss_grad) against the fp64 oracle (oracle/head.py).

Tolerances.  Per-step outputs (the layer's outputs, v_s, advantages) meet
|g - o| <= 1e-5 + 1e-4 |o|.  The other outputs are sums: d_weight and d_bias
over every step of the batch (of hidden[r, h] G[r, c] and G[r, c]), the lane
losses over a lane's steps, the loss totals over all steps, and each d_hidden
element over the A + 1 output columns.  An error of up to 1e-4 of each term
(the per-element bound) adds up, for independent errors, to about 1e-4 times
the root-sum-square of the terms, so sums use
|g - o| <= 1e-5 + 1e-4 |o| + 1e-4 RSS, as the plain loss's sums do; here the
layer's float32 logits add their own rounding to every term.  bfloat16
d_hidden adds its rounding (2^-8 relative).
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_1802_01561_amd as vt
from gpu_util import (ATOL, RTOL, assert_close, call_params, f32, assert_sum_close, head_kappa_hidden, head_kappa_loss,
                      head_kappa_param, log_case, np_out, require_gpu)
from synth import HEAD_WORKLOADS, Params, make_head, make_head_config, subset_head_lanes

pytestmark = pytest.mark.gpu

BF16_ATOL, BF16_RTOL = 1.1e-5, 4.1e-3  # float32 bound widened by one bfloat16 rounding (2^-8)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def bf16_tensor(bits, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def head_to_device(hb, behaviour=None, behaviour_bf16=False):
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to("cuda")
    if behaviour is not None:
        beh = d(behaviour)
    elif behaviour_bf16:
        from synth import f32_to_bf16_bits
        beh = bf16_tensor(f32_to_bf16_bits(hb.behaviour_logits))
    else:
        beh = d(hb.behaviour_logits)
    return dict(hidden=bf16_tensor(hb.hidden_bits), head_weight=bf16_tensor(hb.weight_bits),
                head_bias=d(hb.bias), behaviour_logits=beh, actions=d(hb.actions),
                rewards=d(hb.rewards), discounts=d(hb.discounts),
                bootstrap_value=d(hb.bootstrap_value))


def run_head(dev, p, **kw):
    out = vt.vtrace_head_loss_grad(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                                   baseline_cost=p.baseline_cost, entropy_cost=p.entropy_cost,
                                   with_vs=True, with_pg_advantages=True, with_lane_losses=True,
                                   with_outputs=True, **kw)
    torch.cuda.synchronize()
    return out


def check_head(hb, p, out, *, behaviour_values=None, grad_bf16=False, lanes=None, whole=True,
               **variant):
    """Every output of a call against the oracle on the same inputs (or on the
    given lanes alone, where the per-lane outputs are compared)."""
    sub = hb if lanes is None else subset_head_lanes(hb, lanes)
    beh = sub.behaviour_logits if behaviour_values is None else behaviour_values
    if lanes is not None and behaviour_values is not None:
        beh = behaviour_values[:, lanes]
    q = call_params(p)
    if "epsilon" in variant or variant.get("correction") == "epsilon":
        variant = dict(variant, epsilon=f32(variant.get("epsilon", 1e-6)))
    o = oracle.head_loss_and_grads(sub.hidden, sub.weight, sub.bias, beh, sub.actions,
                                   sub.rewards, sub.discounts, sub.bootstrap_value, q.rho_bar,
                                   q.c_bar, q.lam, q.baseline_cost, q.entropy_cost, **variant)
    pick = (lambda x: x) if lanes is None else (lambda x: x[:, lanes])
    assert_close("outputs", pick(np_out(out.outputs)), o.outputs)
    assert_close("vs", pick(np_out(out.vs)), o.vs)
    assert_close("pg_advantages", pick(np_out(out.pg_advantages)), o.pg_advantages)
    kl, kh = head_kappa_loss(sub.H), head_kappa_hidden(sub.H)
    lane = np_out(out.lane_losses)
    rss_lane = np.sqrt((o.step_losses ** 2).sum(axis=0))
    assert_sum_close("lane_losses", lane if lanes is None else lane[lanes], o.lane_losses, rss_lane, kl)
    W = sub.weight.astype(np.float64)
    rss_h = np.sqrt((o.d_outputs ** 2) @ (W.T ** 2))
    dh = pick(np_out(out.d_hidden))
    if grad_bf16:
        assert_sum_close("d_hidden (bf16)", dh, o.d_hidden, rss_h, kh, rtol=BF16_RTOL, atol=BF16_ATOL)
    else:
        assert_sum_close("d_hidden", dh, o.d_hidden, rss_h, kh)
    if lanes is None and whole:
        rss_w, rss_b = oracle.sum_term_scale(sub.hidden, o.d_outputs)
        kp = head_kappa_param(sub.H, sub.T, sub.B)
        assert_sum_close("d_weight", np_out(out.d_weight), o.d_weight, rss_w, kp)
        assert_sum_close("d_bias", np_out(out.d_bias), o.d_bias, rss_b, kp)
        s2 = (o.step_losses ** 2).sum(axis=(0, 1))
        rss_tot = np.sqrt(np.concatenate([[s2.sum()], s2]))
        assert_sum_close("losses", np_out(out.losses), o.losses, rss_tot, kl)
    return o


PARAMS = [Params(1.0, 1.0, 1.0), Params(math.inf, math.inf, 1.0), Params(2.0, 1.0, 0.9),
          Params(1.0, 0.5, 0.95)]


@pytest.mark.parametrize("name", ["tiny", "dmlab", "atari"])
def test_head_configs(name):
    hb = make_head_config(name)
    dev = head_to_device(hb)
    for p in PARAMS:
        log_case(f"head {name} T={hb.T} B={hb.B} A={hb.A} H={hb.H} {p.label()}")
        check_head(hb, p, run_head(dev, p))


@pytest.mark.parametrize("shape", [(37, 7, 18, 256), (16, 9, 9, 128), (21, 5, 15, 64), (17, 6, 16, 64),
                                   (19, 4, 31, 128), (12, 3, 1, 64), (1, 1, 5, 64)])
def test_head_shapes(shape):
    """Ragged T and B, each hidden size, A + 1 = 16 and 17 (one or two column
    tiles), the largest A, a single action, a single step."""
    T, B, A, H = shape
    hb = make_head(T, B, A, H, 500 + T + B + A + H, end_prob=0.05)
    dev = head_to_device(hb)
    for p in (Params(1.0, 1.0, 1.0), Params(math.inf, math.inf, 1.0)):
        log_case(f"head shape T={T} B={B} A={A} H={H} {p.label()}")
        check_head(hb, p, run_head(dev, p))


def test_head_many_lanes_per_workgroup():
    """More lane groups than workgroups: each workgroup walks several groups."""
    hb = make_head(3, 2060, 18, 64, 77)
    assert (hb.B + 3) // 4 > 512
    dev = head_to_device(hb)
    p = Params(1.0, 1.0, 1.0)
    log_case(f"head T={hb.T} B={hb.B} (lane groups beyond the workgroup count)")
    check_head(hb, p, run_head(dev, p))


@pytest.mark.parametrize("correction", ["none", "epsilon", "one_step_is"])
@pytest.mark.parametrize("q_estimate", ["vtrace", "baseline"])
def test_head_correction_variants(correction, q_estimate):
    hb = make_head_config("atari")
    dev = head_to_device(hb)
    for p in (Params(1.0, 1.0, 1.0), Params(2.0, 1.0, 0.9)):
        log_case(f"head atari {correction}/{q_estimate} {p.label()}")
        out = run_head(dev, p, correction=correction, q_estimate=q_estimate)
        check_head(hb, p, out, correction=correction, q_estimate=q_estimate)


@pytest.mark.parametrize("H", [64, 256])
def test_head_epsilon_correction_with_a_certain_action(H):
    """The epsilon-correction with a single action, where pi(a) = 1: every
    policy-gradient term is -adv log(1 + eps), about -adv eps, and their sums
    must still meet the bound; pi(a) + eps rounded to float32 (1.00000095 for
    eps = 1e-6) would be 5% off in every term."""
    A = 1
    hb = make_head(40, 33, A, H, 4100 + H, end_prob=0.05)
    hb.rewards = (hb.rewards * 2.5).astype(np.float32)
    dev = head_to_device(hb)
    for p in (Params(1.0, math.inf, 0.95), Params(1.0, 1.0, 1.0)):
        log_case(f"head epsilon-correction A={A} H={H} {p.label()}")
        out = run_head(dev, p, correction="epsilon", reward_transform="asymmetric")
        check_head(hb, p, out, correction="epsilon", reward_transform="asymmetric")


@pytest.mark.parametrize("log_probs", [False, True])
@pytest.mark.parametrize("reward_transform", [None, "asymmetric"])
@pytest.mark.parametrize("grad_bf16", [False, True])
def test_head_io_variants(log_probs, reward_transform, grad_bf16):
    hb = make_head(40, 10, 18, 128, 31)
    hb.rewards = (hb.rewards * 2.5).astype(np.float32)
    beh_vals = None
    if log_probs:
        import scipy.special
        lp = scipy.special.log_softmax(hb.behaviour_logits.astype(np.float64), axis=-1)
        beh_vals = np.take_along_axis(lp, hb.actions[..., None].astype(np.int64), -1)[..., 0]
        beh_vals = beh_vals.astype(np.float32)
    dev = head_to_device(hb, behaviour=beh_vals)
    gd = torch.bfloat16 if grad_bf16 else torch.float32
    kw = dict(behaviour="log_probs" if log_probs else "logits", reward_transform=reward_transform)
    for p in (Params(1.0, 1.0, 1.0), Params(math.inf, math.inf, 1.0)):
        log_case(f"head io lp={log_probs} r={reward_transform} bf16-grad={grad_bf16} {p.label()}")
        out = run_head(dev, p, grad_dtype=gd, **kw)
        assert out.d_hidden.dtype == gd
        check_head(hb, p, out, behaviour_values=beh_vals, grad_bf16=grad_bf16, **kw)


def _head_sweep_cases():
    """Seeded draws over the output-layer call's axes: shapes (one or two
    column tiles, each hidden size, ragged T and B, a single action),
    clipping levels, corrections and Q estimates, behaviour log-probabilities,
    reward transforms and bf16 d_hidden."""
    rng = np.random.default_rng(20261203)
    cases = []
    for _ in range(16):
        cases.append(dict(
            T=int(rng.choice([1, 5, 16, 17, 31, 40])), B=int(rng.choice([1, 3, 4, 7, 16, 33])),
            A=int(rng.choice([1, 5, 9, 15, 16, 18, 31])), H=int(rng.choice([64, 128, 256])),
            p=Params(float(rng.choice([1.0, math.inf, 2.0])), float(rng.choice([1.0, 0.5, math.inf])),
                     float(rng.choice([1.0, 0.95]))),
            log_probs=bool(rng.random() < 0.3), reward_transform=rng.choice([None, "clip", "asymmetric"]),
            grad_bf16=bool(rng.random() < 0.3),
            correction=str(rng.choice(["vtrace", "vtrace", "none", "epsilon", "one_step_is"])),
            q_estimate=str(rng.choice(["vtrace", "baseline"]))))
    return cases


@pytest.mark.parametrize("i", range(len(_head_sweep_cases())))
def test_head_random_sweep(i):
    """Each seeded draw against the oracle (every output, d_W, d_b and the
    loss totals)."""
    c = _head_sweep_cases()[i]
    hb = make_head(c["T"], c["B"], c["A"], c["H"], 20000 + i, end_prob=0.05)
    hb.rewards = (hb.rewards * 2.5).astype(np.float32)
    beh_vals = None
    if c["log_probs"]:
        import scipy.special
        lp = scipy.special.log_softmax(hb.behaviour_logits.astype(np.float64), axis=-1)
        beh_vals = np.take_along_axis(lp, hb.actions[..., None].astype(np.int64), -1)[..., 0]
        beh_vals = beh_vals.astype(np.float32)
    dev = head_to_device(hb, behaviour=beh_vals)
    kw = dict(behaviour="log_probs" if c["log_probs"] else "logits", reward_transform=c["reward_transform"],
              correction=c["correction"], q_estimate=c["q_estimate"])
    log_case(f"head sweep {i}: " + ", ".join(f"{k}={v}" for k, v in c.items()))
    out = run_head(dev, c["p"], grad_dtype=torch.bfloat16 if c["grad_bf16"] else torch.float32, **kw)
    check_head(hb, c["p"], out, behaviour_values=beh_vals, grad_bf16=c["grad_bf16"], **kw)


def test_head_bf16_behaviour_logits():
    from synth import bf16_bits_to_f32, f32_to_bf16_bits
    hb = make_head(33, 8, 9, 256, 32)
    hb.behaviour_logits = bf16_bits_to_f32(f32_to_bf16_bits(hb.behaviour_logits))
    dev = head_to_device(hb, behaviour_bf16=True)
    assert dev["behaviour_logits"].dtype == torch.bfloat16
    p = Params(1.0, 1.0, 1.0)
    log_case("head bf16 behaviour logits")
    check_head(hb, p, run_head(dev, p))


def test_head_deterministic_and_invariants():
    hb = make_head(50, 12, 18, 256, 33)
    dev = head_to_device(hb)
    p = Params(1.0, 1.0, 1.0)
    log_case("head determinism")
    a = run_head(dev, p)
    b = run_head(dev, p)
    for name in ("losses", "d_hidden", "d_weight", "d_bias", "vs", "lane_losses"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    # policy columns of d_bias and of each d_weight row sum to zero
    db = np_out(a.d_bias)
    dw = np_out(a.d_weight)
    A = hb.A
    assert abs(db[:A].sum()) <= 1e-4 * np.abs(db[:A]).sum() + 1e-5
    assert np.all(np.abs(dw[:, :A].sum(axis=1)) <= 1e-4 * np.abs(dw[:, :A]).sum(axis=1) + 1e-5)
    # loss totals are the lane sums
    lane = np_out(a.lane_losses).astype(np.float64)
    tot = np_out(a.losses)
    assert np.allclose(tot[1:], lane.sum(axis=0), rtol=1e-5, atol=1e-5)


def test_head_out_of_range_action_sets_flag():
    hb = make_head(20, 8, 9, 64, 34)
    hb.actions[7, 3] = 9
    dev = head_to_device(hb)
    ws = vt.Workspace(hb.T, hb.B, hb.A, H=hb.H)
    log_case("head out-of-range action")
    out = vt.vtrace_head_loss_grad(**dev, workspace=ws, with_vs=True)
    assert vt.vtrace_error_flag(ws) == 1
    assert torch.isnan(out.d_bias).any()
    vs = np_out(out.vs)
    assert np.isfinite(vs[8:, 3]).all()  # later steps of the lane do not depend on step 7
    assert np.isfinite(vs[:, [0, 1, 2, 4, 5, 6, 7]]).all()


def test_head_matches_plain_kernel_on_its_outputs():
    """The fused call and the plain loss kernel fed the layer's outputs agree
    on the V-trace quantities."""
    hb = make_head(64, 16, 18, 128, 35)
    dev = head_to_device(hb)
    p = Params(1.0, 1.0, 1.0)
    log_case("head vs plain kernel on the layer outputs")
    out = run_head(dev, p)
    o = out.outputs
    plain = vt.vtrace_loss_grad(o[..., :hb.A].contiguous(), dev["behaviour_logits"], dev["actions"],
                                dev["rewards"], dev["discounts"], o[..., hb.A].contiguous(),
                                dev["bootstrap_value"], with_vs=True, with_pg_advantages=True)
    torch.cuda.synchronize()
    assert_close("vs", np_out(out.vs), np_out(plain.vs), rtol=2e-5, atol=2e-6)
    assert_close("pg", np_out(out.pg_advantages), np_out(plain.pg_advantages), rtol=2e-5, atol=2e-6)


def test_head_stress_every_lane():
    """The full stress shape with (1, 1, 1): every per-step and per-lane output
    against the oracle, 512 lanes at a time, and d_W, d_b and the loss totals
    against the oracle's sums over all chunks (the sum bound, kappa times the
    RSS of all their terms)."""
    from synth import SEED_BASE, head_batch_from_device, make_head_device
    c = HEAD_WORKLOADS["stress"]
    log_case("head stress, every lane: generating on the device")
    d = make_head_device(c["T"], c["B"], c["A"], c["H"], SEED_BASE + 1004, "cuda")
    dev = dict(hidden=d["hidden"], head_weight=d["weight"], head_bias=d["bias"],
               behaviour_logits=d["behaviour_logits"], actions=d["actions"], rewards=d["rewards"],
               discounts=d["discounts"], bootstrap_value=d["bootstrap_value"])
    p = Params(1.0, 1.0, 1.0)
    out = vt.vtrace_head_loss_grad(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                                   with_vs=True, with_pg_advantages=True, with_lane_losses=True,
                                   with_outputs=True)
    torch.cuda.synchronize()
    C = c["A"] + 1
    dw = np.zeros((c["H"], C)); db = np.zeros(C); tot = np.zeros(3)
    rw2 = np.zeros((c["H"], C)); rb2 = np.zeros(C); s2 = np.zeros(3)
    for l0 in range(0, c["B"], 512):
        lanes = list(range(l0, min(c["B"], l0 + 512)))
        log_case(f"head stress, lanes {l0}..{lanes[-1]}")
        hb = head_batch_from_device(d, lanes)
        sel = torch.as_tensor(lanes, device="cuda")
        view = vt.HeadLossGrad(out.losses, out.d_hidden[:, sel].cpu(), out.d_weight, out.d_bias,
                               out.vs[:, sel].cpu(), out.pg_advantages[:, sel].cpu(),
                               out.lane_losses[sel], out.outputs[:, sel].cpu())
        o = check_head(hb, p, view, whole=False)
        rw, rb = oracle.sum_term_scale(hb.hidden, o.d_outputs)
        dw += o.d_weight; db += o.d_bias; tot += o.losses[1:]
        rw2 += rw ** 2; rb2 += rb ** 2; s2 += (o.step_losses ** 2).sum(axis=(0, 1))
    kp = head_kappa_param(c["H"], c["T"], c["B"])
    assert_sum_close("d_weight", np_out(out.d_weight), dw, np.sqrt(rw2), kp)
    assert_sum_close("d_bias", np_out(out.d_bias), db, np.sqrt(rb2), kp)
    assert_sum_close("losses", np_out(out.losses), np.concatenate([[tot.sum()], tot]),
                     np.sqrt(np.concatenate([[s2.sum()], s2])), head_kappa_loss(c["H"]))
    del out, d, dev
    torch.cuda.empty_cache()


def test_head_stress_sampled_lanes():
    """The full stress shape (T=1000, B=16384, A=18, H=256), drawn on the
    device, in the launch configuration the benchmark times; the oracle runs
    on 64 lanes spread over the batch."""
    from synth import SEED_BASE, head_batch_from_device, make_head_device
    from synth.trajectories import STRESS_SUBSET
    c = HEAD_WORKLOADS["stress"]
    log_case("head stress: generating on the device")
    d = make_head_device(c["T"], c["B"], c["A"], c["H"], SEED_BASE + 1004, "cuda")
    dev = dict(hidden=d["hidden"], head_weight=d["weight"], head_bias=d["bias"],
               behaviour_logits=d["behaviour_logits"], actions=d["actions"], rewards=d["rewards"],
               discounts=d["discounts"], bootstrap_value=d["bootstrap_value"])
    hb = head_batch_from_device(d, STRESS_SUBSET)
    for p in (Params(1.0, 1.0, 1.0), Params(1.0, 0.5, 0.95)):
        log_case(f"head stress {p.label()}")
        out = vt.vtrace_head_loss_grad(**dev, rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam,
                                       with_vs=True, with_pg_advantages=True, with_lane_losses=True,
                                       with_outputs=True)
        torch.cuda.synchronize()
        sub = {k: v[:, STRESS_SUBSET].cpu()
               for k, v in dict(outputs=out.outputs, vs=out.vs, pg_advantages=out.pg_advantages,
                                d_hidden=out.d_hidden).items()}
        view = vt.HeadLossGrad(out.losses, sub["d_hidden"], out.d_weight, out.d_bias, sub["vs"],
                               sub["pg_advantages"], out.lane_losses[STRESS_SUBSET], sub["outputs"])
        check_head(hb, p, view, whole=False)
        lane = np_out(out.lane_losses).astype(np.float64)
        assert np.allclose(np_out(out.losses)[1:], lane.sum(axis=0), rtol=1e-4, atol=1e-3)
        db = np_out(out.d_bias)
        assert abs(db[:c["A"]].sum()) <= 1e-4 * np.abs(db[:c["A"]]).sum() + 1e-5
        del out
    del d, dev
    torch.cuda.empty_cache()
