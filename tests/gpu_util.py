"""Helpers for the GPU tests: device upload of synthetic batches and the parity
checks used throughout.

Every output is held element by element to |g - o| <= 1e-5 + 1e-4 |o|.  The
fused output-layer call's sums alone (its lane and total losses, d_W, d_b and
each d_hidden element) add a term kappa * RSS, RSS the root-sum-square of the
sum's terms and kappa the relative precision its terms are formed with
(``head_kappa_*``: the layer's float32 outputs, its bfloat16 high/low split of
dL/do and its float32 accumulation of d_W and d_b)."""

from __future__ import annotations

import dataclasses

import numpy as np
import torch

ATOL = 1e-5
RTOL = 1e-4


def require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU (run with -m 'not gpu' elsewhere)"


def log_case(msg: str):
    print(f"\n[case] {msg}", flush=True)


def to_device(tr, device="cuda"):
    """The batch as contiguous device tensors, logits in the kernel's dtype."""
    zt, yt = tr.logits_for_device()
    if tr.dtype == "bf16":
        z = torch.from_numpy(np.ascontiguousarray(zt).view(np.int16)).view(torch.bfloat16)
        y = torch.from_numpy(np.ascontiguousarray(yt).view(np.int16)).view(torch.bfloat16)
    else:
        z = torch.from_numpy(np.ascontiguousarray(zt))
        y = torch.from_numpy(np.ascontiguousarray(yt))
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(device)
    return dict(target_logits=z.to(device), behaviour_logits=y.to(device), actions=d(tr.actions),
                rewards=d(tr.rewards), discounts=d(tr.discounts), values=d(tr.values),
                bootstrap_value=d(tr.bootstrap_value))


def f32(x):
    """x as the float32 a C ABI float argument carries (infinities stay)."""
    return float(np.float32(x))


def call_params(p):
    """The call's scalars as the kernels receive them: the C ABI takes rho_bar,
    c_bar, lambda and the two loss costs as float32, so the oracle is evaluated
    at those float32 values (lambda = 0.95 arrives as 0.949999988...; where a
    lane's loss terms cancel, that difference alone moves its sum by more than
    the tolerance)."""
    return dataclasses.replace(p, rho_bar=f32(p.rho_bar), c_bar=f32(p.c_bar), lam=f32(p.lam),
                               baseline_cost=f32(p.baseline_cost), entropy_cost=f32(p.entropy_cost))


def oracle_args(tr):
    return (tr.target_logits, tr.behaviour_logits, tr.actions, tr.rewards, tr.discounts,
            tr.values, tr.bootstrap_value)


def np_out(t):
    return None if t is None else t.detach().float().cpu().numpy()


def assert_close(name, got, expect, rtol=RTOL, atol=ATOL):
    """|got - expect| <= atol + rtol*|expect| element by element, with a report
    of the worst element when it fails."""
    got = np.asarray(got, dtype=np.float64)
    expect = np.asarray(expect, dtype=np.float64)
    assert got.shape == expect.shape, (name, got.shape, expect.shape)
    err = np.abs(got - expect)
    bound = atol + rtol * np.abs(expect)
    bad = ~(err <= bound)  # NaN counts as a failure
    if bad.any():
        ratio = np.where(np.isfinite(err), err / bound, np.inf)
        worst = np.unravel_index(np.argmax(ratio), ratio.shape)
        raise AssertionError(
            f"{name}: {int(bad.sum())} of {bad.size} elements outside |err| <= {atol} + {rtol}|o|; "
            f"worst at {worst}: got {got[worst]!r} expected {expect[worst]!r}")


U32 = 2.0 ** -24  # float32 unit roundoff
G_SPLIT = 2.0 ** -17  # dL/do as a bfloat16 high and low pair: relative precision


def head_kappa_loss(H: int) -> float:
    """Relative precision of a loss term of the output-layer call: the layer's
    outputs are H-term bfloat16 dot products accumulated in float32, within
    about 2^-24 sqrt(H) of themselves, and the step's softmax statistics are
    float32 (a few roundings, 8 allowed)."""
    return U32 * (float(np.sqrt(H)) + 8.0)


def head_kappa_hidden(H: int) -> float:
    """Of a term G[c] W[k, c] of d_hidden: dL/do enters the product as a
    bfloat16 high and low pair (2^-17), computed from outputs within
    2^-24 sqrt(H)."""
    return G_SPLIT + U32 * float(np.sqrt(H))


def head_kappa_param(H: int, T: int, B: int) -> float:
    """Of a term of d_W or d_b: as for d_hidden, and the workgroup accumulates
    its terms in float32 over all its steps and lanes (about 2^-24 sqrt(n) for
    n of them: T steps of the 4-lane groups it walks, at most 512 workgroups)
    before the workgroups' partials are added in float64."""
    quads = -(-B // 4)
    nwg = min(quads, 512)
    n = T * 4 * (-(-quads // nwg))
    return G_SPLIT + U32 * (float(np.sqrt(H)) + float(np.sqrt(n)))


def assert_sum_close(name, got, expect, rss, kappa, rtol=RTOL, atol=ATOL):
    """|got - expect| <= atol + rtol |expect| + kappa rss: the element-wise bound
    plus kappa times the root-sum-square of the sum's terms."""
    got = np.asarray(got, dtype=np.float64)
    expect = np.asarray(expect, dtype=np.float64)
    assert got.shape == expect.shape, (name, got.shape, expect.shape)
    err = np.abs(got - expect)
    bound = atol + rtol * np.abs(expect) + kappa * np.asarray(rss, dtype=np.float64)
    bad = ~(err <= bound)
    if bad.any():
        ratio = np.where(np.isfinite(err), err / bound, np.inf)
        worst = np.unravel_index(np.argmax(ratio), ratio.shape)
        raise AssertionError(f"{name}: {int(bad.sum())} of {bad.size} outside the sum bound; worst at "
                             f"{worst}: got {got[worst]!r} expected {expect[worst]!r} rss "
                             f"{np.broadcast_to(rss, bound.shape)[worst]!r}")


def loss_term_rss(o):
    """Root-sum-square of the per-step terms behind the oracle's lane losses
    ([B, 3]) and loss totals ([4]: total, policy gradient, baseline, entropy)."""
    s2 = np.asarray(o.step_losses, dtype=np.float64) ** 2
    per_part = s2.sum(axis=(0, 1))
    return np.sqrt(s2.sum(axis=0)), np.sqrt(np.concatenate([[per_part.sum()], per_part]))
