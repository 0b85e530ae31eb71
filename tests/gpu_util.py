"""Helpers for the GPU tests: device upload of synthetic batches and the parity
checks used throughout.

Element-wise outputs meet |g - o| <= 1e-5 + 1e-4 |o|.  Outputs that are sums of
many terms (a lane's loss over its steps, the loss totals over the batch) are
held to |g - o| <= 1e-5 + 1e-4 |o| + 1e-4 RSS, RSS the root-sum-square of the
terms: each term within 1e-4 of itself gives, for independent errors, an
error of about 1e-4 RSS in the sum.  When the terms cancel (a policy-gradient
loss of a few hundredths from a thousand terms of order one) that is far more
than 1e-4 of the total: the float32 log-probability in each term alone
contributes about 1e-7 of it per step."""

from __future__ import annotations

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


def assert_sum_close(name, got, expect, rss, rtol=RTOL, atol=ATOL):
    """The sum bound above, |got - expect| <= atol + rtol (|expect| + rss)."""
    got = np.asarray(got, dtype=np.float64)
    expect = np.asarray(expect, dtype=np.float64)
    assert got.shape == expect.shape, (name, got.shape, expect.shape)
    err = np.abs(got - expect)
    bound = atol + rtol * np.abs(expect) + rtol * np.asarray(rss, dtype=np.float64)
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
