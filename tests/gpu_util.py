"""Helpers for the GPU tests: device upload of synthetic batches and the
element-wise parity check used throughout."""

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
