"""vtrace_loss_grad_static, the loss entry point that allocates nothing, through
the C ABI: two calls in a row, the second on a smaller batch, each against
vtrace_loss_grad_ex on the same inputs (bit for bit: the same kernels, with
their workspace in the library's fixed device array instead of the caller's)
and against the oracle (element-wise 1e-5 + 1e-4|o|).  Outputs are
preallocated, so nothing in the timed calls allocates."""

import numpy as np
import pytest
import torch

import oracle
import paper_1802_01561_amd as vt
from gpu_util import assert_close, call_params, log_case, np_out, oracle_args, require_gpu, to_device
from synth import PARAM_SETS, make_config, make_random

pytestmark = pytest.mark.gpu


def _outputs(T, B, A):
    f32 = dict(dtype=torch.float32, device="cuda")
    return vt.LossGrad(torch.empty(4, **f32), torch.empty((T, B, A), **f32),
                       torch.empty((T, B), **f32), torch.empty((T, B), **f32),
                       torch.empty((T, B), **f32), torch.empty((B, 3), **f32))


def _same_bits(name, got, expect):
    g, e = np_out(got), np_out(expect)
    assert g.tobytes() == e.tobytes(), f"{name}: static and workspace calls differ"


def test_static_entry_matches_workspace_entry_twice():
    require_gpu()
    cases = [(make_config(3), PARAM_SETS[3][0]),                       # T=100 B=4096 A=9
             (make_random(37, 300, 18, 4242, noise_std=1.0), PARAM_SETS[4][1])]  # smaller, (inf, inf, 1)
    for tr, p in cases:
        log_case(f"static entry T={tr.T} B={tr.B} A={tr.A} {p.label()}")
        dev = to_device(tr)
        kw = dict(rho_bar=p.rho_bar, c_bar=p.c_bar, lam=p.lam, baseline_cost=p.baseline_cost,
                  entropy_cost=p.entropy_cost)
        ref = vt.vtrace_loss_grad(**dev, **kw, out=_outputs(tr.T, tr.B, tr.A))
        out = vt.vtrace_loss_grad_static(**dev, **kw, out=_outputs(tr.T, tr.B, tr.A))
        torch.cuda.synchronize()
        for name in ("losses", "d_logits", "d_values", "vs", "pg_advantages", "lane_losses"):
            _same_bits(name, getattr(out, name), getattr(ref, name))
        q = call_params(p)
        o = oracle.loss_and_grads(*oracle_args(tr), q.rho_bar, q.c_bar, q.lam, q.baseline_cost,
                                  q.entropy_cost)
        assert_close("vs", np_out(out.vs), o.vs)
        assert_close("pg_advantages", np_out(out.pg_advantages), o.pg_advantages)
        assert_close("d_logits", np_out(out.d_logits), o.d_logits)
        assert_close("d_values", np_out(out.d_values), o.d_values)
        assert_close("lane_losses", np_out(out.lane_losses), o.lane_losses)
        assert_close("losses", np_out(out.losses), o.losses)


def test_static_entry_rejects_wide_batches():
    require_gpu()
    tr = make_random(2, 65537, 2, 5, noise_std=1.0)
    with pytest.raises(vt.VtraceError, match="WORKSPACE"):
        vt.vtrace_loss_grad_static(**to_device(tr))
