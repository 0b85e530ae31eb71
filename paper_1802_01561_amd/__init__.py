"""libvtrace: the learner-side V-trace actor-critic step of IMPALA
(Espeholt et al., 2018) as hand-written HIP kernels for AMD Instinct MI355X.

The computation lives in ``libvtrace.so`` (C ABI in ``include/vtrace.h``);
this package only loads it and marshals torch tensors into it.
"""

from ._lib import LIB_PATH, VtraceError  # noqa: F401
from .binding import (  # noqa: F401
    HeadLossGrad,
    LossGrad,
    Workspace,
    vtrace_abi_version,
    vtrace_error_flag,
    vtrace_gather_logits,
    vtrace_head_loss_grad,
    vtrace_head_workspace_bytes,
    vtrace_loss_grad,
    vtrace_loss_grad_static,
    vtrace_max_elements,
    vtrace_targets,
    vtrace_workspace_bytes,
)
