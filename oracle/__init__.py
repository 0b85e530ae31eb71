"""fp64 CPU oracle for the learner-side V-trace actor-critic step.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
and the benchmark's CPU-baseline leg may import this package.  It shares no
code with the HIP library and the library never calls it; its inputs come from
the seeded generators in ``synth`` and nothing else.

Everything is evaluated in float64 with plain NumPy, one time step at a time,
in the order and notation of Sec. 4 of Espeholt et al. (2018).
"""

from .definitions import (  # noqa: F401
    VtraceOut,
    LossGradOut,
    log_softmax,
    gather_action_logits,
    truncated_is_weights,
    temporal_differences,
    vtrace_targets_recursive,
    vtrace_targets_direct_sum,
    pg_advantages,
    vtrace,
    loss_and_grads,
    total_loss_frozen_targets,
    transform_rewards,
)
from .head import HeadOut, head_forward, head_loss_and_grads, sum_term_scale  # noqa: F401
