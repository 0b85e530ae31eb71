"""Seeded synthetic trajectory batches shaped like the IMPALA paper's learner workloads.

This package only draws random inputs (logits, actions, rewards, discounts,
values).  It holds none of the V-trace arithmetic: both the fp64 oracle and
the HIP path consume what it produces, and neither imports the other.
"""

from .trajectories import (  # noqa: F401
    WORKLOADS,
    PARAM_SETS,
    SEED_BASE,
    Params,
    Trajectories,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_config,
    make_random,
    subset_lanes,
)
from .head import (  # noqa: F401
    HEAD_WORKLOADS,
    HeadBatch,
    head_batch_from_device,
    make_head,
    make_head_config,
    make_head_device,
    subset_head_lanes,
)
