"""Seeded synthetic V-trace learner batches.

Every array is time-major, ``[T, B]`` or ``[T, B, A]`` with the action axis
innermost, which is the layout the learner sees after folding time into the
batch (paper Sec. 3.1).  Shapes follow the paper's workloads:

* DeepMind Lab: 9 actions (action-set table, App. D), unroll n = 100, batch 32,
  discount 0.99, rewards clipped to [-1, 1] (fixed-hyperparameter table, App. D).
* Atari: the full 18-action set, unroll 20, batch 32 (App. G tables).
* DMLab-30: 30 tasks sharing one learner batch (Sec. 5.3).

No environment data exists here; these seeded draws stand in for it.

Random-number recipe
--------------------
``numpy.random.Generator(PCG64)`` streams spawned from
``SeedSequence(180201561 + 10 * config)``, one stream per quantity, in this
order: per-group parameters, target logits, behaviour noise, action Gumbel
noise, values, bootstrap values, rewards, discount mask.  Values stored in
float32 are drawn in float32.  Because each quantity has its own stream, the
large configuration can be generated in time-chunks and still yields exactly the
arrays an unchunked draw would.

Actions are sampled from the behaviour policy softmax(behaviour_logits) with the
Gumbel-max construction, ``a = argmax_j (y_j + g_j)`` with ``g_j ~ Gumbel(0, 1)``
drawn in float64.  This samples exactly from the softmax without evaluating it,
so the generator computes no part of the method.

bf16 variants round both logit tensors to bfloat16 (round-to-nearest-even)
before the actions are sampled; the float32 copies hold the exact upcast values,
so every consumer reads the same numbers.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

SEED_BASE = 180201561
_CHUNK_ELEMS = 1 << 23  # bound on [t-chunk, B, A] temporaries while generating


@dataclasses.dataclass
class Params:
    """Scalars of one V-trace call.  Defaults are the paper's: rho_bar = c_bar = 1
    (Sec. 5.2.3), baseline loss scaling 0.5 and entropy cost 0.01 (App. D/G)."""

    rho_bar: float = 1.0
    c_bar: float = 1.0
    lam: float = 1.0
    baseline_cost: float = 0.5
    entropy_cost: float = 0.01

    def label(self) -> str:
        def f(x):
            return "inf" if math.isinf(x) else f"{x:g}"
        return f"rho{f(self.rho_bar)}_c{f(self.c_bar)}_lam{f(self.lam)}"


@dataclasses.dataclass
class Trajectories:
    """One learner batch.  ``target_logits``/``behaviour_logits`` are float32
    (for bf16 batches: the exact upcast of ``*_bits``)."""

    name: str
    T: int
    B: int
    A: int
    dtype: str  # "f32" or "bf16": the logits dtype handed to the kernel
    target_logits: np.ndarray  # [T,B,A] float32
    behaviour_logits: np.ndarray  # [T,B,A] float32
    actions: np.ndarray  # [T,B] int32
    rewards: np.ndarray  # [T,B] float32
    discounts: np.ndarray  # [T,B] float32
    values: np.ndarray  # [T,B] float32
    bootstrap_value: np.ndarray  # [B] float32
    target_bits: Optional[np.ndarray] = None  # [T,B,A] uint16 when dtype == "bf16"
    behaviour_bits: Optional[np.ndarray] = None
    seed: Optional[int] = None

    @property
    def steps(self) -> int:
        return self.T * self.B

    def logits_for_device(self):
        """The two logit tensors in the dtype the kernel reads."""
        if self.dtype == "bf16":
            return self.target_bits, self.behaviour_bits
        return self.target_logits, self.behaviour_logits


WORKLOADS = {
    0: dict(name="tiny", T=5, B=4, A=9),
    1: dict(name="dmlab", T=100, B=32, A=9),
    2: dict(name="atari", T=20, B=32, A=18),
    3: dict(name="multitask", T=100, B=4096, A=9),
    4: dict(name="stress", T=1000, B=16384, A=18),
}

PARAM_SETS = {
    0: [Params()],
    1: [Params()],
    2: [Params()],
    3: [Params()],
    4: [
        Params(1.0, 1.0, 1.0),
        Params(math.inf, math.inf, 1.0),
        Params(1.0, 0.5, 0.95),
    ],
}

# Lanes of the large configuration that the oracle evaluates: b_k = round(k*(B-1)/63).
STRESS_SUBSET = [int(round(k * 16383 / 63)) for k in range(64)]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest-even), returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _gumbel_argmax(rng: np.random.Generator, logits: np.ndarray) -> np.ndarray:
    """Sample one action per row from softmax(logits) by the Gumbel-max trick."""
    T, B, A = logits.shape
    out = np.empty((T, B), dtype=np.int32)
    tc = max(1, _CHUNK_ELEMS // max(1, B * A))
    for t0 in range(0, T, tc):
        t1 = min(T, t0 + tc)
        g = rng.gumbel(size=(t1 - t0, B, A))
        g += logits[t0:t1]
        out[t0:t1] = np.argmax(g, axis=-1)
    return out


def _normal_f32(rng, shape, out=None):
    if out is None:
        return rng.standard_normal(shape, dtype=np.float32)
    rng.standard_normal(dtype=np.float32, out=out)
    return out


def _generate(name, T, B, A, seed, *, noise_std, reward_kind, end_prob,
              groups=0, logit_scale=1.0, bf16=False, discount=0.99):
    ss = np.random.SeedSequence(seed)
    (r_grp, r_tgt, r_noise, r_act, r_val, r_boot, r_rew, r_disc) = [
        np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(8)
    ]

    # Per-task-group parameters (multi-task batch): reward scale 10^U[-1,1] and
    # behaviour-noise std U[0.1, 1.5]; lanes are split into contiguous groups.
    lane_scale = np.ones(B, dtype=np.float32)
    lane_std = np.full(B, noise_std, dtype=np.float32)
    if groups:
        g_scale = (10.0 ** r_grp.uniform(-1.0, 1.0, size=groups)).astype(np.float32)
        g_std = r_grp.uniform(0.1, 1.5, size=groups).astype(np.float32)
        gid = (np.arange(B) * groups) // B
        lane_scale = g_scale[gid]
        lane_std = g_std[gid]

    z = np.empty((T, B, A), dtype=np.float32)
    y = np.empty((T, B, A), dtype=np.float32)
    tc = max(1, _CHUNK_ELEMS // max(1, B * A))
    for t0 in range(0, T, tc):
        t1 = min(T, t0 + tc)
        _normal_f32(r_tgt, None, out=z[t0:t1])
        if logit_scale != 1.0:
            z[t0:t1] *= np.float32(logit_scale)
    for t0 in range(0, T, tc):
        t1 = min(T, t0 + tc)
        _normal_f32(r_noise, None, out=y[t0:t1])
        y[t0:t1] *= lane_std[None, :, None]
        y[t0:t1] += z[t0:t1]

    zb = yb = None
    if bf16:
        zb = f32_to_bf16_bits(z)
        yb = f32_to_bf16_bits(y)
        z = bf16_bits_to_f32(zb)
        y = bf16_bits_to_f32(yb)

    actions = _gumbel_argmax(r_act, y)
    values = r_val.standard_normal((T, B), dtype=np.float32)
    bootstrap = r_boot.standard_normal(B, dtype=np.float32)

    if reward_kind == "uniform":
        rewards = r_rew.uniform(-1.0, 1.0, size=(T, B)).astype(np.float32)
    elif reward_kind == "sparse":
        # 0 w.p. 0.9, else U[0, 10]; scaled per task group, then clipped to [-1, 1].
        hit = r_rew.random((T, B)) >= 0.9
        mag = r_rew.uniform(0.0, 10.0, size=(T, B))
        base = np.where(hit, mag, 0.0) * lane_scale[None, :]
        rewards = np.clip(base, -1.0, 1.0).astype(np.float32)
    elif reward_kind == "ternary":
        u = r_rew.random((T, B))
        rewards = np.where(u < 0.05, -1.0, np.where(u < 0.95, 0.0, 1.0)).astype(np.float32)
    else:
        raise ValueError(reward_kind)

    ends = r_disc.random((T, B)) < end_prob
    discounts = np.where(ends, 0.0, discount).astype(np.float32)

    return Trajectories(
        name=name, T=T, B=B, A=A, dtype="bf16" if bf16 else "f32",
        target_logits=z, behaviour_logits=y, actions=actions,
        rewards=rewards, discounts=discounts, values=values,
        bootstrap_value=bootstrap, target_bits=zb, behaviour_bits=yb, seed=seed,
    )


def make_config(cfg: int, bf16: bool = False) -> Trajectories:
    """The five fixed workloads (tiny, DMLab-shaped, Atari-shaped, 30-task, stress)."""
    c = WORKLOADS[cfg]
    seed = SEED_BASE + 10 * cfg
    name = c["name"] + ("_bf16" if bf16 else "")
    T, B, A = c["T"], c["B"], c["A"]
    if cfg == 0:
        return _generate(name, T, B, A, seed, noise_std=0.5, reward_kind="uniform",
                         end_prob=0.05, bf16=bf16)
    if cfg == 1:
        return _generate(name, T, B, A, seed, noise_std=0.5, reward_kind="sparse",
                         end_prob=0.001, bf16=bf16)
    if cfg == 2:
        return _generate(name, T, B, A, seed, noise_std=1.0, reward_kind="ternary",
                         end_prob=0.01, bf16=bf16)
    if cfg == 3:
        return _generate(name, T, B, A, seed, noise_std=0.5, reward_kind="sparse",
                         end_prob=0.002, groups=30, bf16=bf16)
    if cfg == 4:
        return _generate(name, T, B, A, seed, noise_std=1.0, reward_kind="ternary",
                         end_prob=0.01, bf16=bf16)
    raise KeyError(cfg)


def make_random(T: int, B: int, A: int, seed: int, *, noise_std: float = 0.5,
                end_prob: float = 0.05, logit_scale: float = 1.0, bf16: bool = False,
                reward_kind: str = "uniform", discount: float = 0.99) -> Trajectories:
    """A batch of arbitrary shape for edge-case and property tests."""
    return _generate(f"random_T{T}_B{B}_A{A}_s{seed}", T, B, A, seed,
                     noise_std=noise_std, reward_kind=reward_kind, end_prob=end_prob,
                     logit_scale=logit_scale, bf16=bf16, discount=discount)


def subset_lanes(tr: Trajectories, lanes: Sequence[int]) -> Trajectories:
    """Copy of ``tr`` restricted to the given lanes (columns of B)."""
    idx = np.asarray(lanes, dtype=np.int64)
    pick = lambda x: None if x is None else np.ascontiguousarray(x[:, idx])
    return Trajectories(
        name=f"{tr.name}[{len(idx)} lanes]", T=tr.T, B=len(idx), A=tr.A, dtype=tr.dtype,
        target_logits=pick(tr.target_logits), behaviour_logits=pick(tr.behaviour_logits),
        actions=pick(tr.actions), rewards=pick(tr.rewards), discounts=pick(tr.discounts),
        values=pick(tr.values), bootstrap_value=np.ascontiguousarray(tr.bootstrap_value[idx]),
        target_bits=pick(tr.target_bits), behaviour_bits=pick(tr.behaviour_bits), seed=tr.seed,
    )
