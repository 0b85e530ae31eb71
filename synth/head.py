"""Seeded inputs for the learner's output layer followed by V-trace.

A batch holds the LSTM outputs of an unroll ``hidden[T, B, H]``, the parameters
of the fully connected output layer (``weight[H, A + 1]``, ``bias[A + 1]``; the
last column is the baseline), and the actor's side of the trajectories:
behaviour logits, actions, rewards, discounts and the bootstrap value.

Distributions
-------------
* hidden = tanh(N(0, 1)), rounded to bfloat16: LSTM outputs lie in (-1, 1);
  E[tanh(N(0,1))^2] is about 0.394.
* weight = N(0, 1 / (0.394 H)), rounded to bfloat16, so that the layer's outputs
  (the logits and the baseline) have roughly unit variance, like the logits of
  the plain workloads; bias = N(0, 0.1^2) in float32.
* behaviour logits = N(0, s^2), drawn independently of the layer (computing
  the layer's output here would put the method's arithmetic in the
  generator).  The two policies therefore differ more than a few updates of
  policy lag would make them, which exercises the truncation of the weights.
* actions: Gumbel-max samples from softmax(behaviour logits); rewards, discounts
  and the bootstrap value as in the Atari-shaped workload (rewards in
  {-1, 0, 1} w.p. {.05, .9, .05}, discount 0.99 with episode ends w.p.
  ``end_prob``, bootstrap N(0, 1)).

``make_head`` draws with NumPy (``Generator(PCG64)`` streams spawned from one
``SeedSequence``, one per quantity).  ``make_head_device`` draws the same kinds
of values with torch's seeded generator on a GPU, for batches too large to
build on the host; the two do not produce the same numbers.
"""

from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

from .trajectories import SEED_BASE, _gumbel_argmax, bf16_bits_to_f32, f32_to_bf16_bits

TANH_SQ_MEAN = 0.394  # E[tanh(X)^2] for X ~ N(0, 1), to three digits

HEAD_WORKLOADS = {
    "tiny": dict(T=5, B=4, A=9, H=64),
    "dmlab": dict(T=100, B=32, A=9, H=256),
    "atari": dict(T=20, B=32, A=18, H=256),
    "stress": dict(T=1000, B=16384, A=18, H=256),
}


@dataclasses.dataclass
class HeadBatch:
    T: int
    B: int
    A: int
    H: int
    hidden_bits: np.ndarray       # [T,B,H] uint16 (bfloat16)
    weight_bits: np.ndarray       # [H,A+1] uint16 (bfloat16)
    bias: np.ndarray              # [A+1] float32
    behaviour_logits: np.ndarray  # [T,B,A] float32
    actions: np.ndarray           # [T,B] int32
    rewards: np.ndarray           # [T,B] float32
    discounts: np.ndarray         # [T,B] float32
    bootstrap_value: np.ndarray   # [B] float32
    seed: Optional[int] = None

    @property
    def hidden(self) -> np.ndarray:
        """Exact float32 values of the bfloat16 hidden states."""
        return bf16_bits_to_f32(self.hidden_bits)

    @property
    def weight(self) -> np.ndarray:
        return bf16_bits_to_f32(self.weight_bits)


def make_head(T: int, B: int, A: int, H: int, seed: int, *, behaviour_std: float = 1.0,
              end_prob: float = 0.01, hidden_scale: float = 1.0,
              weight_scale: float = 1.0) -> HeadBatch:
    """A batch drawn on the host (small and medium shapes)."""
    ss = np.random.SeedSequence(seed)
    r_h, r_w, r_b, r_y, r_act, r_boot, r_rew, r_disc = [
        np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(8)
    ]
    hidden = np.tanh(r_h.standard_normal((T, B, H), dtype=np.float32)) * np.float32(hidden_scale)
    sw = weight_scale / np.sqrt(TANH_SQ_MEAN * H)
    weight = (r_w.standard_normal((H, A + 1), dtype=np.float32) * np.float32(sw))
    bias = (r_b.standard_normal(A + 1, dtype=np.float32) * np.float32(0.1))
    y = r_y.standard_normal((T, B, A), dtype=np.float32) * np.float32(behaviour_std)
    actions = _gumbel_argmax(r_act, y)
    bootstrap = r_boot.standard_normal(B, dtype=np.float32)
    u = r_rew.random((T, B))
    rewards = np.where(u < 0.05, -1.0, np.where(u < 0.95, 0.0, 1.0)).astype(np.float32)
    ends = r_disc.random((T, B)) < end_prob
    discounts = np.where(ends, 0.0, 0.99).astype(np.float32)
    return HeadBatch(T, B, A, H, f32_to_bf16_bits(hidden), f32_to_bf16_bits(weight), bias, y,
                     actions, rewards, discounts, bootstrap, seed)


def make_head_config(name: str) -> HeadBatch:
    c = HEAD_WORKLOADS[name]
    if name == "stress":
        raise ValueError("the stress head batch is drawn on the device: make_head_device")
    seed = SEED_BASE + 1000 + list(HEAD_WORKLOADS).index(name)
    return make_head(c["T"], c["B"], c["A"], c["H"], seed)


def subset_head_lanes(hb: HeadBatch, lanes: Sequence[int]) -> HeadBatch:
    idx = np.asarray(lanes, dtype=np.int64)
    pick = lambda x: np.ascontiguousarray(x[:, idx])
    return HeadBatch(hb.T, len(idx), hb.A, hb.H, pick(hb.hidden_bits), hb.weight_bits, hb.bias,
                     pick(hb.behaviour_logits), pick(hb.actions), pick(hb.rewards),
                     pick(hb.discounts), np.ascontiguousarray(hb.bootstrap_value[idx]), hb.seed)


def make_head_device(T: int, B: int, A: int, H: int, seed: int, device, *,
                     behaviour_std: float = 1.0, end_prob: float = 0.01):
    """The same kinds of draws as ``make_head``, made on ``device`` with torch's
    seeded generator in time-chunks.  Returns a dict of device tensors: hidden
    and weight as bfloat16, the rest float32 / int32."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed)
    dev = dict(device=device)
    hidden = torch.empty((T, B, H), dtype=torch.bfloat16, **dev)
    tc = max(1, (1 << 27) // max(1, B * H))
    for t0 in range(0, T, tc):
        t1 = min(T, t0 + tc)
        x = torch.randn((t1 - t0, B, H), generator=g, dtype=torch.float32, **dev)
        hidden[t0:t1] = torch.tanh(x).to(torch.bfloat16)
        del x
    sw = 1.0 / float(np.sqrt(TANH_SQ_MEAN * H))
    weight = (torch.randn((H, A + 1), generator=g, dtype=torch.float32, **dev) * sw).to(torch.bfloat16)
    bias = torch.randn(A + 1, generator=g, dtype=torch.float32, **dev) * 0.1
    y = torch.empty((T, B, A), dtype=torch.float32, **dev)
    actions = torch.empty((T, B), dtype=torch.int32, **dev)
    tc = max(1, (1 << 26) // max(1, B * A))
    for t0 in range(0, T, tc):
        t1 = min(T, t0 + tc)
        yc = torch.randn((t1 - t0, B, A), generator=g, dtype=torch.float32, **dev) * behaviour_std
        y[t0:t1] = yc
        u = torch.rand((t1 - t0, B, A), generator=g, dtype=torch.float64, **dev)
        gumbel = -torch.log(-torch.log(u.clamp_min(1e-300)))
        actions[t0:t1] = torch.argmax(yc.double() + gumbel, dim=-1).to(torch.int32)
        del yc, u, gumbel
    u = torch.rand((T, B), generator=g, dtype=torch.float64, **dev)
    rewards = torch.where(u < 0.05, -1.0, torch.where(u < 0.95, 0.0, 1.0)).to(torch.float32)
    ends = torch.rand((T, B), generator=g, dtype=torch.float64, **dev) < end_prob
    discounts = torch.where(ends, 0.0, 0.99).to(torch.float32)
    bootstrap = torch.randn(B, generator=g, dtype=torch.float32, **dev)
    return dict(hidden=hidden, weight=weight, bias=bias, behaviour_logits=y, actions=actions,
                rewards=rewards, discounts=discounts, bootstrap_value=bootstrap)


def head_batch_from_device(d, lanes: Optional[Sequence[int]] = None) -> HeadBatch:
    """Host copy of a device batch (all lanes, or the given ones) as a HeadBatch."""
    import torch

    def host(x):  # a [T, B, ...] tensor, restricted to the lanes
        if lanes is not None:
            x = x[:, torch.as_tensor(list(lanes), device=x.device)]
        return x.contiguous().cpu()

    def bits(x):
        return host(x).view(torch.int16).numpy().view(np.uint16)

    hid = bits(d["hidden"])
    T, B, H = hid.shape
    A = d["behaviour_logits"].shape[-1]
    boot = d["bootstrap_value"]
    if lanes is not None:
        boot = boot[torch.as_tensor(list(lanes), device=boot.device)]
    return HeadBatch(T, B, A, H, hid, d["weight"].contiguous().cpu().view(torch.int16).numpy().view(np.uint16),
                     d["bias"].cpu().numpy(), host(d["behaviour_logits"]).numpy(),
                     host(d["actions"]).numpy(), host(d["rewards"]).numpy(),
                     host(d["discounts"]).numpy(), boot.contiguous().cpu().numpy())
