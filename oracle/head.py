"""Plain fp64 definition of the learner's output layer followed by the V-trace
actor-critic losses, and the gradients of those losses with respect to the
layer's input and parameters.

TEST INFRASTRUCTURE: see the package docstring.

Sec. 3.1: the learner computes every LSTM state of the unroll and then applies
the fully connected output layer to all time steps at once (time folded into
the batch).  Here that layer is one affine map per step,

    o[t, b, :] = hidden[t, b, :] @ weight + bias,     weight: [H, A + 1],

whose first A outputs are the policy logits z and whose last output is the
baseline V(x_t) (one layer for both heads; a reading, since the paper gives the
layer but not its split).  The losses are those of ``definitions.loss_and_grads``
on (z, V); their gradient with respect to o is G = [d_logits, d_values], and by
the chain rule

    d_hidden = G @ weight^T,   d_weight = sum over (t, b) of hidden^T G,
    d_bias   = sum over (t, b) of G.

The bootstrap value V(x_T) is an input, as in the plain loss: it is a target
and receives no gradient (Sec. 4.2).
"""

from __future__ import annotations

from typing import NamedTuple

import numpy as np

from .definitions import _f64, loss_and_grads


class HeadOut(NamedTuple):
    losses: np.ndarray       # [4] total, policy gradient, baseline, entropy
    lane_losses: np.ndarray  # [B, 3]
    d_hidden: np.ndarray     # [T, B, H]
    d_weight: np.ndarray     # [H, A + 1]
    d_bias: np.ndarray       # [A + 1]
    outputs: np.ndarray      # [T, B, A + 1]: policy logits, then the baseline
    d_outputs: np.ndarray    # [T, B, A + 1]: G = [d_logits, d_values]
    vs: np.ndarray           # [T, B]
    pg_advantages: np.ndarray
    step_losses: np.ndarray  # [T, B, 3]: per-step policy-gradient, baseline, entropy terms


def head_forward(hidden, weight, bias):
    """o = hidden @ weight + bias over every (t, b) (Sec. 3.1), in fp64."""
    return _f64(hidden) @ _f64(weight) + _f64(bias)


def head_loss_and_grads(hidden, weight, bias, behaviour_logits, actions, rewards, discounts,
                        bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0, baseline_cost=0.5,
                        entropy_cost=0.01, **variant) -> HeadOut:
    """Output layer, V-trace losses (Sec. 4.2) and gradients through the layer.

    ``variant`` takes the keyword arguments of ``loss_and_grads`` (correction,
    q_estimate, epsilon, behaviour, reward_transform)."""
    hidden = _f64(hidden)
    weight = _f64(weight)
    A = weight.shape[1] - 1
    o = head_forward(hidden, weight, bias)
    z, V = o[..., :A], o[..., A]
    lg = loss_and_grads(z, behaviour_logits, actions, rewards, discounts, V, bootstrap_value,
                        rho_bar, c_bar, lam, baseline_cost, entropy_cost, **variant)
    G = np.concatenate([lg.d_logits, lg.d_values[..., None]], axis=-1)
    H = hidden.shape[-1]
    d_hidden = G @ weight.T
    d_weight = hidden.reshape(-1, H).T @ G.reshape(-1, A + 1)
    d_bias = G.reshape(-1, A + 1).sum(axis=0)
    return HeadOut(lg.losses, lg.lane_losses, d_hidden, d_weight, d_bias, o, G, lg.vs,
                   lg.pg_advantages, lg.step_losses)


def sum_term_scale(hidden, d_outputs):
    """Root-sum-square of the terms hidden[r, h] * G[r, c] that make up each
    d_weight[h, c], and of the G[r, c] that make up d_bias[c]: the natural
    magnitude of these long sums, used to state their rounding tolerance."""
    H = hidden.shape[-1]
    C = d_outputs.shape[-1]
    h2 = _f64(hidden).reshape(-1, H) ** 2
    g2 = _f64(d_outputs).reshape(-1, C) ** 2
    return np.sqrt(h2.T @ g2), np.sqrt(g2.sum(axis=0))
