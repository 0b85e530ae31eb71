"""Plain fp64 definitions of V-trace and the V-trace actor-critic losses.

TEST INFRASTRUCTURE: see the package docstring.  Nothing here is blocked,
fused or reordered beyond what the paper's definitions state.

Notation (Sec. 4 of the paper), all arrays time-major:
  z = target_logits[t, b, :]     logits of the learner policy pi
  y = behaviour_logits[t, b, :]  logits of the actor policy mu
  a_t = actions[t, b], r_t = rewards[t, b], V(x_t) = values[t, b],
  V(x_T) = bootstrap_value[b].
``discounts[t, b]`` is gamma_t, the discount between x_t and x_{t+1}; 0 marks an
episode that ended after step t.  With a constant gamma this is exactly the
paper's gamma^(t-s); with per-step discounts gamma^(t-s) becomes the product
gamma_s ... gamma_{t-1}.

Readings where the paper is silent (each is also listed in the design notes):
  * every v_s uses the remaining steps of the unroll (n = T - s) and
    v_T = V(x_T) (the empty sum of Eq. (1));
  * lambda scales c only (Remark 2), never rho;
  * the policy gradient uses the same rho_t as delta_t V;
  * losses are summed over batch and time (App. D, hyperparameter-range table);
    baseline loss c_v * 1/2 * (v_s - V(x_s))^2, whose gradient is the paper's
    value direction scaled by c_v; entropy loss c_e * sum_a pi log pi, whose
    negative gradient is the paper's entropy-bonus direction;
  * rho, c, v_s and the advantages are targets: no gradient flows through them.

Correction variants (Sec. 5.2.3) and the alternative advantage of App. E.3 are
selected by ``correction`` and ``q_estimate``:
  * "vtrace": V-trace as above (the default);
  * "none": no off-policy correction: rho = c = 1 in the value target and no
    weight on the advantage; lambda still scales the trace, c_t = lambda;
  * "epsilon": as "none", and the policy-gradient term uses log(pi(a) + eps)
    instead of log pi(a) (eps = 1e-6 in the paper);
  * "one_step_is": value target without correction (as "none"), advantage
    multiplied by the truncated weight rho_s;
  * q_estimate "vtrace": q_s = r_s + gamma_s v_{s+1};
    q_estimate "baseline": q_s = r_s + gamma_s V(x_{s+1}).
"""

from __future__ import annotations

from typing import NamedTuple

import numpy as np

CORRECTIONS = ("vtrace", "none", "epsilon", "one_step_is")
Q_ESTIMATES = ("vtrace", "baseline")


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def log_softmax(logits):
    """log pi(.|x) over the action axis, with the row maximum subtracted first."""
    x = _f64(logits)
    m = x.max(axis=-1, keepdims=True)
    return x - (m + np.log(np.exp(x - m).sum(axis=-1, keepdims=True)))


def gather_action_logits(target_logits, behaviour_logits, actions):
    """Copies of z[a_t] and y[a_t] as a [T, B, 2] array, in the inputs' own dtype."""
    a = np.asarray(actions, dtype=np.int64)[..., None]
    z = np.take_along_axis(np.asarray(target_logits), a, axis=-1)[..., 0]
    y = np.take_along_axis(np.asarray(behaviour_logits), a, axis=-1)[..., 0]
    return np.stack([z, y], axis=-1)


def transform_rewards(rewards, kind=None):
    """Reward preprocessing of App. D: None leaves rewards as given; "clip" clips
    them to [-1, 1] (single tasks); "asymmetric" is the optimistic asymmetric
    clipping 0.3 min(tanh r, 0) + 5 max(tanh r, 0) (DMLab-30)."""
    r = _f64(rewards)
    if kind is None:
        return r
    if kind == "clip":
        return np.clip(r, -1.0, 1.0)
    if kind == "asymmetric":
        t = np.tanh(r)
        return 0.3 * np.minimum(t, 0.0) + 5.0 * np.maximum(t, 0.0)
    raise ValueError(kind)


def truncated_is_weights(target_logits, behaviour_logits, actions, rho_bar, c_bar, lam,
                         behaviour="logits"):
    """Truncated importance weights of Sec. 4.1, with lambda as in Remark 2.

    rho_t = min(rho_bar, pi(a_t|x_t) / mu(a_t|x_t))
    c_t   = lambda * min(c_bar, pi(a_t|x_t) / mu(a_t|x_t))
    ``behaviour_logits`` holds mu's logits [T, B, A], or, with
    behaviour="log_probs", log mu(a_t|x_t) itself [T, B] (what the actors send,
    Sec. 3).  Returns (log pi(a_t|x_t), log mu(a_t|x_t), rho, c).
    """
    a = np.asarray(actions, dtype=np.int64)
    A = np.shape(target_logits)[-1]
    if a.size and (a.min() < 0 or a.max() >= A):
        raise ValueError("action index out of range")
    log_pi_a = np.take_along_axis(log_softmax(target_logits), a[..., None], axis=-1)[..., 0]
    if behaviour == "logits":
        log_mu_a = np.take_along_axis(log_softmax(behaviour_logits), a[..., None], axis=-1)[..., 0]
    elif behaviour == "log_probs":
        log_mu_a = _f64(behaviour_logits)
    else:
        raise ValueError(behaviour)
    ratio = np.exp(log_pi_a - log_mu_a)
    rho = np.minimum(np.float64(rho_bar), ratio)
    c = np.float64(lam) * np.minimum(np.float64(c_bar), ratio)
    return log_pi_a, log_mu_a, rho, c


def _values_next(values, bootstrap_value):
    """V(x_{t+1}) for t = 0..T-1, with V(x_T) the bootstrap value."""
    return np.concatenate([_f64(values)[1:], _f64(bootstrap_value)[None]], axis=0)


def temporal_differences(rho, rewards, discounts, values, bootstrap_value):
    """delta_t V = rho_t (r_t + gamma_t V(x_{t+1}) - V(x_t))   (Sec. 4.1)."""
    return _f64(rho) * (_f64(rewards) + _f64(discounts) * _values_next(values, bootstrap_value)
                        - _f64(values))


def vtrace_targets_recursive(values, bootstrap_value, deltas, discounts, c):
    """Remark 1, walked backwards from v_T = V(x_T):

    v_s = V(x_s) + delta_s V + gamma_s c_s (v_{s+1} - V(x_{s+1})).
    """
    V = _f64(values)
    T = V.shape[0]
    V_ext = np.concatenate([V, _f64(bootstrap_value)[None]], axis=0)
    vs = np.empty_like(V_ext)
    vs[T] = V_ext[T]
    for s in range(T - 1, -1, -1):
        vs[s] = V_ext[s] + deltas[s] + _f64(discounts[s]) * c[s] * (vs[s + 1] - V_ext[s + 1])
    return vs[:T]


def vtrace_targets_direct_sum(values, deltas, discounts, c):
    """Eq. (1) summed term by term (O(T^2); small inputs only):

    v_s = V(x_s) + sum_{t=s}^{T-1} (gamma_s...gamma_{t-1}) (c_s...c_{t-1}) delta_t V,
    where an empty product is 1.
    """
    V = _f64(values)
    g = _f64(discounts)
    T = V.shape[0]
    vs = np.empty_like(V)
    for s in range(T):
        total = V[s].copy()
        for t in range(s, T):
            discount_prod = np.prod(g[s:t], axis=0)
            trace_prod = np.prod(c[s:t], axis=0)
            total = total + discount_prod * trace_prod * deltas[t]
        vs[s] = total
    return vs


def pg_advantages(rho, rewards, discounts, values, vs, bootstrap_value, q_estimate="vtrace"):
    """rho_s (q_s - V(x_s)) with q_s = r_s + gamma_s v_{s+1} and v_T = V(x_T)   (Sec. 4.2);
    with q_estimate="baseline", q_s = r_s + gamma_s V(x_{s+1})   (App. E.3)."""
    if q_estimate == "vtrace":
        nxt = np.concatenate([_f64(vs)[1:], _f64(bootstrap_value)[None]], axis=0)
    elif q_estimate == "baseline":
        nxt = _values_next(values, bootstrap_value)
    else:
        raise ValueError(q_estimate)
    q = _f64(rewards) + _f64(discounts) * nxt
    return _f64(rho) * (q - _f64(values))


class VtraceOut(NamedTuple):
    log_pi_a: np.ndarray
    log_mu_a: np.ndarray
    rho: np.ndarray
    c: np.ndarray
    deltas: np.ndarray
    vs: np.ndarray
    pg_advantages: np.ndarray


def vtrace(target_logits, behaviour_logits, actions, rewards, discounts, values,
           bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0, *, direct_sum=False,
           correction="vtrace", q_estimate="vtrace", behaviour="logits",
           reward_transform=None) -> VtraceOut:
    """V-trace targets v_s and policy-gradient advantages for a [T, B] batch.

    ``rho`` and ``c`` in the result are always the truncated weights; which of
    them enter the value target and the advantage depends on ``correction``.
    ``behaviour`` says what ``behaviour_logits`` holds (see truncated_is_weights);
    ``reward_transform`` preprocesses the rewards (see transform_rewards)."""
    if correction not in CORRECTIONS:
        raise ValueError(correction)
    rewards = transform_rewards(rewards, reward_transform)
    log_pi_a, log_mu_a, rho, c = truncated_is_weights(
        target_logits, behaviour_logits, actions, rho_bar, c_bar, lam, behaviour)
    if correction == "vtrace":
        rho_value, c_value, rho_pg = rho, c, rho
    else:
        ones = np.ones_like(rho)
        rho_value, c_value = ones, np.float64(lam) * ones
        rho_pg = rho if correction == "one_step_is" else ones
    deltas = temporal_differences(rho_value, rewards, discounts, values, bootstrap_value)
    if direct_sum:
        vs = vtrace_targets_direct_sum(values, deltas, discounts, c_value)
    else:
        vs = vtrace_targets_recursive(values, bootstrap_value, deltas, discounts, c_value)
    adv = pg_advantages(rho_pg, rewards, discounts, values, vs, bootstrap_value, q_estimate)
    return VtraceOut(log_pi_a, log_mu_a, rho, c, deltas, vs, adv)


class LossGradOut(NamedTuple):
    losses: np.ndarray  # [4]: total, policy-gradient, baseline, entropy
    lane_losses: np.ndarray  # [B, 3]: per-lane policy-gradient, baseline, entropy
    d_logits: np.ndarray  # [T, B, A]
    d_values: np.ndarray  # [T, B]
    vs: np.ndarray
    pg_advantages: np.ndarray
    step_losses: np.ndarray  # [T, B, 3]: the per-step terms the lane losses sum


def _pg_log_prob(log_pi_a, correction, epsilon):
    """log pi(a|x) in the policy-gradient term; log(pi(a|x) + eps) for "epsilon"."""
    if correction == "epsilon":
        return np.log(np.exp(log_pi_a) + np.float64(epsilon))
    return log_pi_a


def total_loss_frozen_targets(target_logits, values, actions, pg_adv, vs,
                              baseline_cost, entropy_cost, correction="vtrace", epsilon=1e-6):
    """Sum over batch and time of the three losses, with the targets held fixed.

    policy gradient: -pg_adv_s * log pi(a_s|x_s)   (log(pi + eps) for "epsilon")
    baseline:        baseline_cost * 1/2 * (v_s - V(x_s))^2
    entropy:         entropy_cost * sum_a pi(a|x_s) log pi(a|x_s)
    """
    log_pi = log_softmax(target_logits)
    a = np.asarray(actions, dtype=np.int64)[..., None]
    log_pi_a = np.take_along_axis(log_pi, a, axis=-1)[..., 0]
    pi = np.exp(log_pi)
    pg = -np.sum(_f64(pg_adv) * _pg_log_prob(log_pi_a, correction, epsilon))
    base = np.float64(baseline_cost) * 0.5 * np.sum((_f64(vs) - _f64(values)) ** 2)
    ent = np.float64(entropy_cost) * np.sum(pi * log_pi)
    return pg + base + ent


def loss_and_grads(target_logits, behaviour_logits, actions, rewards, discounts, values,
                   bootstrap_value, rho_bar=1.0, c_bar=1.0, lam=1.0,
                   baseline_cost=0.5, entropy_cost=0.01, *, correction="vtrace",
                   q_estimate="vtrace", epsilon=1e-6, behaviour="logits",
                   reward_transform=None) -> LossGradOut:
    """The three losses of the V-trace actor-critic update (Sec. 4.2) and their
    gradients with respect to the target logits and the values."""
    vt = vtrace(target_logits, behaviour_logits, actions, rewards, discounts, values,
                bootstrap_value, rho_bar, c_bar, lam, correction=correction,
                q_estimate=q_estimate, behaviour=behaviour, reward_transform=reward_transform)
    c_v = np.float64(baseline_cost)
    c_e = np.float64(entropy_cost)
    log_pi = log_softmax(target_logits)
    pi = np.exp(log_pi)
    neg_entropy = np.sum(pi * log_pi, axis=-1)  # sum_a pi log pi = -H

    pg_tb = -vt.pg_advantages * _pg_log_prob(vt.log_pi_a, correction, epsilon)
    base_tb = c_v * 0.5 * (vt.vs - _f64(values)) ** 2
    ent_tb = c_e * neg_entropy
    lane = np.stack([pg_tb.sum(axis=0), base_tb.sum(axis=0), ent_tb.sum(axis=0)], axis=-1)
    pg_l, base_l, ent_l = pg_tb.sum(), base_tb.sum(), ent_tb.sum()
    losses = np.array([pg_l + base_l + ent_l, pg_l, base_l, ent_l], dtype=np.float64)

    # d/dz_j of -adv*log pi_a is adv*(pi_j - 1[j = a]); of -adv*log(pi_a + eps)
    # it is adv*w*(pi_j - 1[j = a]) with w = pi_a/(pi_a + eps);
    # d/dz_j of sum_k pi_k log pi_k is pi_j*(log pi_j + H).
    onehot = np.zeros_like(pi)
    np.put_along_axis(onehot, np.asarray(actions, dtype=np.int64)[..., None], 1.0, axis=-1)
    entropy = -neg_entropy
    w = np.ones_like(vt.pg_advantages)
    if correction == "epsilon":
        pi_a = np.exp(vt.log_pi_a)
        w = pi_a / (pi_a + np.float64(epsilon))
    d_logits = ((vt.pg_advantages * w)[..., None] * (pi - onehot)
                + c_e * pi * (log_pi + entropy[..., None]))
    d_values = c_v * (_f64(values) - vt.vs)
    step_losses = np.stack([pg_tb, base_tb, ent_tb], axis=-1)
    return LossGradOut(losses, lane, d_logits, d_values, vt.vs, vt.pg_advantages, step_losses)
