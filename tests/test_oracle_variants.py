"""Pins of the oracle's correction variants (Sec. 5.2.3) and of the alternative
advantage estimate q_s = r_s + gamma_s V(x_{s+1}) (App. E.3).

Each variant is checked against a statement that does not go through the
oracle's own V-trace code: the on-policy closed forms (Eq. (2) with per-step
discounts, the lambda-return of Remark 2), importance ratios from
scipy.special.softmax, torch autograd of the epsilon-corrected log-probability,
finite differences, and the identity "advantage with q_s = r_s + gamma_s V(x_{s+1})
is the temporal difference delta_s".  Mutation tests plant mistakes in copies
of the oracle and check that these pins catch them.
"""

import math

import numpy as np
import pytest
import scipy.special

import oracle
from oracle import definitions as ov
from synth import make_random

EPS = 1e-6


def _args(tr):
    return (tr.target_logits, tr.behaviour_logits, tr.actions, tr.rewards, tr.discounts,
            tr.values, tr.bootstrap_value)


def _batch(seed, T=9, B=4, A=5, end_prob=0.15, noise=1.0):
    return make_random(T, B, A, 2000 + seed, noise_std=noise, end_prob=end_prob)


def _lambda_return(tr, lam):
    """Truncated lambda-return G_s = r_s + gamma_s((1-lam) V(x_{s+1}) + lam G_{s+1}),
    G_T = V(x_T): the on-policy target (n-step Bellman target when lam = 1)."""
    T = tr.T
    V = np.concatenate([tr.values, tr.bootstrap_value[None]]).astype(np.float64)
    G = np.empty((T + 1, tr.B))
    G[T] = V[T]
    for s in range(T - 1, -1, -1):
        G[s] = tr.rewards[s] + tr.discounts[s].astype(np.float64) * ((1 - lam) * V[s + 1] + lam * G[s + 1])
    return G[:T]


def _ratio(tr):
    pi = scipy.special.softmax(tr.target_logits.astype(np.float64), axis=-1)
    mu = scipy.special.softmax(tr.behaviour_logits.astype(np.float64), axis=-1)
    a = tr.actions[..., None].astype(np.int64)
    return (np.take_along_axis(pi, a, -1) / np.take_along_axis(mu, a, -1))[..., 0], pi


def _onpolicy_adv(tr, G):
    nxt = np.concatenate([G[1:], tr.bootstrap_value[None].astype(np.float64)])
    return tr.rewards.astype(np.float64) + tr.discounts.astype(np.float64) * nxt - tr.values


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("lam", [1.0, 0.9, 0.0])
@pytest.mark.parametrize("params", [(1.0, 1.0), (math.inf, math.inf), (2.0, 0.5)])
def test_no_correction_is_the_on_policy_target(seed, lam, params):
    """No-correction ignores mu: its target is the on-policy lambda-return and its
    advantage carries no weight, whatever the behaviour policy and truncation levels."""
    tr = _batch(seed)
    out = oracle.vtrace(*_args(tr), params[0], params[1], lam, correction="none")
    G = _lambda_return(tr, lam)
    np.testing.assert_allclose(out.vs, G, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out.pg_advantages, _onpolicy_adv(tr, G), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("rho_bar", [1.0, 10.0, math.inf])
def test_one_step_importance_sampling(seed, rho_bar):
    """Value target without correction; advantage times the truncated weight."""
    tr = _batch(seed)
    out = oracle.vtrace(*_args(tr), rho_bar, 1.0, 1.0, correction="one_step_is")
    G = _lambda_return(tr, 1.0)
    ratio, _ = _ratio(tr)
    np.testing.assert_allclose(out.vs, G, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out.pg_advantages, np.minimum(rho_bar, ratio) * _onpolicy_adv(tr, G),
                               rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("correction", ["vtrace", "none", "one_step_is"])
def test_baseline_q_estimate_is_the_temporal_difference(seed, correction):
    """With q_s = r_s + gamma_s V(x_{s+1}) the advantage rho_s (q_s - V(x_s)) is the
    one-step temporal difference weighted as the correction prescribes."""
    tr = _batch(seed)
    out = oracle.vtrace(*_args(tr), 1.0, 1.0, 1.0, correction=correction, q_estimate="baseline")
    ratio, _ = _ratio(tr)
    V = tr.values.astype(np.float64)
    Vn = np.concatenate([V[1:], tr.bootstrap_value[None].astype(np.float64)])
    td = tr.rewards + tr.discounts * Vn - V
    w = np.ones_like(ratio) if correction == "none" else np.minimum(1.0, ratio)
    np.testing.assert_allclose(out.pg_advantages, w * td, rtol=1e-11, atol=1e-13)
    # the value target is unaffected by the choice of q_s
    ref = oracle.vtrace(*_args(tr), 1.0, 1.0, 1.0, correction=correction)
    np.testing.assert_array_equal(out.vs, ref.vs)


@pytest.mark.parametrize("seed", range(4))
def test_epsilon_correction_gradient_via_autograd(seed):
    """The epsilon-corrected policy-gradient term -adv log(pi(a) + eps), with the
    baseline and entropy terms, differentiated by torch autograd in fp64."""
    torch = pytest.importorskip("torch")
    tr = _batch(seed, A=6, noise=1.5)
    # push some pi(a) towards eps so that the correction matters
    tr.target_logits[..., 0] += np.float32(-14.0)
    tr.actions[::2, :] = 0
    cv, ce = 0.5, 0.05
    out = oracle.loss_and_grads(*_args(tr), 1.0, 1.0, 1.0, cv, ce, correction="epsilon", epsilon=EPS)
    G = _lambda_return(tr, 1.0)
    adv = _onpolicy_adv(tr, G)
    np.testing.assert_allclose(out.pg_advantages, adv, rtol=1e-12, atol=1e-12)
    z = torch.tensor(tr.target_logits, dtype=torch.float64, requires_grad=True)
    V = torch.tensor(tr.values, dtype=torch.float64, requires_grad=True)
    a = torch.tensor(tr.actions, dtype=torch.int64)
    p = torch.softmax(z, dim=-1)
    logp = torch.log_softmax(z, dim=-1)
    pa = p.gather(-1, a[..., None])[..., 0]
    objective = (-(torch.tensor(adv) * torch.log(pa + EPS)).sum()
                 + cv * 0.5 * ((torch.tensor(G) - V) ** 2).sum() + ce * (p * logp).sum())
    objective.backward()
    np.testing.assert_allclose(out.d_logits, z.grad.numpy(), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(out.d_values, V.grad.numpy(), rtol=1e-12, atol=1e-14)
    assert out.losses[0] == pytest.approx(objective.item(), rel=1e-12)


@pytest.mark.parametrize("correction", ["none", "epsilon", "one_step_is"])
def test_variant_gradients_central_differences(correction):
    tr = _batch(7, T=5, B=3, A=4)
    cv, ce = 0.5, 0.2
    out = oracle.loss_and_grads(*_args(tr), 2.0, 1.0, 0.9, cv, ce, correction=correction,
                                q_estimate="baseline", epsilon=0.05)
    f = lambda zz, VV: ov.total_loss_frozen_targets(zz, VV, tr.actions, out.pg_advantages, out.vs,
                                                     cv, ce, correction=correction, epsilon=0.05)
    z0 = tr.target_logits.astype(np.float64)
    V0 = tr.values.astype(np.float64)
    h = 1e-6
    for idx in np.ndindex(*z0.shape):
        zp, zm = z0.copy(), z0.copy()
        zp[idx] += h
        zm[idx] -= h
        assert (f(zp, V0) - f(zm, V0)) / (2 * h) == pytest.approx(out.d_logits[idx], rel=1e-6, abs=1e-8)
    for idx in np.ndindex(*V0.shape):
        vp, vm = V0.copy(), V0.copy()
        vp[idx] += h
        vm[idx] -= h
        assert (f(z0, vp) - f(z0, vm)) / (2 * h) == pytest.approx(out.d_values[idx], rel=1e-6, abs=1e-8)


def test_unknown_variant_rejected():
    tr = _batch(0)
    with pytest.raises(ValueError):
        oracle.vtrace(*_args(tr), correction="retrace")
    with pytest.raises(ValueError):
        oracle.vtrace(*_args(tr), q_estimate="v")


# --------------------------------------------------------------------------------------
# Mutation tests for the variants
# --------------------------------------------------------------------------------------

def _variant_pins_pass(mod):
    ok = True
    for seed in range(3):
        tr = _batch(seed)
        G1 = _lambda_return(tr, 1.0)
        G9 = _lambda_return(tr, 0.9)
        ratio, _ = _ratio(tr)
        o = mod.vtrace(*_args(tr), 2.0, 2.0, 0.9, correction="none")
        ok &= np.allclose(o.vs, G9, rtol=1e-10, atol=1e-12)
        ok &= np.allclose(o.pg_advantages, _onpolicy_adv(tr, G9), rtol=1e-10, atol=1e-12)
        o = mod.vtrace(*_args(tr), 2.0, 1.0, 1.0, correction="one_step_is")
        ok &= np.allclose(o.vs, G1, rtol=1e-10, atol=1e-12)
        ok &= np.allclose(o.pg_advantages, np.minimum(2.0, ratio) * _onpolicy_adv(tr, G1),
                          rtol=1e-10, atol=1e-12)
        o = mod.vtrace(*_args(tr), 1.0, 1.0, 1.0, q_estimate="baseline")
        V = tr.values.astype(np.float64)
        Vn = np.concatenate([V[1:], tr.bootstrap_value[None].astype(np.float64)])
        ok &= np.allclose(o.pg_advantages, np.minimum(1.0, ratio) * (tr.rewards + tr.discounts * Vn - V),
                          rtol=1e-10, atol=1e-12)
        lg = mod.loss_and_grads(*_args(tr), 1.0, 1.0, 1.0, 0.5, 0.1, correction="epsilon", epsilon=0.3)
        f = lambda zz: ov.total_loss_frozen_targets(zz, tr.values, tr.actions, lg.pg_advantages, lg.vs,
                                                     0.5, 0.1, correction="epsilon", epsilon=0.3)
        _, pi = _ratio(tr)
        pa = np.take_along_axis(pi, tr.actions[..., None].astype(np.int64), -1)[..., 0]
        ok &= np.isclose(lg.losses[1], -np.sum(lg.pg_advantages * np.log(pa + 0.3)), rtol=1e-10)
        z0 = tr.target_logits.astype(np.float64)
        for j in range(tr.A):
            idx = (0, 0, j)
            zp, zm = z0.copy(), z0.copy()
            zp[idx] += 1e-6
            zm[idx] -= 1e-6
            ok &= abs((f(zp) - f(zm)) / 2e-6 - lg.d_logits[idx]) < 1e-6
    return bool(ok)


def _mutant(replacements):
    import inspect
    import types
    src = inspect.getsource(ov)
    for old, new in replacements:
        assert old in src, old
        src = src.replace(old, new, 1)
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src, "oracle_mutant", "exec"), mod.__dict__)
    return mod


VARIANT_MUTATIONS = {
    "none_keeps_rho_in_delta": [("rho_value, c_value = ones, np.float64(lam) * ones",
                                 "rho_value, c_value = rho, np.float64(lam) * ones")],
    "none_drops_lambda": [("rho_value, c_value = ones, np.float64(lam) * ones",
                           "rho_value, c_value = ones, ones")],
    "one_step_is_drops_weight": [('rho_pg = rho if correction == "one_step_is" else ones',
                                  "rho_pg = ones")],
    "baseline_q_uses_vs": [("nxt = _values_next(values, bootstrap_value)",
                            "nxt = np.concatenate([_f64(vs)[1:], _f64(bootstrap_value)[None]], axis=0)")],
    "epsilon_weight_missing": [("w = pi_a / (pi_a + np.float64(epsilon))", "w = np.ones_like(pi_a)")],
    "epsilon_in_log_missing": [("return np.log(np.exp(log_pi_a) + np.float64(epsilon))", "return log_pi_a")],
}


def test_unmutated_oracle_passes_variant_pins():
    assert _variant_pins_pass(ov)


@pytest.mark.parametrize("name", sorted(VARIANT_MUTATIONS))
def test_planted_variant_mistake_is_caught(name):
    assert not _variant_pins_pass(_mutant(VARIANT_MUTATIONS[name]))


# --------------------------------------------------------------------------------------
# Input/output variants: behaviour log-probabilities, reward preprocessing
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("correction", ["vtrace", "one_step_is", "epsilon"])
def test_behaviour_log_probs_input(seed, correction):
    """Passing log mu(a_t|x_t) (here from scipy's log-softmax) instead of mu's
    logits gives the same result."""
    tr = _batch(seed)
    lmu = np.take_along_axis(scipy.special.log_softmax(tr.behaviour_logits.astype(np.float64), -1),
                             tr.actions[..., None].astype(np.int64), -1)[..., 0]
    a = oracle.loss_and_grads(*_args(tr), 2.0, 1.0, 0.9, correction=correction)
    args = list(_args(tr))
    args[1] = lmu
    b = oracle.loss_and_grads(*args, 2.0, 1.0, 0.9, correction=correction, behaviour="log_probs")
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-13)


def test_reward_transforms():
    r = np.array([-50.0, -1.5, -1.0, -0.3, 0.0, 0.4, math.atanh(0.5), 1.0, 2.0, 80.0])
    clip = ov.transform_rewards(r, "clip")
    assert clip.tolist() == [-1.0, -1.0, -1.0, -0.3, 0.0, 0.4, math.atanh(0.5), 1.0, 1.0, 1.0]
    asym = ov.transform_rewards(r, "asymmetric")
    # 0.3 min(tanh r, 0) + 5 max(tanh r, 0): 0 at 0, 2.5 where tanh r = 1/2, limits -0.3 and 5
    assert asym[4] == 0.0
    assert asym[6] == pytest.approx(2.5, rel=1e-15)
    assert asym[0] == pytest.approx(-0.3, rel=1e-15) and asym[-1] == pytest.approx(5.0, rel=1e-15)
    assert asym[3] == pytest.approx(0.3 * math.tanh(-0.3), rel=1e-15)
    assert np.all(np.diff(asym) >= 0)
    assert ov.transform_rewards(r, None).tolist() == r.tolist()
    with pytest.raises(ValueError):
        ov.transform_rewards(r, "tanh")


@pytest.mark.parametrize("kind", ["clip", "asymmetric"])
def test_reward_transform_is_applied_first(kind):
    """The preprocessed batch equals the raw batch with transformed rewards."""
    tr = _batch(3)
    tr.rewards = (tr.rewards * 4).astype(np.float32)
    a = oracle.loss_and_grads(*_args(tr), 1.0, 1.0, 1.0, reward_transform=kind)
    args = list(_args(tr))
    args[3] = np.clip(tr.rewards.astype(np.float64), -1, 1) if kind == "clip" else \
        np.where(tr.rewards < 0, 0.3, 5.0) * np.tanh(tr.rewards.astype(np.float64))
    b = oracle.loss_and_grads(*args, 1.0, 1.0, 1.0)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-13, atol=1e-14)
