"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these checks retypes an oracle formula: each compares the oracle with a
different statement of the same quantity (the Eq. (1) direct sum against the
Remark 1 recursion, closed forms of special cases, textbook identities, library
routines, finite differences, exact rational arithmetic).  The mutation tests at
the bottom plant plausible mistakes in copies of the oracle and check that at
least one pin catches each.
"""

import math
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
from oracle import definitions as ov
from synth import make_random

PARAMS = [
    (1.0, 1.0, 1.0),
    (math.inf, math.inf, 1.0),
    (1.0, 0.5, 0.95),
    (2.0, 1.0, 0.7),
    (0.5, 1.5, 1.0),  # rho_bar < c_bar: outside the paper's assumption, still defined
    (1.0, 0.0, 1.0),
]


def _tiny(seed, T=None, B=None, A=None, end_prob=0.3, noise_std=0.8):
    rng = np.random.default_rng(seed)
    T = T or int(rng.integers(1, 9))
    B = B or int(rng.integers(1, 6))
    A = A or int(rng.integers(1, 6))
    tr = make_random(T, B, A, seed, noise_std=noise_std, end_prob=end_prob)
    # random per-step discounts in [0, 1] with exact zeros
    disc = rng.uniform(0.0, 1.0, size=(T, B)).astype(np.float32)
    disc[rng.random((T, B)) < end_prob] = 0.0
    tr.discounts = disc
    return tr


def _args(tr):
    return (tr.target_logits, tr.behaviour_logits, tr.actions, tr.rewards, tr.discounts,
            tr.values, tr.bootstrap_value)


# --------------------------------------------------------------------------------------
# v_s: Eq. (1) by brute force against the Remark 1 recursion
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(40))
@pytest.mark.parametrize("params", PARAMS)
def test_recursion_matches_direct_sum(seed, params):
    tr = _tiny(seed)
    rec = oracle.vtrace(*_args(tr), *params)
    direct = oracle.vtrace(*_args(tr), *params, direct_sum=True)
    np.testing.assert_allclose(rec.vs, direct.vs, rtol=1e-12, atol=1e-12)


def test_direct_sum_exact_rationals():
    """Eq. (1) in exact rational arithmetic, from given rho and c, against the
    oracle's recursion in fp64."""
    rng = np.random.default_rng(5)
    T, B = 6, 3
    fr = lambda x: Fraction(float(x))
    V = rng.integers(-4, 5, size=(T, B)) / 4.0
    boot = rng.integers(-4, 5, size=B) / 4.0
    r = rng.integers(-2, 3, size=(T, B)) / 2.0
    g = rng.choice([0.0, 0.5, 0.75, 1.0], size=(T, B))
    rho = rng.choice([0.25, 0.5, 1.0, 1.5], size=(T, B))
    c = rng.choice([0.0, 0.5, 1.0, 1.25], size=(T, B))
    deltas = ov.temporal_differences(rho, r, g, V, boot)
    got = ov.vtrace_targets_recursive(V, boot, deltas, g, c)
    for b in range(B):
        Vx = [fr(v) for v in V[:, b]] + [fr(boot[b])]
        for s in range(T):
            total = Vx[s]
            for t in range(s, T):
                disc = Fraction(1)
                trace = Fraction(1)
                for i in range(s, t):
                    disc *= fr(g[i, b])
                    trace *= fr(c[i, b])
                delta_t = fr(rho[t, b]) * (fr(r[t, b]) + fr(g[t, b]) * Vx[t + 1] - Vx[t])
                total += disc * trace * delta_t
            assert got[s, b] == float(total)


# --------------------------------------------------------------------------------------
# Special cases with closed forms
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("clip", [math.inf, 1.0, 3.0])
def test_on_policy_is_n_step_bellman_target(seed, clip):
    """Eq. (2): with pi = mu and c_bar >= 1, v_s is the n-step Bellman target."""
    tr = _tiny(seed, end_prob=0.2)
    tr.behaviour_logits = tr.target_logits.copy()
    out = oracle.vtrace(*_args(tr), clip, clip, 1.0)
    T, B = tr.rewards.shape
    r = tr.rewards.astype(np.float64)
    g = tr.discounts.astype(np.float64)
    boot = tr.bootstrap_value.astype(np.float64)
    for b in range(B):
        for s in range(T):
            acc, disc = 0.0, 1.0
            for t in range(s, T):
                acc += disc * r[t, b]
                disc *= g[t, b]
            expect = acc + disc * boot[b]
            assert out.vs[s, b] == pytest.approx(expect, rel=1e-12, abs=1e-12)


def test_on_policy_constant_gamma_literal_eq2():
    """Eq. (2) with the paper's constant gamma: sum gamma^(t-s) r_t + gamma^n V(x_{s+n})."""
    tr = make_random(7, 3, 4, 11, end_prob=0.0)
    tr.behaviour_logits = tr.target_logits.copy()
    gamma = 0.99
    tr.discounts[:] = np.float32(gamma)
    gam = float(np.float32(gamma))
    out = oracle.vtrace(*_args(tr), 1.0, 1.0, 1.0)
    T = tr.T
    for b in range(tr.B):
        for s in range(T):
            n = T - s
            expect = sum(gam ** (t - s) * float(tr.rewards[t, b]) for t in range(s, s + n))
            expect += gam ** n * float(tr.bootstrap_value[b])
            assert out.vs[s, b] == pytest.approx(expect, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("lam", [0.0, 0.3, 0.95, 1.0])
@pytest.mark.parametrize("seed", range(5))
def test_on_policy_lambda_is_td_lambda(lam, seed):
    """Remark 2: on-policy V-trace with lambda is the truncated lambda-return,
    G_s = r_s + gamma_s((1 - lambda) V(x_{s+1}) + lambda G_{s+1}), G_T = V(x_T)."""
    tr = _tiny(seed, T=8, end_prob=0.15)
    tr.behaviour_logits = tr.target_logits.copy()
    out = oracle.vtrace(*_args(tr), 1.0, 1.0, lam)
    T, B = tr.rewards.shape
    V = np.concatenate([tr.values, tr.bootstrap_value[None]]).astype(np.float64)
    G = V[T].copy()
    for s in range(T - 1, -1, -1):
        G = tr.rewards[s] + tr.discounts[s].astype(np.float64) * ((1 - lam) * V[s + 1] + lam * G)
        np.testing.assert_allclose(out.vs[s], G, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_cbar_zero_is_one_step_td(seed):
    tr = _tiny(seed)
    V = tr.values.astype(np.float64)
    Vn = np.concatenate([V[1:], tr.bootstrap_value[None].astype(np.float64)])
    for rho_bar, c_bar, lam in [(1.0, 0.0, 1.0), (2.0, 1.0, 0.0), (math.inf, 0.0, 0.5)]:
        out = oracle.vtrace(*_args(tr), rho_bar, c_bar, lam)
        pi = scipy.special.softmax(tr.target_logits.astype(np.float64), axis=-1)
        mu = scipy.special.softmax(tr.behaviour_logits.astype(np.float64), axis=-1)
        a = tr.actions[..., None].astype(np.int64)
        ratio = (np.take_along_axis(pi, a, -1) / np.take_along_axis(mu, a, -1))[..., 0]
        rho = np.minimum(rho_bar, ratio)
        expect = V + rho * (tr.rewards + tr.discounts * Vn - V)
        np.testing.assert_allclose(out.vs, expect, rtol=1e-11, atol=1e-12)
    # on-policy one-step TD target
    tr.behaviour_logits = tr.target_logits.copy()
    out = oracle.vtrace(*_args(tr), 1.0, 0.0, 1.0)
    np.testing.assert_allclose(out.vs, tr.rewards + tr.discounts * Vn, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_episode_cut_is_exact(seed):
    """gamma_t = 0 makes everything at s <= t independent of data after t (bit-exact)."""
    rng = np.random.default_rng(100 + seed)
    tr = make_random(9, 4, 5, 300 + seed, end_prob=0.0)
    tcut = int(rng.integers(0, 8))
    tr.discounts[tcut, :] = 0.0
    base = oracle.loss_and_grads(*_args(tr), math.inf, math.inf, 1.0)
    tr2 = make_random(9, 4, 5, 900 + seed, end_prob=0.1)
    for name in ("target_logits", "behaviour_logits", "actions", "rewards", "discounts", "values"):
        arr = getattr(tr, name).copy()
        arr[tcut + 1:] = getattr(tr2, name)[tcut + 1:]
        setattr(tr, name, arr)
    tr.bootstrap_value = tr2.bootstrap_value
    pert = oracle.loss_and_grads(*_args(tr), math.inf, math.inf, 1.0)
    assert np.array_equal(base.vs[:tcut + 1], pert.vs[:tcut + 1])
    assert np.array_equal(base.pg_advantages[:tcut + 1], pert.pg_advantages[:tcut + 1])
    assert np.array_equal(base.d_logits[:tcut + 1], pert.d_logits[:tcut + 1])
    assert np.array_equal(base.d_values[:tcut + 1], pert.d_values[:tcut + 1])


def test_pg_advantage_special_cases():
    tr = _tiny(3, T=7, B=4, A=5)
    # all discounts zero: rho_s (r_s - V(x_s))
    tr.discounts[:] = 0.0
    out = oracle.vtrace(*_args(tr), 1.0, 1.0, 1.0)
    np.testing.assert_allclose(out.pg_advantages, out.rho * (tr.rewards - tr.values.astype(np.float64)),
                               rtol=1e-13)
    # on-policy: rho = 1, advantage = r_s + gamma_s v_{s+1} - V(x_s), v_T = V(x_T)
    tr = _tiny(4, T=7, B=4, A=5)
    tr.behaviour_logits = tr.target_logits.copy()
    out = oracle.vtrace(*_args(tr), 1.0, 1.0, 1.0)
    assert np.all(out.rho == 1.0)
    vnext = np.concatenate([out.vs[1:], tr.bootstrap_value[None].astype(np.float64)])
    expect = tr.rewards + tr.discounts * vnext - tr.values
    np.testing.assert_allclose(out.pg_advantages, expect, rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------------------------------
# Importance weights and gathers against library routines
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_log_softmax_and_weights_against_scipy(seed):
    tr = make_random(6, 5, 7, 40 + seed, logit_scale=4.0)
    np.testing.assert_allclose(ov.log_softmax(tr.target_logits),
                               scipy.special.log_softmax(tr.target_logits.astype(np.float64), axis=-1),
                               rtol=1e-13, atol=1e-13)
    for rho_bar, c_bar, lam in PARAMS:
        lpa, lma, rho, c = ov.truncated_is_weights(tr.target_logits, tr.behaviour_logits,
                                                   tr.actions, rho_bar, c_bar, lam)
        pi = scipy.special.softmax(tr.target_logits.astype(np.float64), axis=-1)
        mu = scipy.special.softmax(tr.behaviour_logits.astype(np.float64), axis=-1)
        T, B = tr.actions.shape
        for t in range(T):
            for b in range(B):
                a = tr.actions[t, b]
                ratio = pi[t, b, a] / mu[t, b, a]
                assert rho[t, b] == pytest.approx(min(rho_bar, ratio), rel=1e-12)
                assert c[t, b] == pytest.approx(lam * min(c_bar, ratio), rel=1e-12, abs=1e-300)


def test_extreme_logits_stay_finite():
    tr = make_random(5, 4, 9, 77, logit_scale=80.0)
    out = oracle.loss_and_grads(*_args(tr), 1.0, 1.0, 1.0)
    for x in (out.vs, out.pg_advantages, out.d_logits, out.d_values, out.losses):
        assert np.all(np.isfinite(x))


def test_gather_is_bit_copy():
    tr = make_random(4, 3, 6, 12)
    got = ov.gather_action_logits(tr.target_logits, tr.behaviour_logits, tr.actions)
    for t in range(tr.T):
        for b in range(tr.B):
            a = tr.actions[t, b]
            assert got[t, b, 0].tobytes() == tr.target_logits[t, b, a].tobytes()
            assert got[t, b, 1].tobytes() == tr.behaviour_logits[t, b, a].tobytes()


def test_out_of_range_action_rejected():
    tr = make_random(3, 2, 4, 1)
    tr.actions[1, 1] = 4
    with pytest.raises(ValueError):
        oracle.vtrace(*_args(tr))


# --------------------------------------------------------------------------------------
# Losses and gradients
# --------------------------------------------------------------------------------------

def _frozen_total(tr, out, cv, ce, z=None, V=None):
    return ov.total_loss_frozen_targets(tr.target_logits if z is None else z,
                                        tr.values if V is None else V, tr.actions,
                                        out.pg_advantages, out.vs, cv, ce)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("params", PARAMS[:3])
def test_gradients_central_differences(seed, params):
    tr = make_random(4, 3, 5, 500 + seed, noise_std=1.0, end_prob=0.2)
    cv, ce = 0.5, 0.3
    out = oracle.loss_and_grads(*_args(tr), *params, cv, ce)
    z0 = tr.target_logits.astype(np.float64)
    V0 = tr.values.astype(np.float64)
    h = 1e-6
    fd = np.empty_like(z0)
    for idx in np.ndindex(*z0.shape):
        zp, zm = z0.copy(), z0.copy()
        zp[idx] += h
        zm[idx] -= h
        fd[idx] = (_frozen_total(tr, out, cv, ce, z=zp) - _frozen_total(tr, out, cv, ce, z=zm)) / (2 * h)
    np.testing.assert_allclose(out.d_logits, fd, rtol=1e-6, atol=1e-8)
    fdv = np.empty_like(V0)
    for idx in np.ndindex(*V0.shape):
        vp, vm = V0.copy(), V0.copy()
        vp[idx] += h
        vm[idx] -= h
        fdv[idx] = (_frozen_total(tr, out, cv, ce, V=vp) - _frozen_total(tr, out, cv, ce, V=vm)) / (2 * h)
    np.testing.assert_allclose(out.d_values, fdv, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("seed", range(4))
def test_gradients_match_paper_directions_via_autograd(seed):
    """The paper's update directions (Sec. 4.2), evaluated with torch autograd in
    fp64: -rho_s grad log pi(a_s) (r_s + gamma_s v_{s+1} - V(x_s)); the value
    direction -(v_s - V(x_s)); the entropy bonus direction."""
    torch = pytest.importorskip("torch")
    tr = make_random(5, 4, 6, 700 + seed, noise_std=1.0, end_prob=0.2)
    cv, ce = 0.5, 0.05
    out = oracle.loss_and_grads(*_args(tr), 1.0, 0.5, 0.9, cv, ce)
    z = torch.tensor(tr.target_logits, dtype=torch.float64, requires_grad=True)
    V = torch.tensor(tr.values, dtype=torch.float64, requires_grad=True)
    a = torch.tensor(tr.actions, dtype=torch.int64)
    adv = torch.tensor(out.pg_advantages)
    vs = torch.tensor(out.vs)
    logp = torch.log_softmax(z, dim=-1)
    p = torch.softmax(z, dim=-1)
    logp_a = logp.gather(-1, a[..., None])[..., 0]
    # descent on this objective moves along the paper's three directions
    objective = (-(adv * logp_a).sum() + cv * 0.5 * ((vs - V) ** 2).sum()
                 - ce * (-(p * logp).sum()))
    objective.backward()
    np.testing.assert_allclose(out.d_logits, z.grad.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(out.d_values, V.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_loss_values_against_library_routines():
    tr = make_random(6, 5, 9, 31, noise_std=1.0, end_prob=0.1)
    cv, ce = 0.5, 0.01
    out = oracle.loss_and_grads(*_args(tr), 1.0, 1.0, 1.0, cv, ce)
    pi = scipy.special.softmax(tr.target_logits.astype(np.float64), axis=-1)
    H = scipy.stats.entropy(pi, axis=-1)
    assert out.losses[3] == pytest.approx(-ce * H.sum(), rel=1e-12)
    logp_a = np.log(np.take_along_axis(pi, tr.actions[..., None].astype(np.int64), -1)[..., 0])
    assert out.losses[1] == pytest.approx(-(out.pg_advantages * logp_a).sum(), rel=1e-10)
    assert out.losses[2] == pytest.approx(cv * 0.5 * np.sum((out.vs - tr.values) ** 2), rel=1e-12)
    assert out.losses[0] == pytest.approx(out.losses[1:].sum(), rel=1e-13)
    np.testing.assert_allclose(out.lane_losses.sum(axis=0), out.losses[1:], rtol=1e-12)


def test_gradient_invariants():
    tr = make_random(6, 5, 9, 32, noise_std=1.0)
    out = oracle.loss_and_grads(*_args(tr), 1.0, 1.0, 1.0, 0.5, 0.0)
    np.testing.assert_allclose(out.d_logits.sum(axis=-1), 0.0, atol=1e-12)
    # with no entropy term the taken action's entry has the opposite sign of the advantage
    a = tr.actions[..., None].astype(np.int64)
    taken = np.take_along_axis(out.d_logits, a, -1)[..., 0]
    nz = out.pg_advantages != 0
    assert np.all(np.sign(taken[nz]) == -np.sign(out.pg_advantages[nz]))
    # a single action: the policy gradient vanishes identically
    tr1 = make_random(6, 5, 1, 33)
    out1 = oracle.loss_and_grads(*_args(tr1), 1.0, 1.0, 1.0, 0.5, 0.01)
    assert np.all(out1.d_logits == 0.0)


# --------------------------------------------------------------------------------------
# Mutation tests: a plausible mistake planted in a copy of the oracle must be caught
# --------------------------------------------------------------------------------------

def _pins_pass(mod):
    """Run a compact version of the pins against a (possibly mutated) oracle module."""
    ok = True
    for seed in range(6):
        tr = _tiny(seed, T=6, B=3, A=4)
        for params in [(1.0, 1.0, 1.0), (2.0, 0.5, 0.8), (math.inf, math.inf, 1.0)]:
            rec = mod.vtrace(*_args(tr), *params)
            direct = mod.vtrace(*_args(tr), *params, direct_sum=True)
            ok &= np.allclose(rec.vs, direct.vs, rtol=1e-10, atol=1e-12)
        # on-policy Bellman target
        tp = _tiny(seed, T=6, B=3, A=4)
        tp.behaviour_logits = tp.target_logits.copy()
        out = mod.vtrace(*_args(tp), 1.0, 1.0, 1.0)
        T, B = tp.rewards.shape
        exp_vs = np.empty((T, B))
        acc = tp.bootstrap_value.astype(np.float64)
        for s in range(T - 1, -1, -1):
            acc = tp.rewards[s] + tp.discounts[s].astype(np.float64) * acc
            exp_vs[s] = acc
        ok &= np.allclose(out.vs, exp_vs, rtol=1e-10, atol=1e-12)
        vnext = np.concatenate([exp_vs[1:], tp.bootstrap_value[None]])
        ok &= np.allclose(out.pg_advantages, tp.rewards + tp.discounts * vnext - tp.values,
                          rtol=1e-10, atol=1e-12)
        # one-step TD with lambda = 0, off-policy, against scipy probabilities
        lo = mod.vtrace(*_args(tr), 2.0, 1.0, 0.0)
        pi = scipy.special.softmax(tr.target_logits.astype(np.float64), axis=-1)
        mu = scipy.special.softmax(tr.behaviour_logits.astype(np.float64), axis=-1)
        a = tr.actions[..., None].astype(np.int64)
        rho = np.minimum(2.0, (np.take_along_axis(pi, a, -1) / np.take_along_axis(mu, a, -1))[..., 0])
        V = tr.values.astype(np.float64)
        Vn = np.concatenate([V[1:], tr.bootstrap_value[None]])
        ok &= np.allclose(lo.vs, V + rho * (tr.rewards + tr.discounts * Vn - V), rtol=1e-10)
        # all discounts zero: advantage rho_s (r_s - V(x_s)), off-policy
        tz = _tiny(seed, T=6, B=3, A=4)
        tz.discounts[:] = 0.0
        zo = mod.vtrace(*_args(tz), 2.0, 1.0, 1.0)
        piz = scipy.special.softmax(tz.target_logits.astype(np.float64), axis=-1)
        muz = scipy.special.softmax(tz.behaviour_logits.astype(np.float64), axis=-1)
        az = tz.actions[..., None].astype(np.int64)
        rhoz = np.minimum(2.0, (np.take_along_axis(piz, az, -1) / np.take_along_axis(muz, az, -1))[..., 0])
        ok &= np.allclose(zo.pg_advantages, rhoz * (tz.rewards.astype(np.float64) - tz.values), rtol=1e-10, atol=1e-13)
        # gradients against the paper's directions via finite differences
        lg = mod.loss_and_grads(*_args(tr), 1.0, 0.5, 0.9, 0.5, 0.3)
        zf = tr.target_logits.astype(np.float64)
        h = 1e-6
        idx = (0, 0, 0)
        zp, zm = zf.copy(), zf.copy()
        zp[idx] += h
        zm[idx] -= h
        f = lambda zz: oracle.total_loss_frozen_targets(zz, tr.values, tr.actions, lg.pg_advantages,
                                                        lg.vs, 0.5, 0.3)
        ok &= abs((f(zp) - f(zm)) / (2 * h) - lg.d_logits[idx]) < 1e-6
        ok &= np.allclose(lg.d_values, 0.5 * (V - lg.vs), rtol=1e-12)
        for i in range(zf.shape[-1]):
            idx = (1 % T, 0, i)
            zp, zm = zf.copy(), zf.copy()
            zp[idx] += h
            zm[idx] -= h
            ok &= abs((f(zp) - f(zm)) / (2 * h) - lg.d_logits[idx]) < 1e-6
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


MUTATIONS = {
    "trace_drops_c": [("_f64(discounts[s]) * c[s] * (vs", "_f64(discounts[s]) * (vs")],
    "trace_uses_rho": [("rho_value, c_value, rho_pg = rho, c, rho", "rho_value, c_value, rho_pg = rho, rho, rho")],
    "delta_uses_V_t": [("_f64(discounts) * _values_next(values, bootstrap_value)", "_f64(discounts) * _f64(values)")],
    "delta_sign": [("\n                        - _f64(values))", "\n                        + _f64(values))")],
    "lambda_scales_rho": [("rho = np.minimum(np.float64(rho_bar), ratio)",
                           "rho = np.float64(lam) * np.minimum(np.float64(rho_bar), ratio)")],
    "min_swapped_bars": [("rho = np.minimum(np.float64(rho_bar), ratio)", "rho = np.minimum(np.float64(c_bar), ratio)")],
    "ratio_inverted": [("ratio = np.exp(log_pi_a - log_mu_a)", "ratio = np.exp(log_mu_a - log_pi_a)")],
    "pg_uses_v_s": [("nxt = np.concatenate([_f64(vs)[1:], _f64(bootstrap_value)[None]], axis=0)",
                     "nxt = _f64(vs)")],
    "pg_drops_rho": [("return _f64(rho) * (q - _f64(values))", "return (q - _f64(values))")],
    "pg_drops_discount": [("q = _f64(rewards) + _f64(discounts) * nxt", "q = _f64(rewards) + nxt")],
    "recursion_wrong_V": [("(vs[s + 1] - V_ext[s + 1])", "(vs[s + 1] - V_ext[s])")],
    "grad_entropy_sign": [("+ c_e * pi * (log_pi + entropy[..., None]))", "- c_e * pi * (log_pi + entropy[..., None]))")],
    "grad_onehot_shift": [("np.asarray(actions, dtype=np.int64)[..., None], 1.0, axis=-1)",
                           "(np.asarray(actions, dtype=np.int64)[..., None] + 1) % pi.shape[-1], 1.0, axis=-1)")],
    "grad_values_sign": [("d_values = c_v * (_f64(values) - vt.vs)", "d_values = c_v * (vt.vs - _f64(values))")],
    "log_softmax_no_max": [("return x - (m + np.log(np.exp(x - m).sum(axis=-1, keepdims=True)))",
                            "return x - np.log(np.exp(x - m).sum(axis=-1, keepdims=True))")],
    "direct_sum_off_by_one": [("discount_prod = np.prod(g[s:t], axis=0)", "discount_prod = np.prod(g[s:t + 1], axis=0)")],
}


def test_unmutated_oracle_passes_compact_pins():
    assert _pins_pass(ov)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name):
    assert not _pins_pass(_mutant(MUTATIONS[name]))
