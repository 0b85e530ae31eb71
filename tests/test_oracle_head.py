"""Pins of the output-layer oracle (oracle/head.py) against facts that do not
come from its own code: finite differences of the loss, an autograd
derivation written separately, the identity layer, invariances of the softmax,
and planted mistakes that these checks must catch."""

import inspect
import math
import types

import numpy as np
import pytest

import oracle
from oracle import definitions as od
from oracle import head as oh
from synth import make_head

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def tiny(seed, T=5, B=3, A=4, H=6, **kw):
    hb = make_head(T, B, A, H, seed, **kw)
    return (hb.hidden.astype(np.float64), hb.weight.astype(np.float64), hb.bias.astype(np.float64),
            hb.behaviour_logits, hb.actions, hb.rewards, hb.discounts, hb.bootstrap_value)


def frozen_loss(mod, h, W, b, y, a, r, d, boot, p, correction="vtrace", **kw):
    """The total loss as a function of the layer's input and parameters, with
    every target (rho, c, v_s, advantages) held at the unperturbed point."""
    ref = mod.head_loss_and_grads(h, W, b, y, a, r, d, boot, *p, correction=correction, **kw)

    def L(h2, W2, b2):
        o = h2 @ W2 + b2
        A = W2.shape[1] - 1
        return od.total_loss_frozen_targets(o[..., :A], o[..., A], a, ref.pg_advantages, ref.vs,
                                            p[3], p[4], correction=correction,
                                            epsilon=kw.get("epsilon", 1e-6))
    return ref, L


PARAMS = [(1.0, 1.0, 1.0, 0.5, 0.01), (math.inf, math.inf, 1.0, 0.5, 0.01),
          (2.0, 0.5, 0.9, 0.7, 0.03)]


@pytest.mark.parametrize("p", PARAMS)
@pytest.mark.parametrize("correction", ["vtrace", "epsilon", "one_step_is"])
def test_gradients_match_finite_differences(p, correction):
    h, W, b, y, a, r, d, boot = tiny(11)
    ref, L = frozen_loss(oh, h, W, b, y, a, r, d, boot, p, correction)
    assert np.isclose(L(h, W, b), ref.losses[0], rtol=1e-12, atol=1e-12)
    eps = 1e-6

    def fd(arr, idx, which):
        hp, Wp, bp = h.copy(), W.copy(), b.copy()
        hm, Wm, bm = h.copy(), W.copy(), b.copy()
        {"h": hp, "W": Wp, "b": bp}[which][idx] += eps
        {"h": hm, "W": Wm, "b": bm}[which][idx] -= eps
        return (L(hp, Wp, bp) - L(hm, Wm, bm)) / (2 * eps)

    rng = np.random.default_rng(3)
    for _ in range(12):
        idx = tuple(rng.integers(0, n) for n in h.shape)
        assert np.isclose(fd(h, idx, "h"), ref.d_hidden[idx], rtol=1e-6, atol=1e-8), idx
    for i in range(W.shape[0]):
        for j in range(W.shape[1]):
            assert np.isclose(fd(W, (i, j), "W"), ref.d_weight[i, j], rtol=1e-6, atol=1e-8)
    for j in range(b.shape[0]):
        assert np.isclose(fd(b, (j,), "b"), ref.d_bias[j], rtol=1e-6, atol=1e-8)


def test_gradients_match_autograd():
    torch = pytest.importorskip("torch")
    h, W, b, y, a, r, d, boot = tiny(12, T=7, B=4, A=5, H=8)
    p = (1.0, 1.0, 0.95, 0.5, 0.01)
    ref = oh.head_loss_and_grads(h, W, b, y, a, r, d, boot, *p)
    th = torch.tensor(h, requires_grad=True)
    tW = torch.tensor(W, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    o = th @ tW + tb
    A = W.shape[1] - 1
    logp = torch.log_softmax(o[..., :A], dim=-1)
    lpa = torch.gather(logp, -1, torch.tensor(a, dtype=torch.int64)[..., None])[..., 0]
    adv = torch.tensor(ref.pg_advantages)
    vs = torch.tensor(ref.vs)
    loss = (-(adv * lpa).sum() + p[3] * 0.5 * ((vs - o[..., A]) ** 2).sum()
            + p[4] * (logp.exp() * logp).sum())
    loss.backward()
    assert np.isclose(loss.item(), ref.losses[0], rtol=1e-12)
    np.testing.assert_allclose(th.grad.numpy(), ref.d_hidden, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(tW.grad.numpy(), ref.d_weight, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(tb.grad.numpy(), ref.d_bias, rtol=1e-10, atol=1e-12)


def test_identity_layer_reduces_to_the_plain_loss():
    """H = A + 1, weight = I, bias = 0: the layer passes hidden through, so the
    outputs are the plain loss's, d_hidden is G itself, d_weight = h^T G."""
    T, B, A = 6, 3, 4
    rng = np.random.default_rng(5)
    h = rng.standard_normal((T, B, A + 1))
    y = rng.standard_normal((T, B, A))
    a = rng.integers(0, A, (T, B)).astype(np.int32)
    r = rng.uniform(-1, 1, (T, B))
    d = np.where(rng.random((T, B)) < 0.2, 0.0, 0.99)
    boot = rng.standard_normal(B)
    out = oh.head_loss_and_grads(h, np.eye(A + 1), np.zeros(A + 1), y, a, r, d, boot, 1.0, 1.0, 1.0)
    lg = od.loss_and_grads(h[..., :A], y, a, r, d, h[..., A], boot, 1.0, 1.0, 1.0)
    np.testing.assert_array_equal(out.losses, lg.losses)
    np.testing.assert_array_equal(out.d_hidden[..., :A], lg.d_logits)
    np.testing.assert_array_equal(out.d_hidden[..., A], lg.d_values)
    # d_weight[i, j] = sum over (t, b) of h_i G_j, written as an explicit loop
    G = out.d_hidden
    for i in range(A + 1):
        for j in range(A + 1):
            s = 0.0
            for t in range(T):
                for bb in range(B):
                    s += h[t, bb, i] * G[t, bb, j]
            assert np.isclose(out.d_weight[i, j], s, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out.d_bias, G.sum(axis=(0, 1)), rtol=1e-12, atol=1e-14)


def test_softmax_invariances():
    """The policy gradient of every step sums to zero over actions, so the
    policy columns of d_bias and of every row of d_weight sum to zero; shifting
    all policy biases by one constant changes nothing."""
    h, W, b, y, a, r, d, boot = tiny(13, T=9, B=5, A=6, H=7)
    p = (1.0, 1.0, 1.0, 0.5, 0.01)
    out = oh.head_loss_and_grads(h, W, b, y, a, r, d, boot, *p)
    A = W.shape[1] - 1
    assert abs(out.d_bias[:A].sum()) < 1e-12 * np.abs(out.d_bias).sum() + 1e-14
    np.testing.assert_allclose(out.d_weight[:, :A].sum(axis=1), 0.0, atol=1e-12)
    b2 = b.copy()
    b2[:A] += 3.25
    out2 = oh.head_loss_and_grads(h, W, b2, y, a, r, d, boot, *p)
    np.testing.assert_allclose(out2.losses, out.losses, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(out2.d_hidden, out.d_hidden, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(out2.d_weight, out.d_weight, rtol=1e-9, atol=1e-12)


def test_value_column_only_moves_the_baseline():
    """With zero policy weights and biases the policy is uniform whatever the
    input, so d_hidden lies along the value column: c_v (V - v) w_v."""
    h, W, b, y, a, r, d, boot = tiny(14, T=6, B=3, A=4, H=5)
    A = W.shape[1] - 1
    W[:, :A] = 0.0
    b[:A] = 0.0
    out = oh.head_loss_and_grads(h, W, b, y, a, r, d, boot, 1.0, 1.0, 1.0, 0.5, 0.01)
    V = h @ W[:, A] + b[A]
    expect = (0.5 * (V - out.vs))[..., None] * W[:, A]
    # the uniform policy still has a policy gradient on its logits, but the
    # zero policy weights map it to nothing
    np.testing.assert_allclose(out.d_hidden, expect, rtol=1e-12, atol=1e-14)


def test_term_scale():
    h = np.arange(6.0).reshape(1, 2, 3)
    G = np.array([[[1.0, -2.0], [3.0, 0.5]]])
    sw, sb = oh.sum_term_scale(h, G)
    assert np.isclose(sw[1, 0], math.sqrt((1 * 1) ** 2 + (4 * 3) ** 2))
    assert np.isclose(sb[1], math.sqrt(4 + 0.25))


# --- planted mistakes ---------------------------------------------------------

def _mutant(replacements):
    src = inspect.getsource(oh).replace("from .definitions import", "from oracle.definitions import")
    for old, new in replacements:
        assert old in src, old
        src = src.replace(old, new, 1)
    mod = types.ModuleType("head_mutant")
    exec(compile(src, "head_mutant", "exec"), mod.__dict__)
    return mod


MUTATIONS = {
    "d_hidden_drops_value_column": [("d_hidden = G @ weight.T", "d_hidden = G[..., :A] @ weight[:, :A].T")],
    "d_hidden_reversed_columns": [("d_hidden = G @ weight.T", "d_hidden = G @ weight[:, ::-1].T")],
    "bias_not_added": [("return _f64(hidden) @ _f64(weight) + _f64(bias)", "return _f64(hidden) @ _f64(weight)")],
    "value_from_first_column": [("z, V = o[..., :A], o[..., A]", "z, V = o[..., 1:], o[..., 0]")],
    "d_bias_mean": [("d_bias = G.reshape(-1, A + 1).sum(axis=0)", "d_bias = G.reshape(-1, A + 1).mean(axis=0)")],
    "d_weight_time_shift": [("d_weight = hidden.reshape(-1, H).T @ G.reshape(-1, A + 1)",
                             "d_weight = np.roll(hidden, 1, axis=0).reshape(-1, H).T @ G.reshape(-1, A + 1)")],
    "d_outputs_sign": [("G = np.concatenate([lg.d_logits, lg.d_values[..., None]], axis=-1)",
                        "G = np.concatenate([lg.d_logits, -lg.d_values[..., None]], axis=-1)")],
}


def _pins_pass(mod):
    h, W, b, y, a, r, d, boot = tiny(21, T=6, B=3, A=4, H=5)
    p = (1.0, 1.0, 1.0, 0.5, 0.01)
    try:
        ref, L = frozen_loss(mod, h, W, b, y, a, r, d, boot, p)
        eps = 1e-6
        for i in range(W.shape[0]):
            for j in range(W.shape[1]):
                Wp, Wm = W.copy(), W.copy()
                Wp[i, j] += eps
                Wm[i, j] -= eps
                if not np.isclose((L(h, Wp, b) - L(h, Wm, b)) / (2 * eps), ref.d_weight[i, j],
                                  rtol=1e-6, atol=1e-8):
                    return False
        for j in range(b.shape[0]):
            bp, bm = b.copy(), b.copy()
            bp[j] += eps
            bm[j] -= eps
            if not np.isclose((L(h, W, bp) - L(h, W, bm)) / (2 * eps), ref.d_bias[j],
                              rtol=1e-6, atol=1e-8):
                return False
        for idx in [(0, 0, 0), (2, 1, 3), (5, 2, 4), (3, 0, 1)]:
            hp, hm = h.copy(), h.copy()
            hp[idx] += eps
            hm[idx] -= eps
            if not np.isclose((L(hp, W, b) - L(hm, W, b)) / (2 * eps), ref.d_hidden[idx],
                              rtol=1e-6, atol=1e-8):
                return False
        # the loss itself against a separately written forward pass
        o = h @ W + b
        A = W.shape[1] - 1
        lg = od.loss_and_grads(o[..., :A], y, a, r, d, o[..., A], boot, *p)
        return bool(np.allclose(ref.losses, lg.losses, rtol=1e-12, atol=1e-12))
    except (AssertionError, ValueError, IndexError):
        return False


def test_unmutated_head_oracle_passes():
    assert _pins_pass(oh)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name):
    assert not _pins_pass(_mutant(MUTATIONS[name]))
