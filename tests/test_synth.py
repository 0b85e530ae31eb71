"""The seeded generators: determinism, shapes, chunk independence, bf16 rounding."""

import numpy as np

from synth import bf16_bits_to_f32, f32_to_bf16_bits, make_config, make_random, subset_lanes
import synth.trajectories as st


def test_configs_shapes_and_determinism():
    for cfg in (0, 1, 2):
        a, b = make_config(cfg), make_config(cfg)
        c = st.WORKLOADS[cfg]
        assert a.target_logits.shape == (c["T"], c["B"], c["A"])
        assert a.actions.dtype == np.int32 and a.actions.min() >= 0 and a.actions.max() < c["A"]
        for name in ("target_logits", "behaviour_logits", "actions", "rewards", "discounts",
                     "values", "bootstrap_value"):
            assert np.array_equal(getattr(a, name), getattr(b, name))
            assert getattr(a, name).flags.c_contiguous
        assert set(np.unique(a.discounts)) <= {np.float32(0.0), np.float32(0.99)}
        assert a.rewards.min() >= -1 and a.rewards.max() <= 1


def test_chunked_generation_matches_unchunked(monkeypatch):
    ref = make_random(13, 8, 5, 99)
    monkeypatch.setattr(st, "_CHUNK_ELEMS", 40)  # forces 1-step chunks
    chunked = make_random(13, 8, 5, 99)
    for name in ("target_logits", "behaviour_logits", "actions"):
        assert np.array_equal(getattr(ref, name), getattr(chunked, name))


def test_bf16_rounding_is_nearest_even_and_exact_on_widening():
    x = np.array([1.0, 1.00390625, 1.005859375, -2.5e-3, 3.0e38], dtype=np.float32)
    bits = f32_to_bf16_bits(x)
    back = bf16_bits_to_f32(bits)
    assert np.array_equal(f32_to_bf16_bits(back), bits)
    assert back[0] == 1.0 and back[1] == 1.0  # tie rounds to even
    assert np.all(np.abs(back - x) <= np.abs(x) * 2.0 ** -8)
    tr = make_config(0, bf16=True)
    assert tr.dtype == "bf16"
    assert np.array_equal(bf16_bits_to_f32(tr.target_bits), tr.target_logits)


def test_multitask_groups_and_actions_follow_behaviour():
    tr = make_config(3)
    assert tr.B == 4096 and tr.A == 9
    # actions are samples of softmax(behaviour): the arg-max action is the most frequent
    top = np.argmax(tr.behaviour_logits, axis=-1)
    assert np.mean(top == tr.actions) > 0.3


def test_subset_lanes():
    tr = make_config(2)
    sub = subset_lanes(tr, [0, 5, 31])
    assert sub.B == 3
    assert np.array_equal(sub.target_logits[:, 1], tr.target_logits[:, 5])
    assert np.array_equal(sub.bootstrap_value, tr.bootstrap_value[[0, 5, 31]])


def test_head_batches_are_seeded_and_shaped():
    from synth import HEAD_WORKLOADS, make_head, make_head_config, subset_head_lanes
    a = make_head(9, 5, 7, 64, 42)
    b = make_head(9, 5, 7, 64, 42)
    for f in ("hidden_bits", "weight_bits", "bias", "behaviour_logits", "actions", "rewards",
              "discounts", "bootstrap_value"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    assert a.hidden_bits.shape == (9, 5, 64) and a.hidden_bits.dtype == np.uint16
    assert a.weight_bits.shape == (64, 8) and a.bias.shape == (8,)
    assert np.all(np.abs(a.hidden) <= 1.0)
    assert a.actions.min() >= 0 and a.actions.max() < 7
    assert set(np.unique(a.discounts)) <= {0.0, np.float32(0.99)}
    c = make_head_config("atari")
    assert (c.T, c.B, c.A, c.H) == (HEAD_WORKLOADS["atari"]["T"], 32, 18, 256)
    s = subset_head_lanes(c, [3, 0])
    np.testing.assert_array_equal(s.hidden_bits[:, 1], c.hidden_bits[:, 0])
    np.testing.assert_array_equal(s.bootstrap_value, c.bootstrap_value[[3, 0]])
