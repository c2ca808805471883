"""Oracle elementary operations against closed forms and textbook properties."""
import math

import numpy as np
import pytest

import synth
from oracle import model as om


def test_rms_norm_closed_forms():
    eps = 0.0
    g = np.ones(4)
    # mean square 1 -> unchanged
    np.testing.assert_allclose(om.rms_norm(np.array([1.0, -1.0, 1.0, -1.0]), g, eps), [1, -1, 1, -1])
    # [2,0,0,0]: mean square 1 -> unchanged
    np.testing.assert_allclose(om.rms_norm(np.array([2.0, 0, 0, 0]), g, eps), [2, 0, 0, 0])
    # [3,4]: rms = sqrt(12.5)
    np.testing.assert_allclose(om.rms_norm(np.array([3.0, 4.0]), np.array([1.0, 2.0]), eps),
                               [3 / math.sqrt(12.5), 8 / math.sqrt(12.5)])
    # eps sits inside the square root
    np.testing.assert_allclose(om.rms_norm(np.array([0.0, 0.0]), np.ones(2), 1e-6), [0, 0])
    x = np.array([1e-3, 0.0])
    np.testing.assert_allclose(om.rms_norm(x, np.ones(2), 1e-6), x / math.sqrt(0.5e-6 + 1e-6))


def test_rms_norm_scale_invariance_and_unit_rms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64))
    y = om.rms_norm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-12)
    np.testing.assert_allclose(om.rms_norm(7.5 * x, np.ones(64), 0.0), y, rtol=1e-12)


def test_rope_position_zero_is_identity():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((3, 2, 16))
    np.testing.assert_array_equal(om.rope(v, np.zeros(3, dtype=int), 1e6), v)


def test_rope_d2_is_plane_rotation():
    # d = 2: one pair with frequency theta^0 = 1, so position p rotates by p radians.
    v = np.array([[[1.0, 0.0]], [[0.3, -0.7]]])
    pos = np.array([1, 5])
    out = om.rope(v, pos, 1e6)
    np.testing.assert_allclose(out[0, 0], [math.cos(1), math.sin(1)], rtol=1e-14)
    c, s = math.cos(5), math.sin(5)
    np.testing.assert_allclose(out[1, 0], [0.3 * c + 0.7 * s, -0.7 * c + 0.3 * s], rtol=1e-14)


def test_rope_rotate_half_pairing_and_frequency():
    # d = 4, theta = 100: pair 0 = (x0, x2) at frequency 1, pair 1 = (x1, x3) at 100^(-1/2).
    v = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    out = om.rope(v, np.array([3]), 100.0)
    a = 3 * 0.1
    np.testing.assert_allclose(out[0, 0], [0.0, math.cos(a), 0.0, math.sin(a)], atol=1e-15)


def test_rope_norm_preserving_and_relative():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    for p in (0, 7, 1000):
        np.testing.assert_allclose(np.linalg.norm(om.rope(q, np.array([p]), 1e6)), np.linalg.norm(q))
    dots = []
    for m, n in ((10, 3), (107, 100), (7, 0)):
        dots.append(float(np.sum(om.rope(q, np.array([m]), 1e6) * om.rope(k, np.array([n]), 1e6))))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)


def test_softmax_closed_form():
    np.testing.assert_allclose(om.softmax_rows(np.array([[0.0, math.log(3.0)]])), [[0.25, 0.75]])
    s = np.random.default_rng(3).standard_normal((4, 9))
    p = om.softmax_rows(s)
    np.testing.assert_allclose(p.sum(-1), 1.0)
    np.testing.assert_allclose(om.softmax_rows(s + 100.0), p)
    # masked (-inf) entries get exactly zero weight
    s2 = s.copy(); s2[:, 3] = -np.inf
    assert np.all(om.softmax_rows(s2)[:, 3] == 0.0)


def test_silu_closed_form():
    np.testing.assert_allclose(om.silu(np.array([0.0, 1.0, -2.0])),
                               [0.0, 1 / (1 + math.exp(-1)), -2 / (1 + math.exp(2))])


def test_lora_linear_equals_merged_weight(tiny_weights):
    m = om.OracleModel(tiny_weights)
    lw = m.layers[0]
    x = np.random.default_rng(4).standard_normal((3, m.cfg.hidden))
    A, B = lw["lora"]["q"]
    merged = lw["q"] + m.cfg.lora_scale * (B @ A)
    np.testing.assert_allclose(m.linear(lw, "q", x, True), x @ merged.T, rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(m.linear(lw, "q", x, False), x @ lw["q"].T)


def test_argmax_lowest_index_tie_break_and_exclusion():
    assert om.greedy_argmax(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert om.greedy_argmax(np.array([1.0, 3.0, 3.0, 2.0]), exclude=1) == 2
    assert om.greedy_argmax(np.array([5.0, 1.0]), exclude=0) == 1


def test_lora_parameter_count_matches_paper():
    # App. A.2: 10.1M trainable parameters, 1.666% of 605.9M, with LoRA r=16 on all
    # seven linear projections of the 28 Qwen3-0.6B blocks.
    cfg = synth.QWEN3_0_6B
    n = cfg.n_layers * sum(cfg.lora_rank * (o + i) for _, o, i in cfg.linear_shapes())
    assert n == 10_092_544
    assert round(n / 1e6, 1) == 10.1
    assert round(100 * n / 605.9e6, 3) == 1.666


def test_qwen_shape_weight_bytes():
    # Tied bf16 backbone of the Qwen3-0.6B shape: 596,049,920 parameters.
    cfg = synth.QWEN3_0_6B
    per_layer = sum(o * i for _, o, i in cfg.linear_shapes()) + 2 * cfg.hidden + 2 * cfg.head_dim
    total = cfg.vocab * cfg.hidden + cfg.n_layers * per_layer + cfg.hidden
    assert total == 596_049_920


def test_bf16_rounding_is_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5], dtype=np.float32)
    # bf16 has 7 mantissa bits: spacing 2^-7 near 1.
    np.testing.assert_array_equal(synth.round_bf16(x),
                                  np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5], dtype=np.float32))
