"""Pins of the short-convolution oracle (Section 4.1, Fig. 2: the convolution state
continues over the replacement tokens). Each test fixes the oracle against
something other than itself: a library convolution, closed forms, special cases
and the continuation invariant."""
import numpy as np
import pytest

import oracle
from oracle.bf16 import bf16_to_f64, f64_to_bf16


def _bits(rng, shape, scale=1.0):
    return f64_to_bf16(rng.normal(0.0, scale, size=shape))


@pytest.mark.parametrize("W,C,T", [(4, 24, 37), (2, 8, 5), (3, 16, 1), (4, 8, 2), (5, 40, 64)])
def test_matches_library_convolution(W, C, T):
    rng = np.random.default_rng(W * 100 + T)
    st, x, w = _bits(rng, (W - 1, C)), _bits(rng, (T, C)), _bits(rng, (C, W), 0.5)
    _, y, _ = oracle.short_conv_continue(st, x, w, activation="none")
    xt = bf16_to_f64(np.concatenate([st, x]))
    wf = bf16_to_f64(w)
    for c in range(C):
        ref = np.convolve(xt[:, c], wf[c][::-1], mode="valid")   # valid: T outputs
        np.testing.assert_allclose(y[:, c], ref, rtol=1e-14, atol=1e-14)


def test_continuation_equals_one_pass():
    rng = np.random.default_rng(7)
    W, C = 4, 32
    st, w = _bits(rng, (W - 1, C)), _bits(rng, (C, W), 0.5)
    x = _bits(rng, (50, C))
    y_all, _, s_all = oracle.short_conv_continue(st, x, w)
    for cut in (0, 1, 2, 3, 17, 49, 50):
        y1, _, s1 = oracle.short_conv_continue(st, x[:cut], w)
        y2, _, s2 = oracle.short_conv_continue(s1, x[cut:], w)
        assert np.array_equal(np.concatenate([y1, y2]), y_all)
        assert np.array_equal(s2, s_all)


def test_identity_and_delay_taps():
    rng = np.random.default_rng(3)
    W, C, T = 4, 16, 9
    st, x = _bits(rng, (W - 1, C)), _bits(rng, (T, C))
    one = np.zeros((C, W))
    one[:, W - 1] = 1.0
    y, _, _ = oracle.short_conv_continue(st, x, f64_to_bf16(one), activation="none")
    assert np.array_equal(y, x)                                     # newest tap only: y = x
    ys, _, _ = oracle.short_conv_continue(st, x, f64_to_bf16(one), activation="silu")
    xv = bf16_to_f64(x)
    assert np.array_equal(ys, f64_to_bf16(xv / (1.0 + np.exp(-xv))))
    first = np.zeros((C, W))
    first[:, 0] = 1.0
    yd, _, _ = oracle.short_conv_continue(st, x, f64_to_bf16(first), activation="none")
    assert np.array_equal(yd, np.concatenate([st, x])[:T])          # oldest tap only: delayed by W-1


def test_width_one_is_pointwise():
    rng = np.random.default_rng(4)
    C, T = 8, 11
    x, w = _bits(rng, (T, C)), _bits(rng, (C, 1), 0.7)
    y, _, s = oracle.short_conv_continue(np.zeros((0, C), np.uint16), x, w, activation="none")
    assert s.shape == (0, C)
    assert np.array_equal(y, f64_to_bf16(bf16_to_f64(x) * bf16_to_f64(w)[:, 0][None, :]))


def test_state_update_short_and_empty_tails():
    rng = np.random.default_rng(5)
    W, C = 4, 8
    st, w = _bits(rng, (W - 1, C)), _bits(rng, (C, W))
    y0, _, s0 = oracle.short_conv_continue(st, np.zeros((0, C), np.uint16), w)
    assert y0.shape == (0, C) and np.array_equal(s0, st)
    x = _bits(rng, (2, C))
    _, _, s2 = oracle.short_conv_continue(st, x, w)
    assert np.array_equal(s2, np.concatenate([st[2:], x]))
    x5 = _bits(rng, (5, C))
    _, _, s5 = oracle.short_conv_continue(st, x5, w)
    assert np.array_equal(s5, x5[2:])


def test_silu_closed_forms():
    x = np.array([-40.0, -3.0, -0.5, 0.0, 0.25, 2.0, 40.0])
    s = oracle.silu(x)
    assert s[3] == 0.0
    np.testing.assert_allclose(s - oracle.silu(-x), x, rtol=0, atol=1e-13)   # silu(x) - silu(-x) = x
    np.testing.assert_allclose(s[2:6], x[2:6] / (1.0 + np.exp(-x[2:6])), rtol=1e-15)
    assert abs(s[-1] - 40.0) < 1e-15 and abs(s[0]) < 2e-16


def test_scaling_by_two_is_exact():
    rng = np.random.default_rng(6)
    W, C, T = 4, 16, 12
    st, x, w = _bits(rng, (W - 1, C)), _bits(rng, (T, C)), _bits(rng, (C, W))
    _, y, _ = oracle.short_conv_continue(st, x, w, activation="none")
    st2 = f64_to_bf16(2.0 * bf16_to_f64(st))
    x2 = f64_to_bf16(2.0 * bf16_to_f64(x))
    _, y2, _ = oracle.short_conv_continue(st2, x2, w, activation="none")
    assert np.array_equal(y2, 2.0 * y)
