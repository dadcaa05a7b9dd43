"""Pins for the oracle's bf16 rounding and rotary embedding (CPU only).

Each test checks the oracle against something it does not contain: torch's own
float32->bf16 conversion, exact powers of two, math.cos/math.sin closed forms,
rotation invariants and the relative-position property of rotary embeddings.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- bf16

def test_bf16_roundtrip_exact_values():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = oracle.bf16_to_f64(bits)
    finite = np.isfinite(vals)
    back = oracle.f64_to_bf16(vals[finite])
    # -0.0 encodes as 0x8000 and +0.0 as 0x0000; every finite bf16 value round-trips
    assert np.array_equal(back, bits[finite])


def test_bf16_matches_torch_on_float32_inputs():
    # torch rounds float32 -> bf16 once with round-to-nearest-even: a library
    # routine that agrees with direct rounding whenever the input is a float32.
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.normal(0, 1, 200000), rng.normal(0, 1e-38, 2000),
                        rng.normal(0, 1e30, 2000)]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.f64_to_bf16(x.astype(np.float64)), ref)


def test_bf16_ties_to_even_and_no_double_rounding():
    one = 1.0
    ulp = 2.0 ** -7                  # bf16 spacing in [1, 2)
    # exact ties go to the even neighbour
    assert oracle.f64_to_bf16(np.array([one + ulp / 2]))[0] == 0x3F80
    assert oracle.f64_to_bf16(np.array([one + 3 * ulp / 2]))[0] == 0x3F82
    # just above a tie rounds up even though a float32 intermediate would not
    assert oracle.f64_to_bf16(np.array([one + ulp / 2 + 1e-9]))[0] == 0x3F81
    assert oracle.f64_to_bf16(np.array([-(one + ulp / 2 + 1e-9)]))[0] == 0xBF81
    # subnormal quantum is 2**-133
    assert oracle.f64_to_bf16(np.array([2.0 ** -133]))[0] == 0x0001
    assert oracle.f64_to_bf16(np.array([2.0 ** -134]))[0] == 0x0000    # tie to even (0)
    assert oracle.f64_to_bf16(np.array([3 * 2.0 ** -134]))[0] == 0x0002


# ----------------------------------------------------------------------------- rope

def test_rope_closed_form_small_example():
    # D = r = 4, theta = 100: omega = (1, 0.1). Pairs are (0, 2) and (1, 3).
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    y = oracle.rope_rotate(x, np.array([3]), 4, 100.0)[0, 0]
    a0, a1 = 3.0, 0.3
    want = [1 * math.cos(a0) - 3 * math.sin(a0),
            2 * math.cos(a1) - 4 * math.sin(a1),
            3 * math.cos(a0) + 1 * math.sin(a0),
            4 * math.cos(a1) + 2 * math.sin(a1)]
    np.testing.assert_allclose(y, want, rtol=0, atol=1e-14)


def test_rope_frequencies_closed_form():
    w = oracle.rope_frequencies(8, 1.0e4)
    np.testing.assert_allclose(w, [1.0, 0.1, 0.01, 0.001], rtol=1e-15)


def test_rope_identity_cases():
    rng = np.random.default_rng(2)
    x = rng.normal(size=(5, 3, 16))
    # position 0 is the identity; rotary_dim 0 is the identity at any position
    np.testing.assert_array_equal(oracle.rope_rotate(x, np.zeros(5, dtype=np.int64), 16, 1e7), x)
    np.testing.assert_array_equal(oracle.rope_rotate(x, np.arange(5) * 1000, 0, 1e7), x)
    # partial rotary: dims >= r pass through untouched
    y = oracle.rope_rotate(x, np.arange(5) * 7, 8, 1e4)
    np.testing.assert_array_equal(y[:, :, 8:], x[:, :, 8:])


def test_rope_preserves_pair_norms():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(7, 2, 64))
    pos = rng.integers(0, 500000, size=7)
    y = oracle.rope_rotate(x, pos, 64, 1e7)
    nx = x[:, :, :32] ** 2 + x[:, :, 32:] ** 2
    ny = y[:, :, :32] ** 2 + y[:, :, 32:] ** 2
    np.testing.assert_allclose(ny, nx, rtol=1e-12)


def test_rope_relative_position_at_paper_cursor():
    # Section 6.3 reports a true-tail cursor of 479,547 (stored in golden/).
    with open(os.path.join(GOLDEN, "paper_placement_case.json")) as f:
        case = json.load(f)
    cursor = case["next_position_true_tail"]
    rng = np.random.default_rng(4)
    for theta in (1.0e4, 1.0e7):
        q = rng.normal(size=(1, 1, 256))
        k = rng.normal(size=(1, 1, 256))
        pq, pk = 700, 123
        base = np.sum(oracle.rope_rotate(q, np.array([pq]), 256, theta) *
                      oracle.rope_rotate(k, np.array([pk]), 256, theta))
        d = cursor - pq
        shifted = np.sum(oracle.rope_rotate(q, np.array([pq + d]), 256, theta) *
                         oracle.rope_rotate(k, np.array([pk + d]), 256, theta))
        assert abs(base - shifted) <= 1e-9 * max(1.0, abs(base))


def test_rope_sign_convention_is_a_forward_rotation():
    # (1, 0) in pair j turns to (cos a, sin a): the second component gains +sin.
    x = np.zeros((1, 1, 4))
    x[0, 0, 0] = 1.0
    y = oracle.rope_rotate(x, np.array([1]), 4, 1.0e4)[0, 0]
    np.testing.assert_allclose(y, [math.cos(1.0), 0.0, math.sin(1.0), 0.0], atol=1e-15)
