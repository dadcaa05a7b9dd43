"""Pins for the oracle's gated delta-rule recurrence (CPU only).

P-D1  the chunked (WY/UT) regrouping equals the per-token definition, for
      several chunk sizes including 1 and ragged last chunks;
P-D2  continuing from a carried state equals one uninterrupted pass;
P-D3  closed form with unit keys: S_t k_t = g_t (1 - beta_t) S_{t-1} k_t + beta_t v_t;
P-D4  textbook special cases: beta = 0 is pure decay; g = beta = 1 with k = e_i
      overwrites column i of S with v; d = 1 is a scalar first-order recurrence;
P-S1  removals never touch the state: R rounds equal one pass over the
      concatenated tails;
a hand-worked two-token example, and pure-Python loops on tiny shapes.
"""
import numpy as np
import pytest

import oracle
import synth


def _inputs(rng, T, Hk, Hv, d, unit_k=True):
    q = rng.normal(size=(T, Hk, d))
    k = rng.normal(size=(T, Hk, d))
    if unit_k:
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.normal(size=(T, Hv, d))
    beta = 1 / (1 + np.exp(-rng.normal(size=(T, Hv))))
    g = np.exp(-np.log1p(np.exp(rng.normal(-4, 1, size=(T, Hv)))))
    S0 = rng.normal(0, 0.1, size=(Hv, d, d))
    return S0, q, k, v, beta, g


def test_hand_worked_two_tokens():
    # d_k = d_v = 2, one head, scale 1.
    # t=1: k=(1,0) v=(2,3) beta=.5 g=.5 q=(1,1), S0 = 0.5 I
    #   S0(I - .5 k k^T) = [[.25,0],[0,.5]]; *g -> [[.125,0],[0,.25]]; + .5 v k^T -> [[1.125,0],[1.5,.25]]
    #   o1 = S1 q1 = (1.125, 1.75)
    # t=2: k=(.6,.8) v=(-1,1) beta=.25 g=1 q=(2,0)
    #   S1 k2 = (.675, 1.1); S1 - .25 (S1 k2) k2^T = [[1.02375,-.135],[1.335,.03]]
    #   + .25 v k2^T = [[-.15,-.2],[.15,.2]] -> S2 = [[.87375,-.335],[1.485,.23]]; o2 = (1.7475, 2.97)
    S0 = 0.5 * np.eye(2)[None]
    q = np.array([[[1.0, 1.0]], [[2.0, 0.0]]])
    k = np.array([[[1.0, 0.0]], [[0.6, 0.8]]])
    v = np.array([[[2.0, 3.0]], [[-1.0, 1.0]]])
    beta = np.array([[0.5], [0.25]])
    g = np.array([[0.5], [1.0]])
    o, S = oracle.gated_delta_tokens(S0, q, k, v, beta, g, 1.0)
    np.testing.assert_allclose(o[:, 0], [[1.125, 1.75], [1.7475, 2.97]], atol=1e-14)
    np.testing.assert_allclose(S[0], [[0.87375, -0.335], [1.485, 0.23]], atol=1e-14)


@pytest.mark.parametrize("T,chunk", [(37, 1), (37, 4), (64, 16), (100, 16), (128, 64), (130, 64), (5, 64)])
def test_chunked_equals_per_token(T, chunk):
    rng = np.random.default_rng(20 + T + chunk)
    S0, q, k, v, beta, g = _inputs(rng, T, 2, 4, 16)
    o1, S1 = oracle.gated_delta_tokens(S0, q, k, v, beta, g, 0.25)
    o2, S2 = oracle.gated_delta_chunked(S0, q, k, v, beta, g, 0.25, chunk)
    np.testing.assert_allclose(o2, o1, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(S2, S1, rtol=1e-10, atol=1e-12)


def test_chunked_equals_per_token_under_strong_decay():
    rng = np.random.default_rng(29)
    S0, q, k, v, beta, _ = _inputs(rng, 128, 1, 1, 8)
    g = np.full((128, 1), 1e-3)          # cumulative decay underflows a naive 1/gamma
    o1, S1 = oracle.gated_delta_tokens(S0, q, k, v, beta, g, 1.0)
    o2, S2 = oracle.gated_delta_chunked(S0, q, k, v, beta, g, 1.0, 64)
    assert np.all(np.isfinite(o2))
    np.testing.assert_allclose(o2, o1, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(S2, S1, rtol=1e-9, atol=1e-14)


def test_continuation_equals_one_pass():
    rng = np.random.default_rng(21)
    S0, q, k, v, beta, g = _inputs(rng, 50, 2, 2, 8)
    o_all, S_all = oracle.gated_delta_tokens(S0, q, k, v, beta, g, 0.5)
    cut = 17
    o_a, S_a = oracle.gated_delta_tokens(S0, q[:cut], k[:cut], v[:cut], beta[:cut], g[:cut], 0.5)
    o_b, S_b = oracle.gated_delta_tokens(S_a, q[cut:], k[cut:], v[cut:], beta[cut:], g[cut:], 0.5)
    assert np.array_equal(np.concatenate([o_a, o_b]), o_all)
    assert np.array_equal(S_b, S_all)


def test_unit_key_closed_form():
    rng = np.random.default_rng(22)
    S0, q, k, v, beta, g = _inputs(rng, 12, 1, 1, 6)
    S = S0.copy()
    for t in range(12):
        prev_Sk = S[0] @ k[t, 0]
        _, S = oracle.gated_delta_tokens(S, q[t:t + 1], k[t:t + 1], v[t:t + 1], beta[t:t + 1], g[t:t + 1], 1.0)
        want = g[t, 0] * (1 - beta[t, 0]) * prev_Sk + beta[t, 0] * v[t, 0]
        np.testing.assert_allclose(S[0] @ k[t, 0], want, rtol=1e-12, atol=1e-14)


def test_special_cases():
    rng = np.random.default_rng(23)
    S0, q, k, v, beta, g = _inputs(rng, 9, 1, 2, 5)
    # beta = 0: pure decay, S_T = prod(g) S0, o_t = scale * S_t q_t
    o, S = oracle.gated_delta_tokens(S0, q, k, v, np.zeros_like(beta), g, 0.3)
    np.testing.assert_allclose(S, np.prod(g, axis=0)[:, None, None] * S0, rtol=1e-13)
    # g = beta = 1 and k = e_i: column i of S becomes v, other columns unchanged
    i = 3
    e = np.zeros((1, 1, 5))
    e[0, 0, i] = 1
    _, S1 = oracle.gated_delta_tokens(S0, q[:1], e, v[:1], np.ones((1, 2)), np.ones((1, 2)), 1.0)
    for h in range(2):
        want = S0[h].copy()
        want[:, i] = v[0, h]
        np.testing.assert_allclose(S1[h], want, rtol=1e-15, atol=1e-15)
    # d = 1: s_t = g_t (1 - beta_t k_t^2) s_{t-1} + beta_t v_t k_t ; o_t = scale s_t q_t
    T = 20
    q1 = rng.normal(size=(T, 1, 1))
    k1 = rng.normal(size=(T, 1, 1))
    v1 = rng.normal(size=(T, 1, 1))
    b1 = rng.random(size=(T, 1))
    g1 = rng.random(size=(T, 1))
    s = 0.7
    o, S = oracle.gated_delta_tokens(np.array([[[s]]]), q1, k1, v1, b1, g1, 2.0)
    for t in range(T):
        s = g1[t, 0] * (1 - b1[t, 0] * k1[t, 0, 0] ** 2) * s + b1[t, 0] * v1[t, 0, 0] * k1[t, 0, 0]
        assert abs(o[t, 0, 0] - 2.0 * s * q1[t, 0, 0]) < 1e-12
    assert abs(S[0, 0, 0] - s) < 1e-13


def test_output_is_read_after_update():
    # from a zero state one token gives o = scale * beta * v * (k . q)
    rng = np.random.default_rng(24)
    _, q, k, v, beta, g = _inputs(rng, 1, 1, 1, 4)
    o, _ = oracle.gated_delta_tokens(np.zeros((1, 4, 4)), q, k, v, beta, g, 0.5)
    np.testing.assert_allclose(o[0, 0], 0.5 * beta[0, 0] * v[0, 0] * (k[0, 0] @ q[0, 0]), rtol=1e-14)


def test_value_heads_share_key_heads_in_groups():
    # Hv = 4 value heads over Hk = 2 key heads: heads 0,1 read key head 0
    rng = np.random.default_rng(25)
    S0, q, k, v, beta, g = _inputs(rng, 6, 2, 4, 3)
    o, S = oracle.gated_delta_tokens(S0, q, k, v, beta, g, 1.0)
    for h in range(4):
        oh, Sh = oracle.gated_delta_tokens(S0[h:h + 1], q[:, h // 2:h // 2 + 1], k[:, h // 2:h // 2 + 1],
                                           v[:, h:h + 1], beta[:, h:h + 1], g[:, h:h + 1], 1.0)
        np.testing.assert_allclose(o[:, h], oh[:, 0], rtol=1e-14)
        np.testing.assert_allclose(S[h], Sh[0], rtol=1e-14)


def test_brute_force_loops():
    rng = np.random.default_rng(26)
    T, d = 4, 3
    S0, q, k, v, beta, g = _inputs(rng, T, 1, 1, d, unit_k=False)
    o, S = oracle.gated_delta_tokens(S0, q, k, v, beta, g, 0.9)
    St = [[S0[0, i, j] for j in range(d)] for i in range(d)]
    for t in range(T):
        kt = [k[t, 0, j] for j in range(d)]
        Sk = [sum(St[i][j] * kt[j] for j in range(d)) for i in range(d)]
        St = [[g[t, 0] * (St[i][j] - beta[t, 0] * Sk[i] * kt[j]) + beta[t, 0] * v[t, 0, i] * kt[j]
               for j in range(d)] for i in range(d)]
        for i in range(d):
            ref = 0.9 * sum(St[i][j] * q[t, 0, j] for j in range(d))
            assert abs(o[t, 0, i] - ref) < 1e-12
    assert np.allclose(S[0], np.array(St), atol=1e-13)


def test_rounds_equal_one_pass_over_concatenated_tails():
    # cfg-2-shaped (small heads): removals never touch the recurrent state
    shape = synth.DeltaShape(1, 2, 16, 16, 16)
    S0 = synth.gen_delta_state(0, 2, 1, shape)
    parts = [synth.gen_delta_inputs(0, 2, 1, T, shape, rnd=r) for r, T in enumerate([20, 33, 7])]
    S = S0.astype(np.float64)
    outs = []
    for (q, k, v, b, g) in parts:
        o, S = oracle.delta_layer_update(S, q, k, v, b, g, shape.scale)
        outs.append(o)
    cat = [np.concatenate([p[i] for p in parts]) for i in range(5)]
    o_all, S_all = oracle.delta_layer_update(S0, *cat, shape.scale)
    np.testing.assert_array_equal(np.concatenate(outs), o_all)
    np.testing.assert_array_equal(S, S_all)
