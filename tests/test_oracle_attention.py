"""Pins for the oracle's causal GQA attention and the tail update (CPU only).

P-A1  library cross-check: torch's CPU float64 scaled_dot_product_attention with
      an explicit boolean mask and explicitly repeated KV heads.
P-A2  closed forms: one visible key returns its value; equal keys return the
      running mean of the visible values.
P-A3  zero removals: the tail rows equal the last T rows of a causal prefill of
      prefix + tail (the special case the method reduces to).
P-A4  with removals: the tail rows equal the last T rows of a fresh gapped
      prefill of the final text at the maintained positions (Section 5.2).
Brute force: pure-Python loops on tiny shapes.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth


def _sdpa_reference(q, k, v, L_keep, scale):
    T, Hq, D = q.shape
    N, Hkv, _ = k.shape
    G = Hq // Hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)                          # [Hq, T, D]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)  # [Hq, N, D]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, 0)
    allowed = torch.arange(N)[None, :] <= (L_keep + torch.arange(T))[:, None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=allowed, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("T,L_keep,Hq,Hkv,D", [(5, 0, 2, 1, 8), (7, 13, 4, 2, 16), (32, 240, 2, 1, 64),
                                               (16, 100, 16, 2, 32)])
def test_attention_matches_torch_sdpa(T, L_keep, Hq, Hkv, D):
    rng = np.random.default_rng(10 + T)
    q = rng.normal(size=(T, Hq, D))
    k = rng.normal(size=(L_keep + T, Hkv, D))
    v = rng.normal(size=(L_keep + T, Hkv, D))
    scale = D ** -0.5
    out = oracle.causal_gqa_attention(q, k, v, L_keep, scale)
    np.testing.assert_allclose(out, _sdpa_reference(q, k, v, L_keep, scale), rtol=1e-12, atol=1e-13)
    # row selection and row blocking do not change any row
    rows = [T - 1, 0, T // 2]
    np.testing.assert_allclose(oracle.causal_gqa_attention(q, k, v, L_keep, scale, rows=rows, row_block=2),
                               out[rows], rtol=1e-13, atol=1e-14)


def test_attention_closed_forms():
    rng = np.random.default_rng(11)
    D = 8
    # L_keep = 0: tail row 0 sees only its own key -> O = v_0 whatever q is
    q = rng.normal(size=(3, 2, D)) * 10
    k = rng.normal(size=(3, 1, D))
    v = rng.normal(size=(3, 1, D))
    out = oracle.causal_gqa_attention(q, k, v, 0, 0.3)
    np.testing.assert_allclose(out[0, 0], v[0, 0], rtol=1e-15)
    np.testing.assert_allclose(out[0, 1], v[0, 0], rtol=1e-15)
    # all keys equal -> uniform weights -> running mean of the visible values
    k_eq = np.repeat(rng.normal(size=(1, 1, D)), 6, axis=0)
    v6 = rng.normal(size=(6, 1, D))
    out = oracle.causal_gqa_attention(rng.normal(size=(4, 1, D)), k_eq, v6, 2, 1.0)
    for i in range(4):
        np.testing.assert_allclose(out[i, 0], v6[: 2 + i + 1, 0].mean(axis=0), rtol=1e-12)


def test_attention_brute_force_loops():
    rng = np.random.default_rng(12)
    T, L_keep, Hq, Hkv, D = 3, 4, 4, 2, 3
    q = rng.normal(size=(T, Hq, D))
    k = rng.normal(size=(L_keep + T, Hkv, D))
    v = rng.normal(size=(L_keep + T, Hkv, D))
    scale = 0.7
    out = oracle.causal_gqa_attention(q, k, v, L_keep, scale)
    for i in range(T):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            logits = [scale * sum(q[i, h, d] * k[j, g, d] for d in range(D)) for j in range(L_keep + i + 1)]
            mx = max(logits)
            w = [math.exp(s - mx) for s in logits]
            z = sum(w)
            for d in range(D):
                ref = sum(w[j] * v[j, g, d] for j in range(len(w))) / z
                assert abs(out[i, h, d] - ref) < 1e-12


def _raw_context(rng, n, Hq, Hkv, D):
    q = synth.to_bf16_bits(rng.normal(size=(n, Hq, D)))
    k = synth.to_bf16_bits(rng.normal(size=(n, Hkv, D)))
    v = synth.to_bf16_bits(rng.normal(size=(n, Hkv, D)))
    return q, k, v


@pytest.mark.parametrize("theta", [1.0e4, 1.0e7])
def test_zero_removals_equals_prefill(theta):
    rng = np.random.default_rng(13)
    L, T, Hq, Hkv, D = 40, 9, 4, 2, 16
    q, k, v = _raw_context(rng, L + T, Hq, Hkv, D)
    scale = D ** -0.5
    full_out, full_khat = oracle.refill_attention(q, k, v, D, theta, scale)
    # the cache a prefill of the first L tokens leaves behind
    cache_k = full_khat[:L]
    upd = oracle.attention_layer_update(np.arange(L), cache_k, v[:L], np.zeros((0, 2), np.int64), L,
                                        q[L:], k[L:], v[L:], D, theta, scale)
    np.testing.assert_allclose(upd["out"], full_out[L:], rtol=1e-12, atol=1e-13)
    assert np.array_equal(upd["k_cache"], full_khat)


def test_tail_rows_equal_gapped_refill():
    rng = np.random.default_rng(14)
    Hq, Hkv, D, theta = 4, 1, 16, 1.0e7
    scale = D ** -0.5
    # a context with an earlier hole, then a removal of two records, then a tail
    live_pos = np.array(list(range(0, 30)) + list(range(10030, 10060)))   # 10K gap between groups
    n = len(live_pos)
    q, k, v = _raw_context(rng, n, Hq, Hkv, D)
    cache_k = oracle.f64_to_bf16(oracle.rope_rotate(oracle.bf16_to_f64(k), live_pos, D, theta))
    cursor = 10060
    ranges = np.array([[5, 12], [10040, 10047]])
    T = 6
    tq, tk, tv = _raw_context(rng, T, Hq, Hkv, D)
    upd = oracle.attention_layer_update(live_pos, cache_k, v, ranges, cursor, tq, tk, tv, D, theta, scale,
                                        live=live_pos)
    src = upd["src_index"]
    final_pos = np.concatenate([live_pos[src], cursor + np.arange(T)])
    gq = np.concatenate([q[src], tq])
    gk = np.concatenate([k[src], tk])
    gv = np.concatenate([v[src], tv])
    g_out, g_khat = oracle.gapped_refill_attention(gq, gk, gv, final_pos, D, theta, scale)
    np.testing.assert_allclose(upd["out"], g_out[-T:], rtol=1e-12, atol=1e-13)
    assert np.array_equal(upd["k_cache"], g_khat)
    assert np.array_equal(upd["pos"], final_pos)


def test_post_prefill_delimiter_removal():
    # Section 4.1: maintenance delimiters are processed with the tail, then their direct
    # KV is removed. The retained cache must be the surviving rows plus the rotated keys
    # and values of the non-delimiter tail tokens at their own tail positions, built
    # here without the compaction routine; outputs are those of the full tail.
    rng = np.random.default_rng(15)
    L, T, Hq, Hkv, D, theta = 30, 12, 4, 2, 16, 1.0e7
    scale = D ** -0.5
    q, k, v = _raw_context(rng, L, Hq, Hkv, D)
    pos = np.arange(L)
    cache_k = oracle.f64_to_bf16(oracle.rope_rotate(oracle.bf16_to_f64(k), pos, D, theta))
    tq, tk, tv = _raw_context(rng, T, Hq, Hkv, D)
    ranges = np.array([[3, 7]])
    cursor = L
    post = np.array([[cursor, cursor + 2], [cursor + 9, cursor + 12]])   # an opening and a closing wrapper
    plain = oracle.attention_layer_update(pos, cache_k, v, ranges, cursor, tq, tk, tv, D, theta, scale)
    upd = oracle.attention_layer_update(pos, cache_k, v, ranges, cursor, tq, tk, tv, D, theta, scale,
                                        post_ranges=post)
    assert np.array_equal(upd["out"], plain["out"])
    keep_tail = np.ones(T, bool)
    keep_tail[0:2] = False
    keep_tail[9:12] = False
    tail_pos = cursor + np.arange(T)
    kh = oracle.f64_to_bf16(oracle.rope_rotate(oracle.bf16_to_f64(tk[keep_tail]), tail_pos[keep_tail], D, theta))
    survivors = np.concatenate([np.arange(0, 3), np.arange(7, L)])
    assert np.array_equal(upd["k_cache"], np.concatenate([cache_k[survivors], kh]))
    assert np.array_equal(upd["v_cache"], np.concatenate([v[survivors], tv[keep_tail]]))
    assert np.array_equal(upd["pos"], np.concatenate([survivors, tail_pos[keep_tail]]))
    assert upd["cursor"] == cursor + T                       # delimiter positions become holes
    empty = oracle.attention_layer_update(pos, cache_k, v, ranges, cursor, tq, tk, tv, D, theta, scale,
                                          post_ranges=np.zeros((0, 2), np.int64))
    assert np.array_equal(empty["k_cache"], plain["k_cache"]) and np.array_equal(empty["pos"], plain["pos"])
    with pytest.raises(ValueError):
        oracle.attention_layer_update(pos, cache_k, v, ranges, cursor, tq, tk, tv, D, theta, scale,
                                      post_ranges=np.array([[cursor - 1, cursor + 1]]))
