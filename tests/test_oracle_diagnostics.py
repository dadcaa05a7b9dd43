"""Pins for the oracle's attention diagnostics (paper Section 5.3, Appendix C; CPU only).

P-G1  library cross-check: the probe distribution equals torch's float32 softmax of
      the masked score matrix (explicit causal mask, heads repeated), averaged.
P-G2  the float32 reference softmax agrees with the float64 definition to float32
      rounding; the distribution sums to one.
P-G3  closed forms: identical keys give each probe query a uniform distribution over
      the rows it sees; a single row gets all the mass.
P-G4  group masses and boundary windows against pure-Python loops, rows in work order.
P-G5  effective group count: m equal groups -> m; one group -> 1; a two-group case by
      hand; total variation: 0 for equal, 1 for disjoint supports, symmetric, a
      worked example, row alignment by a map.
"""
import math

import numpy as np
import torch

import oracle
import synth


def _inputs(seed, L, n, Hq, Hkv, D):
    rng = np.random.default_rng(seed)
    q = synth.to_bf16_bits(rng.normal(size=(n, Hq, D)))
    k = synth.to_bf16_bits(rng.normal(size=(L, Hkv, D)))
    pos = np.sort(rng.choice(10 * L, size=L, replace=False))
    return q, k, pos


def test_probe_matches_torch_float32_softmax():
    for (L, n, Hq, Hkv, D) in [(40, 8, 4, 2, 16), (300, 8, 16, 2, 64), (9, 3, 2, 1, 8)]:
        q, k, pos = _inputs(L, L, n, Hq, Hkv, D)
        theta, scale = 1.0e7, D ** -0.5
        p = oracle.probe_distribution(q, pos[-n:], k, D, theta, scale)
        q_hat = oracle.bf16_to_f64(oracle.f64_to_bf16(oracle.rope_rotate(oracle.bf16_to_f64(q), pos[-n:], D, theta)))
        qt = torch.from_numpy(q_hat).float().permute(1, 0, 2)                                     # [Hq, n, D]
        kt = torch.from_numpy(oracle.bf16_to_f64(k)).float().permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)
        s = (qt @ kt.transpose(1, 2)) * scale                                                     # [Hq, n, L]
        seen = torch.arange(L)[None, :] <= (L - n + torch.arange(n))[:, None]
        probs = torch.softmax(s.masked_fill(~seen, float("-inf")), dim=-1)
        want = probs.double().mean(dim=(0, 1)).numpy()
        np.testing.assert_allclose(p, want, rtol=2e-5, atol=1e-9)


def test_float32_reference_agrees_with_float64():
    q, k, pos = _inputs(3, 500, 8, 8, 2, 128)
    p32 = oracle.probe_distribution(q, pos[-8:], k, 128, 1.0e7, 128 ** -0.5)
    p64 = oracle.probe_distribution(q, pos[-8:], k, 128, 1.0e7, 128 ** -0.5, dtype=np.float64)
    assert abs(p64.sum() - 1.0) < 1e-12 and abs(p32.sum() - 1.0) < 1e-6
    assert np.max(np.abs(p32 - p64)) <= 1e-6 * max(1.0, p64.max())
    assert np.abs(p32 - p64).sum() / p64.sum() < 1e-5


def test_probe_closed_forms():
    rng = np.random.default_rng(4)
    L, n, D = 20, 5, 8
    row = synth.to_bf16_bits(rng.normal(size=(1, 1, D)))
    k = np.repeat(row, L, axis=0)                   # every key identical
    q = synth.to_bf16_bits(rng.normal(size=(n, 2, D)))
    p = oracle.probe_distribution(q, np.arange(L - n, L), k, 0, 1.0e4, 0.7, dtype=np.float64)   # no rotation
    want = np.zeros(L)
    for i in range(n):
        want[: L - n + i + 1] += 1.0 / (L - n + i + 1)
    np.testing.assert_allclose(p, want / n, rtol=1e-13)
    one = oracle.probe_distribution(q[:1], np.array([7]), k[:1], D, 1.0e7, 0.3)
    assert one.shape == (1,) and abs(one[0] - 1.0) < 1e-7


def test_group_masses_against_loops():
    rng = np.random.default_rng(5)
    L = 60
    p = rng.random(L)
    p /= p.sum()
    pos = np.concatenate([np.arange(0, 20), np.arange(100, 130), np.arange(20, 30)])   # work order
    groups = np.array([[5, 25], [100, 104], [110, 140], [200, 210]])
    mass, win = oracle.group_masses(p, pos, groups, window=3)
    for g, (a, b) in enumerate(groups.tolist()):
        m = w = 0.0
        for j in range(L):
            if a <= pos[j] < b:
                m += p[j]
                if pos[j] < a + 3:
                    w += p[j]
        assert abs(mass[g] - m) < 1e-15 and abs(win[g] - w) < 1e-15
    assert mass[3] == 0.0


def test_effective_group_count_and_tv():
    M, eff, share = oracle.group_summary(np.full(7, 0.1), np.full(7, 0.01))
    assert abs(M - 0.7) < 1e-15 and abs(eff - 7.0) < 1e-12 and abs(share - 0.1) < 1e-12
    assert abs(oracle.group_summary([0.0, 0.4, 0.0], [0, 0, 0])[1] - 1.0) < 1e-15
    eff2 = oracle.group_summary([0.1, 0.3], [0, 0])[1]
    assert abs(eff2 - math.exp(-(0.25 * math.log(0.25) + 0.75 * math.log(0.75)))) < 1e-14
    p = np.array([0.5, 0.5, 0.0])
    q = np.array([0.0, 0.5, 0.5])
    assert oracle.tv_distance(p, p) == 0.0
    assert abs(oracle.tv_distance(p, q) - 0.5) < 1e-15 and oracle.tv_distance(q, p) == oracle.tv_distance(p, q)
    assert abs(oracle.tv_distance([1.0, 0.0], [0.0, 1.0]) - 1.0) < 1e-15
    # rows of the second construction in another order
    assert oracle.tv_distance(p, q[[2, 1, 0]], q_row_of_p=[2, 1, 0]) == oracle.tv_distance(p, q)
