"""Attention diagnostics of the paper's measurement protocol (test infrastructure only).

Paper Section 5.3 and Appendix C: attention probabilities at a full-attention
layer are reconstructed with a float32 reference softmax from the queries and
keys the model actually holds; the diagnostics average the last eight query
tokens of a probe, then aggregate over heads (and layers); holes in the position
sequence hold no rows, so they never enter a denominator. From the averaged
token distribution p over the live cache rows:
  * the mass of each memory group (record) g: a_g = sum of p over the group's rows;
    the absolute memory mass M = sum_g a_g;
  * the within-memory shares a_g / M and the effective group count
    exp(-sum_g (a_g / M) log(a_g / M));
  * the boundary-window share: the mass of the first `window` (eight) tokens of every
    group, over M;
  * the token-distribution total variation distance between two constructions of
    the same text: 0.5 * sum_j |p_j - p'_j|, rows aligned token by token.

Probe queries are the last n rows of the context (in cache-row order); probe
query i of n sees rows 0 .. len - n + i, the causal rule of the update.
"""
import numpy as np

from .bf16 import bf16_to_f64, f64_to_bf16
from .rope import rope_rotate


def probe_distribution(q_bits, positions, k_cache, rotary_dim: int, theta: float, scale: float, dtype=np.float32):
    """q_bits: bf16 bits [n, Hq, D], the raw (unrotated) queries of the last n rows;
    positions: int [n], their positions; k_cache: bf16 bits [len, Hkv, D] (stored keys).

    The queries are rotated at their positions (float64 angles, bf16 nearest even, as
    the cache stores keys); scores q.k * scale, the softmax and the averaging are done
    in `dtype` (float32, the paper's reference softmax; float64 for the pins).
    Returns p [len]: the softmax rows averaged over the n queries and Hq heads."""
    q_hat = bf16_to_f64(f64_to_bf16(rope_rotate(bf16_to_f64(q_bits), positions, rotary_dim, theta)))
    k = bf16_to_f64(k_cache)
    n, Hq, D = q_hat.shape
    L, Hkv, _ = k.shape
    G = Hq // Hkv
    p = np.zeros(L, dtype=np.float64)
    for i in range(n):
        vis = L - n + i + 1
        for h in range(Hq):
            s = (q_hat[i, h].astype(dtype) @ k[:vis, h // G].astype(dtype).T) * dtype(scale)
            e = np.exp(s - s.max())
            p[:vis] += (e / e.sum(dtype=dtype)).astype(np.float64)
    return p / (n * Hq)


def group_masses(p, row_positions, groups, window: int = 8):
    """p: [len] token distribution over cache rows; row_positions: [len] their
    positions; groups: [m, 2] half-open position ranges (one per memory group).

    Returns (mass [m], window_mass [m]): the summed p of each group's rows, and of
    the rows among the group's first `window` positions."""
    p = np.asarray(p, dtype=np.float64)
    pos = np.asarray(row_positions, dtype=np.int64)
    groups = np.asarray(groups, dtype=np.int64).reshape(-1, 2)
    mass = np.zeros(len(groups))
    win = np.zeros(len(groups))
    for g, (a, b) in enumerate(groups):
        inside = (pos >= a) & (pos < b)
        mass[g] = p[inside].sum()
        win[g] = p[inside & (pos < a + window)].sum()
    return mass, win


def group_summary(mass, window_mass):
    """(memory mass M, effective group count, boundary-window share of M)."""
    mass = np.asarray(mass, dtype=np.float64)
    M = mass.sum()
    if M <= 0:
        return 0.0, 0.0, 0.0
    a = mass / M
    nz = a[a > 0]
    return float(M), float(np.exp(-np.sum(nz * np.log(nz)))), float(np.asarray(window_mass).sum() / M)


def tv_distance(p, q, q_row_of_p=None):
    """0.5 * sum_j |p_j - q_{map(j)}|, map the identity unless given."""
    p = np.asarray(p, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    if q_row_of_p is not None:
        q = q[np.asarray(q_row_of_p, dtype=np.int64)]
    return 0.5 * float(np.abs(p - q).sum())
