"""Dense masked causal grouped-query attention in float64 (test infrastructure only).

Paper, Section 4.1 (Eq. 3): replacement tokens appended at the tail read the
surviving cache entries; Section 4.3: their attention against the surviving
context is part of the remaining work. Read here as ordinary causal softmax
attention: tail row i (0-based) sees the L_keep surviving rows and the new rows
0..i, i.e. cache rows 0..L_keep+i; query head h reads key/value head
h // (Hq / Hkv); logits are scaled by `scale` (1/sqrt(D) by default); no window,
sink, soft-cap or gating.
"""
from typing import Optional, Sequence

import numpy as np


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, L_keep: int, scale: float,
                         rows: Optional[Sequence[int]] = None, row_block: int = 512) -> np.ndarray:
    """q: float64 [T, Hq, D]; k, v: float64 [L_keep + T, Hkv, D].

    Returns float64 [len(rows), Hq, D] (all T rows by default). `rows` selects
    tail rows; `row_block` only bounds memory: each row's softmax is computed on
    its own and the result does not depend on it.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, Hq, D = q.shape
    N, Hkv, _ = k.shape
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    if N < L_keep + T:
        raise ValueError("cache shorter than L_keep + T")
    G = Hq // Hkv
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), Hq, D), dtype=np.float64)
    for start in range(0, len(rows), row_block):
        rb = rows[start:start + row_block]
        limit = L_keep + rb                           # last visible cache row per tail row
        n_vis = int(limit.max()) + 1
        mask = np.arange(n_vis)[None, :] > limit[:, None]   # [rb, n_vis] True = hidden
        for h in range(Hq):
            g = h // G
            s = (q[rb, h, :] @ k[:n_vis, g, :].T) * scale   # [rb, n_vis]
            s = np.where(mask, -np.inf, s)
            m = np.max(s, axis=1, keepdims=True)
            p = np.exp(s - m)
            out[start:start + len(rb), h, :] = (p @ v[:n_vis, g, :]) / np.sum(p, axis=1, keepdims=True)
    return out
