"""Gated delta-rule recurrence in float64 (test infrastructure only).

Paper, Section 4.1: the recurrent layers are Gated DeltaNet layers (Yang et al.,
2025); only each layer's latest state is kept, and an update continues that
state over the replacement tokens without rollback (Eq. 3). The paper does not
write the recurrence out; it is read here in the Gated DeltaNet form, with the
state S a d_v x d_k matrix per value head:

    S_t = g_t * S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
    o_t = scale * S_t q_t          (read after the update)

g_t in (0, 1] is the multiplicative decay gate, beta_t in (0, 1) the write
strength; value head h reads key/query head h // (Hv / Hk).

`gated_delta_tokens` is the definition (one token at a time). `gated_delta_chunked`
regroups the same recurrence into chunks (the WY/UT form of the chunked delta
rule) and exists only so the tests can check that regrouping against the
definition; it is never the parity reference.
"""
import numpy as np


def _heads(Hk: int, Hv: int) -> np.ndarray:
    if Hv % Hk:
        raise ValueError("Hv must be a multiple of Hk")
    return np.arange(Hv) // (Hv // Hk)


def gated_delta_tokens(S0, q, k, v, beta, g, scale):
    """S0: [Hv, d_v, d_k]; q, k: [T, Hk, d_k]; v: [T, Hv, d_v]; beta, g: [T, Hv].

    Returns (o [T, Hv, d_v], S_T [Hv, d_v, d_k]) in float64.
    """
    S = np.array(S0, dtype=np.float64, copy=True)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    T = q.shape[0]
    Hv, dv, dk = S.shape
    kh = _heads(q.shape[1], Hv)
    o = np.zeros((T, Hv, dv), dtype=np.float64)
    for t in range(T):
        kt = k[t, kh, :]                                  # [Hv, d_k]
        qt = q[t, kh, :]
        bt = beta[t][:, None, None]
        gt = g[t][:, None, None]
        Sk = np.einsum("hij,hj->hi", S, kt)               # S_{t-1} k_t
        erase = np.einsum("hi,hj->hij", Sk, kt)           # S_{t-1} k_t k_t^T
        write = np.einsum("hi,hj->hij", v[t], kt)         # v_t k_t^T
        S = gt * (S - bt * erase) + bt * write
        o[t] = scale * np.einsum("hij,hj->hi", S, qt)
    return o, S


def gated_delta_chunked(S0, q, k, v, beta, g, scale, chunk: int):
    """Same recurrence, regrouped into chunks that start at the first token.

    Within a chunk (rows r, i = 0..C-1), with lg_r = sum_{s<=r} log g_s and
    G[r, i] = exp(lg_r - lg_i) for i <= r:
      M = strictly-lower( diag(beta) (G * K K^T) ),  A = (I + M)^-1
      U = A diag(beta) V - A diag(beta * exp(lg)) K S^T
      O = scale * ( diag(exp(lg)) Q S^T + lower(G * Q K^T) U )
      S <- exp(lg_last) S + U^T diag(G[last, :]) K
    Only ratios exp(lg_r - lg_i) <= 1 are formed, never 1/exp(lg).
    """
    S = np.array(S0, dtype=np.float64, copy=True)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    T = q.shape[0]
    Hv, dv, dk = S.shape
    kh = _heads(q.shape[1], Hv)
    o = np.zeros((T, Hv, dv), dtype=np.float64)
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        C = t1 - t0
        low_strict = np.tril(np.ones((C, C)), -1)
        low = np.tril(np.ones((C, C)), 0)
        for h in range(Hv):
            K = k[t0:t1, kh[h], :]
            Q = q[t0:t1, kh[h], :]
            V = v[t0:t1, h, :]
            b = beta[t0:t1, h]
            lg = np.cumsum(np.log(g[t0:t1, h]))
            G = np.exp(np.minimum(lg[:, None] - lg[None, :], 0.0)) * low
            M = low_strict * (b[:, None] * G * (K @ K.T))
            A = np.linalg.inv(np.eye(C) + M)
            U = A @ (b[:, None] * V) - A @ ((b * np.exp(lg))[:, None] * K) @ S[h].T
            O = np.exp(lg)[:, None] * (Q @ S[h].T) + (low * G * (Q @ K.T)) @ U
            o[t0:t1, h, :] = scale * O
            S[h] = np.exp(lg[-1]) * S[h] + U.T @ (G[-1][:, None] * K)
    return o, S
