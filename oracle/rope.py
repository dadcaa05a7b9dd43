"""Rotary position embedding in float64 (test infrastructure only).

The paper's model encodes positions with rotary embeddings (Section 4.2, citing
Su et al., RoFormer), and the true-tail update evaluates the replacement tokens
at their actual new tail positions. Read here in the rotate-half layout used by
the Qwen family: for a rotary dimension r (even, at most the head dimension)
and base theta, pair j < r/2 couples components j and j + r/2 and turns them by
the angle pos * omega_j with omega_j = theta ** (-2 j / r). Components at index
>= r are left unchanged. Angles are formed in float64.
"""
import numpy as np


def rope_frequencies(rotary_dim: int, theta: float) -> np.ndarray:
    j = np.arange(rotary_dim // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * j / np.float64(rotary_dim))


def rope_rotate(x: np.ndarray, positions: np.ndarray, rotary_dim: int, theta: float) -> np.ndarray:
    """x: float64 [n, H, D]; positions: int [n]. Returns the rotated float64 array."""
    x = np.asarray(x, dtype=np.float64)
    n, H, D = x.shape
    if rotary_dim % 2 or rotary_dim > D or rotary_dim < 0:
        raise ValueError("rotary_dim must be even and at most the head dimension")
    out = x.copy()
    if rotary_dim == 0:
        return out
    half = rotary_dim // 2
    omega = rope_frequencies(rotary_dim, theta)
    angle = np.asarray(positions, dtype=np.float64)[:, None] * omega[None, :]   # [n, half]
    c = np.cos(angle)[:, None, :]
    s = np.sin(angle)[:, None, :]
    a = x[:, :, :half]
    b = x[:, :, half:rotary_dim]
    out[:, :, :half] = a * c - b * s
    out[:, :, half:rotary_dim] = b * c + a * s
    return out
