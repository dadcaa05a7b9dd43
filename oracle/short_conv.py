"""Short causal convolution continued from its carried state, float64 (test
infrastructure only).

Paper, Section 4.1 and the caption of Fig. 2: besides the attention KV and the
recurrent state, the hybrid model's recurrent layers keep a convolution state,
and an update continues it over the replacement tokens without rollback (it
cannot be edited record by record). The paper does not write the convolution
out; it is read here as the short depthwise causal convolution of Gated DeltaNet
layers (the layers the paper cites), applied per channel of a projected tensor
x [T][C]:

    y_t[c] = act( sum_{j=0}^{W-1} w[c][j] * xt[t + j][c] )

where xt = (the W-1 carried input rows, then the T new rows) and act is SiLU
(x * sigmoid(x)) or the identity. The carried state after the call is the last
W-1 rows of xt. Inputs, weights, outputs and state are bfloat16; the outputs are
rounded to bfloat16 (round-to-nearest-even) from the exact float64 value.
"""
import numpy as np

from .bf16 import bf16_to_f64, f64_to_bf16


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x), evaluated without overflow for large |x|."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = x[pos] / (1.0 + np.exp(-x[pos]))
    e = np.exp(x[~pos])
    out[~pos] = x[~pos] * e / (1.0 + e)
    return out


def short_conv_continue(state_bits, x_bits, w_bits, activation: str = "silu"):
    """state_bits [W-1][C], x_bits [T][C], w_bits [C][W] (bf16 bit patterns).

    Returns (y_bits [T][C] bf16, y [T][C] float64 before rounding, new_state_bits [W-1][C]).
    """
    w = bf16_to_f64(w_bits)
    C, W = w.shape
    state_bits = np.asarray(state_bits, dtype=np.uint16).reshape(W - 1, C)
    x_bits = np.asarray(x_bits, dtype=np.uint16).reshape(-1, C)
    T = x_bits.shape[0]
    xt_bits = np.concatenate([state_bits, x_bits], axis=0)     # [W-1+T][C]
    xt = bf16_to_f64(xt_bits)
    y = np.zeros((T, C), dtype=np.float64)
    for j in range(W):
        y += w[:, j][None, :] * xt[j:j + T]
    if activation == "silu":
        y = silu(y)
    elif activation != "none":
        raise ValueError("activation is 'silu' or 'none'")
    y_bits = f64_to_bf16(y) if T else np.zeros((0, C), np.uint16)
    new_state = xt_bits[T:].copy()
    return y_bits, y, new_state
