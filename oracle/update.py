"""The maintained update of one character context, composed from the oracle's
steps in the paper's order (test infrastructure only).

Paper, Section 4.1: a context is the state (A_t, R_t, p_t): attention cache,
recurrent state, next position id. Eq. 2 drops the direct cache entries of the
superseded records; Eq. 3 runs the replacement tokens through the model at the
true tail: positions p_t, p_t + 1, ...; they read the surviving entries; the
recurrence continues from R_t; the cursor advances by the number of new tokens.

Section 5.2 defines the comparison constructions used by the tests: dense
refill reads the whole current text from position 0, and fresh gapped prefill
reads it sequentially with every record at its maintained position.

All bf16 quantities are passed as uint16 bit patterns; floating-point results
are float64.
"""
from typing import Optional, Sequence, Tuple

import numpy as np

from .attention import causal_gqa_attention
from .bf16 import bf16_to_f64, f64_to_bf16
from .compaction import compact, validate_ranges
from .delta import gated_delta_tokens
from .placement import check_new_positions, relocate_keys
from .rope import rope_rotate


def attention_layer_update(pos, k_cache, v_cache, ranges, cursor: int, q, k, v, rotary_dim: int,
                           theta: float, scale: float, live: Optional[Sequence[int]] = None,
                           rows: Optional[Sequence[int]] = None, post_ranges=None, placement: str = "tail",
                           tail_positions=None):
    """One attention layer of one character: Eq. 2 then the attention part of Eq. 3.

    pos: int [L_old] position of every cache row; k_cache, v_cache: bf16 bits
    [L_old, Hkv, D]; ranges: [n, 2] half-open position ranges to remove;
    q: bf16 bits [T, Hq, D]; k, v: bf16 bits [T, Hkv, D] (k before rotation).
    `live`, when given, is checked against the ranges first (Section 4.2).

    post_ranges: [m, 2] position ranges inside the tail [cursor, cursor + T) whose
    rows are removed after the tail is processed (Section 4.1: temporary maintenance
    delimiters, processed and then dropped from the retained KV). Every tail row is
    still computed and attended to first; only the returned cache, positions and
    cursor reflect the removal (the cursor still advances by T).

    placement (Section 5.2; the variants compared in Section 6.3):
      "tail"      the replacement is rotated and kept at cursor + i (the method);
      "slot"      it is rotated at tail_positions[i] (inside the original slot) while
                  it is still computed after every surviving row (the causal work
                  tail), and its rows keep those positions; the cursor becomes
                  max(cursor, max(tail_positions) + 1);
      "relocate"  it is computed exactly as "tail", then its stored keys are rotated
                  from cursor + i to tail_positions[i] (relocate_keys) and its rows
                  relabelled; values are untouched and the cursor advances by T.
    post_ranges are given in the tail's final positions.
    """
    if live is not None:
        validate_ranges(ranges, live, cursor)
    src_index, kept_pos = compact(pos, ranges)
    T = int(np.asarray(q).shape[0])
    L_keep = len(src_index)
    true_tail = cursor + np.arange(T, dtype=np.int64)
    if placement == "tail":
        rot_pos, tail_pos, cursor_after = true_tail, true_tail, cursor + T
    elif placement in ("slot", "relocate"):
        tail_pos = np.asarray(tail_positions, dtype=np.int64).reshape(-1)
        if tail_pos.shape != (T,):
            raise ValueError("one position per tail token")
        check_new_positions(tail_pos, kept_pos)
        if placement == "slot":
            rot_pos = tail_pos
            cursor_after = max(cursor, int(tail_pos.max()) + 1) if T else cursor
        else:
            rot_pos = true_tail
            cursor_after = max(cursor + T, int(tail_pos.max()) + 1) if T else cursor
    else:
        raise ValueError(f"unknown placement {placement!r}")
    q_hat = f64_to_bf16(rope_rotate(bf16_to_f64(q), rot_pos, rotary_dim, theta))
    k_hat = f64_to_bf16(rope_rotate(bf16_to_f64(k), rot_pos, rotary_dim, theta))
    k_all = np.concatenate([np.asarray(k_cache)[src_index], k_hat], axis=0)
    v_all = np.concatenate([np.asarray(v_cache)[src_index], np.asarray(v, dtype=np.uint16)], axis=0)
    out = causal_gqa_attention(bf16_to_f64(q_hat), bf16_to_f64(k_all), bf16_to_f64(v_all), L_keep,
                               scale, rows=rows)
    if placement == "relocate" and T:
        # the stored keys move from their computed positions to the slot, one token at a time
        moves = np.stack([true_tail, true_tail + 1, tail_pos], axis=1)
        _, k_all = relocate_keys(np.concatenate([kept_pos, true_tail]), k_all, moves, rotary_dim, theta)
    final_pos = np.concatenate([kept_pos, tail_pos])
    post_index = np.arange(len(final_pos))
    if post_ranges is not None and len(post_ranges):
        post = np.asarray(post_ranges, dtype=np.int64).reshape(-1, 2)
        in_tail = [np.all(np.isin(np.arange(a, b), tail_pos)) for (a, b) in post]
        if not all(in_tail):
            raise ValueError("post-prefill ranges must lie inside the tail")
        validate_ranges([tuple(r) for r in post], final_pos.tolist(), cursor_after)
        post_index, final_pos = compact(final_pos, [tuple(r) for r in post])
        k_all, v_all = k_all[post_index], v_all[post_index]
    return {
        "src_index": src_index,
        "L_keep": L_keep,
        "pos": np.asarray(final_pos),
        "post_index": np.asarray(post_index),
        "k_cache": k_all,
        "v_cache": v_all,
        "q_hat": q_hat,
        "k_hat": k_hat,
        "out": out,
        "cursor": cursor_after,
    }


def delta_layer_update(S0, q, k, v, beta, g, scale):
    """One gated delta-rule layer: the recurrence continues from the carried state
    over the tail tokens (Eq. 3); removals never touch it. q, k, v are bf16 bits."""
    return gated_delta_tokens(S0, bf16_to_f64(q), bf16_to_f64(k), bf16_to_f64(v),
                              np.asarray(beta, dtype=np.float64), np.asarray(g, dtype=np.float64),
                              scale)


def prefill_attention(q, k, v, positions, rotary_dim: int, theta: float, scale: float,
                      rows: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Sequential prefill of a whole token sequence into an empty cache, each token
    rotated at the given position. Returns (out [N or len(rows), Hq, D], k_hat bits)."""
    positions = np.asarray(positions, dtype=np.int64)
    q_hat = f64_to_bf16(rope_rotate(bf16_to_f64(q), positions, rotary_dim, theta))
    k_hat = f64_to_bf16(rope_rotate(bf16_to_f64(k), positions, rotary_dim, theta))
    out = causal_gqa_attention(bf16_to_f64(q_hat), bf16_to_f64(k_hat), bf16_to_f64(v), 0, scale,
                               rows=rows)
    return out, k_hat


def refill_attention(q, k, v, rotary_dim: int, theta: float, scale: float, rows=None):
    """Dense refill (Section 5.2): the current text from position 0, contiguous."""
    N = int(np.asarray(q).shape[0])
    return prefill_attention(q, k, v, np.arange(N), rotary_dim, theta, scale, rows)


def gapped_refill_attention(q, k, v, positions, rotary_dim: int, theta: float, scale: float,
                            rows=None):
    """Fresh gapped prefill (Section 5.2): the current text read sequentially with
    every token at its maintained position (holes kept as gaps)."""
    return prefill_attention(q, k, v, positions, rotary_dim, theta, scale, rows)
