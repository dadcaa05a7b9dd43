"""Key relocation for the placement variants of the maintained update (test
infrastructure only).

Paper Section 5.2 lists maintenance arms that differ only in the rotary positions
the replacement tokens carry (compared in Section 6.3, Table 2):
  * true tail: the replacement is computed and kept at the next positions after
    the cursor;
  * slot-preserving: the recurrence advances at the causal work tail, but the
    replacement's queries and keys are rotated at positions inside the original
    slot, and the cached rows are then labelled with those positions;
  * tail-and-relocate: computed at the true tail, after which the stored keys are
    rotated back to the old positions; values and the recurrent state stay as they
    are.

Relocating a stored key from position p to p + delta multiplies each rotary pair
(j, j + r/2), read as the complex number x_j + i x_{j+r/2}, by exp(i delta omega_j):
rotations compose, so the stored key R(p) k becomes R(p + delta) k up to the
rounding of the stored bf16 value. The rotation is applied to the stored (already
rounded) key in float64 and rounded to bf16 once more, nearest even.
"""
import numpy as np

from .bf16 import bf16_to_f64, f64_to_bf16
from .rope import rope_rotate


def check_new_positions(new_pos, other_live) -> None:
    """Positions a placement gives to tail rows must be non-negative, distinct and not
    held by any other live row. Raises ValueError otherwise."""
    new_pos = np.asarray(new_pos, dtype=np.int64)
    if np.any(new_pos < 0):
        raise ValueError("negative position")
    if len(np.unique(new_pos)) != len(new_pos):
        raise ValueError("a position is given twice")
    if np.intersect1d(new_pos, np.asarray(other_live, dtype=np.int64)).size:
        raise ValueError("a position is already live")


def relocate_keys(pos, k_bits, moves, rotary_dim: int, theta: float):
    """pos: int [n] position of every cache row; k_bits: bf16 bits [n, Hkv, D] (stored,
    rotated keys); moves: [m, 3] rows (src_begin, src_end, dst_begin).

    Every row whose position p lies in some [src_begin, src_end) is rotated by
    delta = dst_begin - src_begin and relabelled p + delta; other rows are unchanged.
    Returns (new pos, new k bits). Source ranges must be disjoint; the relabelled
    positions must not collide with each other or with the rows that stay.
    """
    pos = np.asarray(pos, dtype=np.int64)
    k_bits = np.asarray(k_bits, dtype=np.uint16)
    moves = np.asarray(moves, dtype=np.int64).reshape(-1, 3)
    delta = np.zeros(len(pos), dtype=np.int64)
    moved = np.zeros(len(pos), dtype=bool)
    for (s, e, d) in moves:
        if e <= s:
            raise ValueError("empty source range")
        hit = (pos >= s) & (pos < e)
        if np.any(moved & hit):
            raise ValueError("source ranges overlap")
        moved |= hit
        delta[hit] = d - s
    new_pos = pos + delta
    check_new_positions(new_pos[moved], new_pos[~moved])
    out = k_bits.copy()
    if np.any(moved):
        out[moved] = f64_to_bf16(rope_rotate(bf16_to_f64(k_bits[moved]), delta[moved], rotary_dim, theta))
    return new_pos, out
