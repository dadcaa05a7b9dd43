"""Range verification and list-based KV compaction (test infrastructure only).

Paper, Section 4.1, Eq. 2: the invalidated cache keeps every attention entry of
the live cache except the direct entries of the superseded records. Section 4.2:
the runtime checks each deletion range against the live spans before removing
anything, retains unrelated entries without replaying them, and leaves holes in
the position sequence (no dummy entries); the position cursor is unchanged by a
removal.

Ranges are half-open intervals [a, b) of position ids. The cache is kept in
position order (rows are appended at increasing positions and removal preserves
order), so "row i" and "the i-th live position" coincide.
"""
from typing import Iterable, List, Sequence, Tuple

import numpy as np


class RangeError(ValueError):
    """A deletion range that does not name live tokens of this context."""


def live_positions(intervals: Sequence[Tuple[int, int]]) -> np.ndarray:
    """Sorted live position ids described by disjoint half-open intervals."""
    parts = [np.arange(a, b, dtype=np.int64) for (a, b) in intervals]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


def validate_ranges(ranges: Iterable[Tuple[int, int]], live: Sequence[int], cursor: int) -> None:
    """Section 4.2 range verification, read as: every range is non-empty, the
    ranges are sorted and pairwise disjoint, every position they cover is below
    the cursor and currently live. Raises RangeError otherwise."""
    live_set = set(int(p) for p in live)
    prev_end = None
    for (a, b) in ranges:
        a = int(a)
        b = int(b)
        if b <= a:
            raise RangeError(f"empty range [{a},{b})")
        if prev_end is not None and a < prev_end:
            raise RangeError("ranges are not sorted and disjoint")
        if b > cursor or a < 0:
            raise RangeError(f"range [{a},{b}) reaches past the cursor {cursor}")
        for p in range(a, b):
            if p not in live_set:
                raise RangeError(f"position {p} is not live")
        prev_end = b


def compact(pos: Sequence[int], ranges: Iterable[Tuple[int, int]]):
    """Eq. 2 as a list filter: walk the cache rows in order and keep the rows
    whose position lies in none of the ranges.

    Returns (src_index, kept_pos): src_index[j] is the old row index of the j-th
    surviving row, kept_pos[j] its position id.
    """
    rs: List[Tuple[int, int]] = [(int(a), int(b)) for (a, b) in ranges]
    src: List[int] = []
    kept: List[int] = []
    for i, p in enumerate(np.asarray(pos).tolist()):
        removed = False
        for (a, b) in rs:
            if a <= p < b:
                removed = True
                break
        if not removed:
            src.append(i)
            kept.append(p)
    return np.asarray(src, dtype=np.int64), np.asarray(kept, dtype=np.int64)
