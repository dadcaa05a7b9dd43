"""Pins for the oracle's range verification and list-based compaction (CPU only).

Eq. 2 and Section 4.2: removal drops exactly the rows of the named records,
keeps every other row in order and bit-identical, leaves the cursor alone and
rejects ranges that do not name live tokens. Checked by brute force over all
masks of small caches and by hypothesis over random holes and ranges.
"""
import itertools

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import synth


def _mask_to_ranges(pos, mask):
    """Maximal runs of removed rows with contiguous positions -> position ranges."""
    ranges = []
    i = 0
    n = len(pos)
    while i < n:
        if mask[i]:
            j = i
            while j + 1 < n and mask[j + 1] and pos[j + 1] == pos[j] + 1:
                j += 1
            ranges.append((int(pos[i]), int(pos[j]) + 1))
            i = j + 1
        else:
            i += 1
    return ranges


def test_compaction_brute_force_all_masks():
    # every removal mask of a 10-row cache whose positions have two holes
    pos = np.array([0, 1, 2, 5, 6, 7, 8, 12, 13, 14])
    for bits in itertools.product([0, 1], repeat=len(pos)):
        mask = np.array(bits, dtype=bool)
        ranges = _mask_to_ranges(pos, mask)
        src, kept = oracle.compact(pos, ranges)
        assert list(src) == [i for i in range(len(pos)) if not mask[i]]
        assert list(kept) == [int(p) for i, p in enumerate(pos) if not mask[i]]


@settings(max_examples=200, deadline=None)
@given(st.integers(1, 300), st.data())
def test_compaction_properties(L, data):
    # positions with holes: a sorted random subset of [0, 3L)
    rng = np.random.default_rng(data.draw(st.integers(0, 2 ** 31)))
    pos = np.sort(rng.choice(3 * L, size=L, replace=False))
    mask = rng.random(L) < data.draw(st.floats(0.0, 0.6))
    ranges = _mask_to_ranges(pos, mask)
    rows = rng.integers(0, 1 << 16, size=(L, 3)).astype(np.uint16)
    oracle.validate_ranges(ranges, pos, int(pos[-1]) + 1)     # they name live tokens
    src, kept = oracle.compact(pos, ranges)
    # order preserved, values identical, count = L - removed
    assert np.all(np.diff(src) > 0)
    assert len(src) == L - int(mask.sum())
    assert np.array_equal(rows[src], rows[~mask])
    assert np.array_equal(kept, pos[~mask])
    # src_index[j] >= j: compaction only moves rows toward the front
    assert np.all(src >= np.arange(len(src)))


def test_compaction_leaves_cursor_and_makes_holes():
    sc = synth.make_scenario(0, seed=0)
    r = sc.chars[0].rounds[0]
    L = r.L_old
    pos = np.arange(L)
    k = np.arange(L * 4, dtype=np.uint16).reshape(L, 1, 4)
    upd = oracle.attention_layer_update(pos, k, k, r.ranges, r.cursor,
                                        np.zeros((0, 2, 4), np.uint16), np.zeros((0, 1, 4), np.uint16),
                                        np.zeros((0, 1, 4), np.uint16), 4, 1e4, 0.5,
                                        live=oracle.live_positions(r.intervals))
    removed = int(np.sum(r.ranges[:, 1] - r.ranges[:, 0]))
    assert upd["L_keep"] == L - removed == 240
    assert upd["cursor"] == r.cursor                   # T = 0: pure deletion
    kept = upd["pos"]
    for (a, b) in r.ranges:                            # holes, no placeholder rows
        assert not np.any((kept >= a) & (kept < b))


@pytest.mark.parametrize("ranges,err", [
    ([(5, 5)], "empty"),
    ([(10, 20), (15, 25)], "sorted"),
    ([(20, 30), (10, 15)], "sorted"),
    ([(3, 9)], "not live"),            # crosses the hole at 4..5
    ([(95, 101)], "cursor"),
    ([(-1, 2)], "cursor"),
])
def test_validate_ranges_rejects(ranges, err):
    live = [p for p in range(100) if p not in (4, 5)]
    with pytest.raises(oracle.RangeError, match=err):
        oracle.validate_ranges(ranges, live, 100)


def test_validate_ranges_accepts_adjacent_and_empty_list():
    live = list(range(50))
    oracle.validate_ranges([(0, 10), (10, 20), (49, 50)], live, 50)
    oracle.validate_ranges([], live, 50)


def test_scenarios_draw_valid_records():
    for cfg in (0, 1, 2, 3):
        sc = synth.make_scenario(cfg, seed=0, n_chars=4 if cfg == 3 else None)
        for ch in sc.chars:
            for r in ch.rounds:
                oracle.validate_ranges(r.ranges, oracle.live_positions(r.intervals), r.cursor)
                assert r.L_keep == r.L_old - int(np.sum(r.ranges[:, 1] - r.ranges[:, 0]))
