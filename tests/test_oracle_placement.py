"""Pins for the placement variants of the oracle (CPU only): slot-preserving and
tail-and-relocate placement of the replacement, and key relocation (paper
Section 5.2; compared in Section 6.3, Table 2).

P-L1  identity: slot placement at the true-tail positions is the true-tail update,
      bit for bit; so is tail-and-relocate with a zero shift.
P-L2  rotation group law, written independently with complex numbers: a stored key
      relocated from p1 to p2 equals the raw key rotated at p2 up to the rounding of
      the stored value (a bound computed element by element), at the paper's cursor
      scale; p1 -> p2 -> p1 returns within that bound twice; a zero shift is exact.
P-L3  closed form of slot placement on a tiny case: scores, softmax and output built
      from complex rotations at the slot positions; every tail row attends to every
      surviving row (work-order causality) whatever their positions.
P-L4  closed form of tail-and-relocate: outputs are those of the true tail, the
      stored keys those of the relocation, values untouched.
P-L5  bookkeeping: positions, cursor, holes; invalid placements are rejected.
"""
import numpy as np
import pytest

import oracle
import synth


def _cplx_rotate(x, pos, rdim, theta):
    """Rotate-half RoPE as complex multiplication: pair j is x_j + i x_{j+r/2} times
    exp(i pos theta^(-2j/r)). x: float64 [n, H, D]; pos: [n]."""
    x = np.asarray(x, np.float64)
    half = rdim // 2
    w = theta ** (-2.0 * np.arange(half) / rdim)
    z = (x[..., :half] + 1j * x[..., half:rdim]) * np.exp(1j * np.asarray(pos, np.float64)[:, None, None] * w)
    out = x.copy()
    out[..., :half] = z.real
    out[..., half:rdim] = z.imag
    return out


def _bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (bf16 keeps 8 significant bits)."""
    x = np.abs(np.asarray(x, np.float64))
    _, e = np.frexp(np.maximum(x, 2.0 ** -126))
    return np.ldexp(1.0, e - 8)


def _raw(rng, n, H, D):
    return synth.to_bf16_bits(rng.normal(size=(n, H, D)))


def _case(seed, L=24, T=6, Hq=4, Hkv=2, D=16):
    rng = np.random.default_rng(seed)
    kc = _raw(rng, L, Hkv, D)
    vc = _raw(rng, L, Hkv, D)
    q, k, v = _raw(rng, T, Hq, D), _raw(rng, T, Hkv, D), _raw(rng, T, Hkv, D)
    return kc, vc, q, k, v


def test_slot_and_zero_shift_relocation_are_the_true_tail():
    kc, vc, q, k, v = _case(1)
    pos = np.arange(24) * 3 + 5                 # a gapped live layout
    cursor, ranges, D, theta = 200, np.array([[14, 30]]), 16, 1.0e7
    base = oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, D ** -0.5)
    at_tail = cursor + np.arange(6)
    for placement in ("slot", "relocate"):
        alt = oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, D ** -0.5,
                                            placement=placement, tail_positions=at_tail)
        for key in ("src_index", "pos", "k_cache", "v_cache", "q_hat", "k_hat", "out"):
            assert np.array_equal(alt[key], base[key]), (placement, key)
        assert alt["cursor"] == base["cursor"] == cursor + 6


@pytest.mark.parametrize("theta", [1.0e4, 1.0e7])
def test_relocation_follows_the_rotation_group_law(theta):
    rng = np.random.default_rng(2)
    n, H, D = 64, 2, 64
    raw = synth.bf16_bits_to_f32(_raw(rng, n, H, D)).astype(np.float64)
    # the paper's cursors: true tail near 479,547, original slots near 261,955 and below
    p1 = rng.integers(400_000, 479_548, size=n)
    p2 = rng.integers(0, 261_956, size=n)
    stored = oracle.f64_to_bf16(_cplx_rotate(raw, p1, D, theta))
    moves = np.stack([p1, p1 + 1, p2], axis=1)
    new_pos, moved = oracle.relocate_keys(p1, stored, moves, D, theta)
    assert np.array_equal(new_pos, p2)
    got = oracle.bf16_to_f64(moved)
    want = _cplx_rotate(raw, p2, D, theta)
    # rounding of the stored key, rotated: per pair at most the norm of that error
    err_in = oracle.bf16_to_f64(stored) - _cplx_rotate(raw, p1, D, theta)
    half = D // 2
    pair = np.sqrt(err_in[..., :half] ** 2 + err_in[..., half:] ** 2)
    bound = np.concatenate([pair, pair], axis=-1) * (1 + 1e-9) + 0.5 * _bf16_ulp(got) + 1e-300
    assert np.all(np.abs(got - want) <= bound)
    # back again: within the rounding of two relocations of the original stored key
    _, back = oracle.relocate_keys(p2, moved, np.stack([p2, p2 + 1, p1], axis=1), D, theta)
    assert np.all(np.abs(oracle.bf16_to_f64(back) - oracle.bf16_to_f64(stored)) <=
                  2 * bound + _bf16_ulp(oracle.bf16_to_f64(stored)))
    # a zero shift and rows outside every source range are untouched
    same_pos, same = oracle.relocate_keys(p1, stored, np.stack([p1, p1 + 1, p1], axis=1), D, theta)
    assert np.array_equal(same, stored) and np.array_equal(same_pos, p1)
    part_pos, part = oracle.relocate_keys(p1, stored, np.array([[p1[0], p1[0] + 1, 7]]), D, theta)
    assert np.array_equal(part[1:], stored[1:]) and part_pos[0] == 7 and np.array_equal(part_pos[1:], p1[1:])


def test_relocation_leaves_dims_past_the_rotary_dimension():
    rng = np.random.default_rng(3)
    stored = _raw(rng, 5, 1, 32)
    pos = np.arange(5) + 100
    _, moved = oracle.relocate_keys(pos, stored, np.array([[100, 105, 3]]), 16, 1.0e7)
    assert np.array_equal(moved[..., 16:], stored[..., 16:])
    assert not np.array_equal(moved[..., :16], stored[..., :16])


def test_slot_placement_closed_form():
    # one KV head, D = 4 (two rotary pairs); cached keys at positions both before and
    # after the slot; the tail is placed in the hole the removed record leaves
    rng = np.random.default_rng(4)
    D, theta, scale = 4, 1.0e4, 0.5
    pos = np.array([0, 1, 2, 3, 4, 5, 40, 41])
    raw_k = synth.bf16_bits_to_f32(_raw(rng, 8, 1, D)).astype(np.float64)
    kc = oracle.f64_to_bf16(_cplx_rotate(raw_k, pos, D, theta))
    vc = _raw(rng, 8, 1, D)
    q, k, v = _raw(rng, 3, 1, D), _raw(rng, 3, 1, D), _raw(rng, 3, 1, D)
    ranges = np.array([[2, 5]])          # positions 2, 3, 4 leave
    slot = np.array([2, 3, 4])
    upd = oracle.attention_layer_update(pos, kc, vc, ranges, 42, q, k, v, D, theta, scale, placement="slot",
                                        tail_positions=slot)
    keep = np.array([0, 1, 5, 6, 7])
    qh = oracle.bf16_to_f64(oracle.f64_to_bf16(_cplx_rotate(synth.bf16_bits_to_f32(q), slot, D, theta)))
    kh = oracle.bf16_to_f64(oracle.f64_to_bf16(_cplx_rotate(synth.bf16_bits_to_f32(k), slot, D, theta)))
    keys = np.concatenate([oracle.bf16_to_f64(kc[keep]), kh])[:, 0]
    vals = np.concatenate([oracle.bf16_to_f64(vc[keep]), oracle.bf16_to_f64(v)])[:, 0]
    for i in range(3):
        vis = 5 + i + 1              # every surviving row (positions 40, 41 included) and tail rows 0..i
        s = scale * keys[:vis] @ qh[i, 0]
        p = np.exp(s - s.max())
        np.testing.assert_allclose(upd["out"][i, 0], p @ vals[:vis] / p.sum(), rtol=1e-12, atol=1e-14)
    assert np.array_equal(upd["pos"], np.array([0, 1, 5, 40, 41, 2, 3, 4]))
    assert upd["cursor"] == 42       # every slot position lies below the cursor


def test_relocate_placement_closed_form():
    kc, vc, q, k, v = _case(5, L=20, T=4, Hq=2, Hkv=1, D=8)
    pos, cursor, D, theta = np.arange(20), 20, 8, 1.0e7
    ranges = np.array([[6, 10]])
    slot = np.array([6, 7, 8, 9])
    tail = oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, D ** -0.5)
    rel = oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, D ** -0.5,
                                        placement="relocate", tail_positions=slot)
    assert np.array_equal(rel["out"], tail["out"])             # computed at the true tail
    assert np.array_equal(rel["v_cache"], tail["v_cache"])     # values are never touched
    keep = tail["L_keep"]
    assert np.array_equal(rel["k_cache"][:keep], tail["k_cache"][:keep])
    want = oracle.f64_to_bf16(_cplx_rotate(oracle.bf16_to_f64(tail["k_hat"]), slot - (cursor + np.arange(4)),
                                           D, theta))
    assert np.array_equal(rel["k_cache"][keep:], want)
    assert np.array_equal(rel["pos"][keep:], slot) and rel["cursor"] == cursor + 4


def test_placement_bookkeeping_and_rejections():
    kc, vc, q, k, v = _case(6, L=12, T=3, Hq=2, Hkv=1, D=8)
    pos, cursor, D, theta = np.arange(12) * 2, 30, 8, 1.0e7       # live: even positions
    ranges = np.array([[4, 7]])                                     # removes 4 and 6
    ok = oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, 0.3, placement="slot",
                                       tail_positions=[4, 5, 50])
    assert ok["cursor"] == 51 and list(ok["pos"][-3:]) == [4, 5, 50]
    for bad in ([4, 4, 5], [2, 5, 7], [-1, 5, 7], [4, 5]):
        for placement in ("slot", "relocate"):
            with pytest.raises(ValueError):
                oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, 0.3,
                                              placement=placement, tail_positions=bad)
    with pytest.raises(ValueError):
        oracle.relocate_keys(pos, kc, np.array([[0, 4, 100], [2, 3, 200]]), D, theta)   # overlapping sources
    with pytest.raises(ValueError):
        oracle.relocate_keys(pos, kc, np.array([[0, 1, 2]]), D, theta)                 # onto a live row
    # post-prefill ranges are given in the tail's final positions
    post = oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, 0.3,
                                         placement="slot", tail_positions=[4, 5, 50], post_ranges=[[50, 51]])
    assert list(post["pos"][-2:]) == [4, 5] and post["cursor"] == 51
    with pytest.raises(ValueError):
        oracle.attention_layer_update(pos, kc, vc, ranges, cursor, q, k, v, D, theta, 0.3, placement="slot",
                                      tail_positions=[4, 5, 50], post_ranges=[[30, 31]])


def test_paper_shaped_trace_is_consistent():
    """The seeded revision trace shaped like the paper's (records in 10K-position slots,
    replacements at fresh slots, framing removed after each tail) is self-consistent and the
    oracle carries it through every revision: removed ranges are whole live records, tail runs
    start at slot boundaries at or past the cursor, framing lies inside the tail, and the
    live-row count and cursor the trace states are the oracle's."""
    import synth
    tr = synth.make_paper_trace(seed=3, head=200, n_records=6, record_len=(40, 80), n_revisions=5,
                                m_range=(30, 60), index=202)
    pos = tr.positions.copy()
    assert np.all(np.diff(pos) > 0)
    assert sum(b - a for a, b in tr.intervals) == len(pos)
    D = 8
    kb = np.zeros((len(pos), 1, D), np.uint16)
    vb = np.zeros_like(kb)
    for rv in tr.revisions:
        assert len(pos) == rv.L_old
        live = set(pos.tolist())
        for a, b in rv.ranges:
            assert all(p in live for p in range(a, b))
        assert rv.runs[0][0] >= rv.cursor and all(a % tr.interval == 0 for a, _ in rv.runs)
        assert sum(b - a for a, b in rv.runs) == rv.T == rv.m + 11
        tail = np.concatenate([np.arange(a, b) for a, b in rv.runs])
        for a, b in rv.post:
            assert np.all(np.isin(np.arange(a, b), tail))
        q = np.zeros((rv.T, 1, D), np.uint16)
        ref = oracle.attention_layer_update(pos, kb, vb, rv.ranges, rv.cursor, q, q, q, D, 1e4, 1.0, live=pos,
                                            rows=np.zeros(0, np.int64), post_ranges=rv.post, placement="slot",
                                            tail_positions=tail)
        assert ref["cursor"] == rv.cursor_after
        assert len(ref["pos"]) == rv.L_old - int(np.sum(rv.ranges[:, 1] - rv.ranges[:, 0])) + rv.m
        pos, kb, vb = ref["pos"], ref["k_cache"], ref["v_cache"]
