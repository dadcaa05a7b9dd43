"""C-ABI tests that need no GPU: the library loads, exports every function the
header declares, and its host-side verification (Section 4.2: deletion ranges
are checked against the live spans before anything is removed) accepts and
rejects exactly what it should, leaving the metadata unchanged on error.

Device pointers below are host addresses that the host-only checks never
dereference.
"""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
import paper_2609_18935_amd as tu
from paper_2609_18935_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tailupdate.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        B_build = __import__("paper_2609_18935_amd.build", fromlist=["build"])
        B_build.build()
    return B.lib()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?(?:int|size_t|char\s*\*|const char\s*\*)\s*\*?\s*(\w+)\s*\(", text, re.M)
    return sorted(set(names))


def test_header_functions_are_exported(L):
    names = _declared_functions()
    assert {"compact_kv", "tail_prefill_attention", "delta_rule_continue", "update_layer_stack"} <= set(names)
    for n in names:
        assert hasattr(L, n), f"{n} declared in tailupdate.h but not exported"
    assert set(names) == set(B._SIGNATURES), "binding signatures out of sync with the header"
    import re
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "tailupdate.h")).read()
    declared = int(re.search(r"#define TU_ABI_VERSION (\d+)", hdr).group(1))
    assert L.tu_abi_version() == declared == B.ABI_VERSION


def _ctx(intervals, cursor, capacity=None, live_cap=64):
    n = sum(b - a for a, b in intervals)
    ctx = tu.Context(capacity if capacity is not None else n + 64, device="cpu", live_cap=live_cap)
    ctx.set_metadata(intervals, cursor)
    return ctx


def test_validate_ranges_matches_oracle(L):
    rng = np.random.default_rng(5)
    for trial in range(300):
        # random live set with holes, random candidate ranges (valid or not)
        cursor = int(rng.integers(10, 200))
        live = np.sort(rng.choice(cursor, size=int(rng.integers(1, cursor)), replace=False))
        ivs = []
        for p in live.tolist():
            if ivs and ivs[-1][1] == p:
                ivs[-1] = (ivs[-1][0], p + 1)
            else:
                ivs.append((p, p + 1))
        ctx = _ctx(ivs, cursor)
        n = int(rng.integers(0, 4))
        starts = np.sort(rng.integers(-2, cursor + 2, size=n))
        ranges = [(int(a), int(a + rng.integers(0, 6))) for a in starts]
        try:
            oracle.validate_ranges(ranges, live, cursor)
            expect_ok = True
        except oracle.RangeError:
            expect_ok = False
        before = (ctx.intervals(), ctx.len, ctx.next_pos)
        if expect_ok:
            assert ctx.validate_ranges(ranges) == sum(b - a for a, b in ranges)
        else:
            with pytest.raises(tu.TailUpdateError) as ei:
                ctx.validate_ranges(ranges)
            assert ei.value.code == B.TU_ERR_RANGE
        assert (ctx.intervals(), ctx.len, ctx.next_pos) == before


def _stack(ctx_list, ranges, tails, kinds, cap_ok=True, post=None):
    attn = tu.attn_params(16, 2, 256)
    delta = tu.delta_params(16, 32, 128, 128, 64)
    fake = torch.zeros(64, dtype=torch.float32)   # 16-byte aligned host buffer, never read
    layers = []
    for kind in kinds:
        if kind == "attn":
            layers.append(tu.LayerIO(B.TU_LAYER_ATTN, fake, fake, fake, fake,
                                     k_cache=[fake] * len(ctx_list), v_cache=[fake] * len(ctx_list)))
        else:
            layers.append(tu.LayerIO(B.TU_LAYER_DELTA, fake, fake, fake, fake, state=[fake] * len(ctx_list),
                                     beta=fake, g=fake))
    return tu.StackUpdate(ctx_list, ranges, tails, layers, attn, delta, post_ranges=post)


def test_validate_update_accepts_and_sizes(L):
    a = _ctx([(0, 1000)], 1000, capacity=2000)
    b = _ctx([(0, 10), (20, 500)], 600, capacity=1000)
    up = _stack([a, b], [[(100, 228)], [(30, 40), (300, 310)]], [512, 256], ["attn", "delta"])
    up.validate()
    assert up.workspace_size() > 0
    # an opening and a closing maintenance delimiter inside each tail
    up2 = _stack([a, b], [[(100, 228)], [(30, 40), (300, 310)]], [512, 256], ["attn", "delta"],
                 post=[[(1000, 1011), (1509, 1512)], [(600, 611)]])
    up2.validate()
    assert up2.workspace_size() >= up.workspace_size()


@pytest.mark.parametrize("case,code", [
    ("capacity", B.TU_ERR_CAPACITY),
    ("range_not_live", B.TU_ERR_RANGE),
    ("range_past_cursor", B.TU_ERR_RANGE),
    ("duplicate_context", B.TU_ERR_ARG),
    ("bad_heads", B.TU_ERR_ARG),
    ("interval_list_full", B.TU_ERR_CAPACITY),
    ("post_before_tail", B.TU_ERR_RANGE),
    ("post_past_tail", B.TU_ERR_RANGE),
    ("post_unsorted", B.TU_ERR_RANGE),
    ("post_empty_range", B.TU_ERR_RANGE),
])
def test_validate_update_rejects(L, case, code):
    a = _ctx([(0, 1000)], 1000, capacity=1600)
    ctxs, ranges, tails, kinds = [a], [[(100, 228)]], [512], ["attn", "delta"]
    if case == "capacity":
        tails = [800]
    elif case == "range_not_live":
        a.set_metadata([(0, 100), (200, 1100)], 1100)
        ranges = [[(90, 110)]]
    elif case == "range_past_cursor":
        ranges = [[(990, 1010)]]
    elif case == "duplicate_context":
        ctxs, ranges, tails = [a, a], [[], []], [1, 1]
    elif case == "interval_list_full":
        a = _ctx([(0, 1000)], 1000, capacity=1600, live_cap=2)
        ctxs = [a]
        ranges = [[(100, 110), (200, 210)]]
    post = None
    if case == "post_before_tail":
        post = [[(990, 1005)]]          # starts before the cursor
    elif case == "post_past_tail":
        post = [[(1500, 1513)]]         # the tail is [1000, 1512)
    elif case == "post_unsorted":
        post = [[(1100, 1110), (1000, 1011)]]
    elif case == "post_empty_range":
        post = [[(1000, 1000)]]
    up = _stack(ctxs, ranges, tails, kinds, post=post)
    if case == "bad_heads":
        up.u.attn.n_q_heads = 15
    before = (a.intervals(), a.len, a.next_pos)
    with pytest.raises(tu.TailUpdateError) as ei:
        up.validate()
    assert ei.value.code == code
    assert (a.intervals(), a.len, a.next_pos) == before
    assert L.update_layer_stack_workspace_size(ctypes.byref(up.u)) == 0


def test_entry_points_reject_before_touching_device(L):
    # invalid calls must fail in the host checks; no device memory is involved
    a = _ctx([(0, 100)], 100, capacity=120)
    fake = torch.zeros(64).view(-1, 1, 64)
    before = (a.intervals(), a.len)
    with pytest.raises(tu.TailUpdateError) as ei:   # range crosses the cursor
        tu.compact_kv(a, [fake], [fake], [(90, 101)], workspace=torch.zeros(1 << 16, dtype=torch.uint8))
    assert ei.value.code == B.TU_ERR_RANGE
    with pytest.raises(tu.TailUpdateError) as ei:   # too small a workspace
        tu.compact_kv(a, [fake], [fake], [(10, 20)],
                      workspace=torch.zeros(16, dtype=torch.uint8))
    assert ei.value.code == B.TU_ERR_WORKSPACE
    assert (a.intervals(), a.len) == before
    p = tu.attn_params(16, 2, 256)
    with pytest.raises(tu.TailUpdateError) as ei:   # capacity
        tu.tail_prefill_attention(a, fake, fake, p, torch.zeros(30, 16, 256, dtype=torch.bfloat16),
                                  fake, fake, fake, workspace=torch.zeros(256, dtype=torch.uint8))
    assert ei.value.code == B.TU_ERR_CAPACITY
    d = tu.delta_params(16, 32, 128, 128, 48)
    with pytest.raises(tu.TailUpdateError) as ei:   # unsupported chunk
        tu.delta_rule_continue(fake, torch.zeros(4, 16, 128, dtype=torch.bfloat16), fake, fake, fake, fake, d, fake,
                               workspace=torch.zeros(256, dtype=torch.uint8))
    assert ei.value.code == B.TU_ERR_ARG
    st = torch.zeros(3, 24, dtype=torch.bfloat16)
    xs = torch.zeros(5, 24, dtype=torch.bfloat16)
    x20 = torch.zeros(5, 20, dtype=torch.bfloat16)
    for args, what in [((st, x20, torch.zeros(20, 4, dtype=torch.bfloat16), x20), "channels % 8"),
                       ((torch.zeros(9, 24, dtype=torch.bfloat16), xs, torch.zeros(24, 10, dtype=torch.bfloat16), xs),
                        "width > 8"),
                       ((None, xs, torch.zeros(24, 4, dtype=torch.bfloat16), xs), "state missing")]:
        with pytest.raises(tu.TailUpdateError) as ei:
            tu.short_conv_continue(*args)
        assert ei.value.code == B.TU_ERR_ARG, what
    assert L.short_conv_continue(None, None, None, 4, 16, 4, 7, None, None) == B.TU_ERR_ARG   # unknown activation
    assert L.short_conv_continue(None, None, None, 0, 16, 4, 1, None, None) == 0   # T == 0: nothing to do


def test_commit_tail_advances_cursor_and_intervals(L):
    a = _ctx([(0, 10), (20, 30)], 40, capacity=100)
    tu.commit_tail(a, 5)
    assert a.intervals() == [(0, 10), (20, 30), (40, 45)] and a.len == 25 and a.next_pos == 45
    tu.commit_tail(a, 3)
    assert a.intervals() == [(0, 10), (20, 30), (40, 48)] and a.next_pos == 48
    with pytest.raises(tu.TailUpdateError):
        tu.commit_tail(a, 1000)


def _runs_of(positions):
    """Maximal runs of consecutive positions, in the given (row) order."""
    out = []
    for p in positions:
        if out and out[-1][1] == p:
            out[-1] = (out[-1][0], p + 1)
        else:
            out.append((p, p + 1))
    return out


def test_live_runs_in_row_order(L):
    # rows hold positions in work order: slot-placed rows carry earlier positions
    rng = np.random.default_rng(8)
    for trial in range(200):
        cursor = int(rng.integers(20, 300))
        live = rng.choice(cursor, size=int(rng.integers(1, cursor)), replace=False)
        order = np.sort(live)
        # cut the sorted positions into blocks and shuffle the blocks (row order)
        cuts = np.sort(rng.choice(np.arange(1, len(order)), size=min(len(order) - 1, int(rng.integers(0, 5))),
                              replace=False)) if len(order) > 1 else []
        blocks = np.split(order, cuts)
        rng.shuffle(blocks)
        rows = np.concatenate(blocks)
        ctx = _ctx(_runs_of(rows.tolist()), cursor, live_cap=512)
        n = int(rng.integers(0, 4))
        starts = np.sort(rng.integers(0, cursor, size=n))
        ranges = [(int(a), int(a + rng.integers(1, 6))) for a in starts]
        try:
            oracle.validate_ranges(ranges, rows, cursor)
            expect_ok = True
        except oracle.RangeError:
            expect_ok = False
        if expect_ok:
            assert ctx.validate_ranges(ranges) == sum(b - a for a, b in ranges)
        else:
            with pytest.raises(tu.TailUpdateError):
                ctx.validate_ranges(ranges)
    # a run list that is not well formed is rejected
    for ivs, cursor in [([(0, 5), (5, 9)], 10),      # consecutive runs not merged
                        ([(0, 5), (3, 9)], 10),      # overlapping runs
                        ([(6, 9), (0, 3), (2, 4)], 10),
                        ([(0, 5)], 4)]:              # beyond the cursor
        ctx = _ctx([(0, 1)], 10)
        ctx.set_metadata(ivs, cursor)
        with pytest.raises(tu.TailUpdateError) as ei:
            ctx.validate_ranges([])
        assert ei.value.code == B.TU_ERR_ARG
    # non-adjacent rows may hold adjacent positions: one range covering both is two row spans
    ctx = _ctx([(0, 10), (50, 60), (10, 20)], 70)
    assert ctx.validate_ranges([(5, 15)]) == 10


def _placed(placement, runs, post=None, T=512, ranges=((100, 228),)):
    a = _ctx([(0, 1000)], 1000, capacity=1600)
    attn = tu.attn_params(16, 2, 256)
    fake = torch.zeros(64, dtype=torch.float32)
    layers = [tu.LayerIO(B.TU_LAYER_ATTN, fake, fake, fake, fake, k_cache=[fake], v_cache=[fake])]
    return a, tu.StackUpdate([a], [list(ranges)], [T], layers, attn, None, post_ranges=post,
                             placement=[placement], place_runs=[runs])


def test_validate_placements(L):
    # slot-preserving: the replacement takes the removed record's slot plus a free range
    for placement in ("slot", "relocate"):
        a, up = _placed(placement, [(100, 228), (5000, 5384)])
        up.validate()
        assert up.workspace_size() > 0
        a, up = _placed(placement, [(100, 228), (5000, 5384)], post=[[(100, 111), (5381, 5384)]])
        up.validate()
    bad = [
        ("slot", [(100, 229), (5000, 5383)], B.TU_ERR_RANGE),      # 228 is still live
        ("slot", [(100, 228), (5000, 5383)], B.TU_ERR_ARG),        # 511 positions for 512 tokens
        ("relocate", [(100, 228), (150, 534)], B.TU_ERR_RANGE),    # runs overlap each other
        ("slot", [(-4, 508)], B.TU_ERR_RANGE),
        ("slot", [(2 ** 31 - 100, 2 ** 31 + 412)], B.TU_ERR_RANGE),
        ("slot", [(10000 + 16 * i, 10016 + 16 * i) for i in range(32)] + [(9000, 9000)], B.TU_ERR_ARG),  # > 32 runs
        ("tail", [(5000, 5512)], B.TU_ERR_ARG),                    # runs with a true-tail update
    ]
    for placement, runs, code in bad:
        a, up = _placed(placement, runs)
        before = (a.intervals(), a.len, a.next_pos)
        with pytest.raises(tu.TailUpdateError) as ei:
            up.validate()
        assert ei.value.code == code, (placement, runs)
        assert (a.intervals(), a.len, a.next_pos) == before
    # post-prefill ranges must be made of the tail's final positions
    a, up = _placed("slot", [(100, 228), (5000, 5384)], post=[[(1000, 1011)]])
    with pytest.raises(tu.TailUpdateError) as ei:
        up.validate()
    assert ei.value.code == B.TU_ERR_RANGE
    a, up = _placed("slot", [(100, 228), (5000, 5384)], post=[[(90, 105)]])   # starts in surviving rows
    with pytest.raises(tu.TailUpdateError) as ei:
        up.validate()
    assert ei.value.code == B.TU_ERR_RANGE
    a, up = _placed("tail", None)
    up.u.seqs[0].placement = 7
    with pytest.raises(tu.TailUpdateError) as ei:
        up.validate()
    assert ei.value.code == B.TU_ERR_ARG


def test_relocate_keys_rejects_before_touching_device(L):
    a = _ctx([(0, 100), (200, 300)], 400, capacity=256)
    p = tu.attn_params(16, 2, 256)
    fake = torch.zeros(64, dtype=torch.float32)
    before = (a.intervals(), a.len, a.next_pos)
    for moves in ([(50, 150, 1000)],             # source not live
                  [(50, 60, 95)],                # destination hits a row that stays
                  [(50, 60, 1000), (55, 65, 2000)],   # overlapping sources
                  [(60, 70, 1000), (50, 55, 2000)],   # unsorted sources
                  [(50, 60, 1000), (250, 260, 1005)],  # destinations overlap each other
                  [(50, 60, -3)], [(50, 60, 2 ** 31 - 5)], [(60, 50, 1000)]):
        with pytest.raises(tu.TailUpdateError) as ei:
            tu.relocate_keys(a, [fake], p, moves)
        assert ei.value.code == B.TU_ERR_RANGE, moves
        assert (a.intervals(), a.len, a.next_pos) == before
    with pytest.raises(tu.TailUpdateError) as ei:
        tu.relocate_keys(a, [fake], tu.attn_params(15, 2, 256), [(50, 60, 1000)])
    assert ei.value.code == B.TU_ERR_ARG
    # a move onto its own positions changes nothing and launches nothing
    tu.relocate_keys(a, [fake], p, [(50, 60, 50)])
    assert (a.intervals(), a.len, a.next_pos) == before


def test_diagnostics_reject_before_touching_device(L):
    a = _ctx([(0, 100), (200, 300)], 400, capacity=256)
    p = tu.attn_params(16, 2, 256)
    fake = torch.zeros(64, dtype=torch.float32)
    q = torch.zeros(8, 16, 256, dtype=torch.bfloat16)
    ws = torch.zeros(1 << 20, dtype=torch.uint8)
    for n, code in [(0, B.TU_ERR_ARG), (201, B.TU_ERR_ARG), (17, B.TU_ERR_ARG)]:   # 17 x 8 rows > 128
        qq = torch.zeros(max(n, 1), 16, 256, dtype=torch.bfloat16)
        rc = L.attention_probe(ctypes.byref(a.c), fake.data_ptr(), ctypes.byref(p), qq.data_ptr(), n, 1.0,
                               fake.data_ptr(), ws.data_ptr(), ws.numel(), None)
        assert rc == code, n
    with pytest.raises(tu.TailUpdateError) as ei:   # workspace too small
        tu.attention_probe(a, fake, p, q, fake, workspace=torch.zeros(256, dtype=torch.uint8))
    assert ei.value.code == B.TU_ERR_WORKSPACE
    for groups in ([(10, 20), (15, 30)], [(30, 40), (10, 20)], [(5, 5)], [(-1, 4)]):
        with pytest.raises(tu.TailUpdateError) as ei:
            tu.attention_group_mass(a, fake, groups, workspace=ws)
        assert ei.value.code == B.TU_ERR_RANGE, groups
    assert L.attention_tv_distance(None, None, None, -1, None, None, 0, None) == B.TU_ERR_ARG
    assert L.attention_tv_distance(fake.data_ptr(), fake.data_ptr(), None, 10, fake.data_ptr(), None, 0,
                                   None) == B.TU_ERR_WORKSPACE


def test_workspace_faults_rejects_null_and_matches_header(L):
    """tu_workspace_faults refuses a null workspace or output before any device access;
    the fault bits of the binding are the header's."""
    out = ctypes.c_int32(0)
    assert L.tu_workspace_faults(None, ctypes.byref(out), None) == B.TU_ERR_ARG
    assert L.tu_workspace_faults(ctypes.c_void_p(16), None, None) == B.TU_ERR_ARG
    assert "faults" in L.tu_last_error().decode()
    hdr = open(HEADER).read()
    assert int(re.search(r"#define TU_FAULT_POSITIONS (\d+)", hdr).group(1)) == tu.TU_FAULT_POSITIONS
    assert int(re.search(r"#define TU_FAULT_WAIT (\d+)", hdr).group(1)) == tu.TU_FAULT_WAIT
    assert int(re.search(r"#define TU_FAULT_RANGE (\d+)", hdr).group(1)) == tu.TU_FAULT_RANGE


def test_new_workspace_is_recorded_on_the_call_stream(monkeypatch):
    """A workspace the binding allocates for a call on another stream than the current
    one is recorded on that stream (the caching allocator must not reuse it while the
    call's kernels run); one for the current stream, or a caller's workspace, is not."""
    recorded = []

    class FakeTensor:
        def record_stream(self, st):
            recorded.append(st)

    class FakeStream:
        def __init__(self, name):
            self.name = name

        def __eq__(self, other):
            return isinstance(other, FakeStream) and other.name == self.name

    current = FakeStream("current")
    monkeypatch.setattr(B.torch, "empty", lambda *a, **k: FakeTensor())
    monkeypatch.setattr(B.torch.cuda, "Stream", FakeStream)
    monkeypatch.setattr(B.torch.cuda, "current_stream", lambda device=None: current)
    side = FakeStream("side")
    B._workspace(1024, "cuda", None, side)
    assert recorded == [side]
    B._workspace(1024, "cuda", None, current)
    B._workspace(1024, "cuda", None, None)
    mine = FakeTensor()
    assert B._workspace(1024, "cuda", mine, side) is mine
    assert recorded == [side]


def test_vt_cache_bytes(L):
    """The V^T copy holds Hkv x ceil(capacity / 64) tiles of D rows x 72 f16 (64 keys plus
    a 16-byte pad); invalid shapes give 0."""
    assert L.tu_vt_cache_bytes(8192, 2, 256) == 2 * (8192 // 64) * 256 * 72 * 2
    assert L.tu_vt_cache_bytes(65, 1, 64) == 1 * 2 * 64 * 72 * 2
    assert L.tu_vt_cache_bytes(0, 2, 256) == 0
    assert L.tu_vt_cache_bytes(100, 2, 96) == 0
    assert L.tu_vt_cache_bytes(-1, 2, 256) == 0
