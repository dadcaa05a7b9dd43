"""The allocation-free compaction (compact_kv_noalloc) against compact_kv (MI355X only).

Callers that cannot allocate (graph capture, serving loops) get compact_kv with its
scratch in a fixed per-GPU array. Its results must equal compact_kv's bit for bit: the
moved K/V rows of every layer, the positions, the index list and the metadata, on two
calls in a row (the array keeps the first call's contents), the second smaller and
with the index list left in the scratch; its device checks must reach the caller's
status block; a call whose scratch would exceed the array is refused before anything
runs, with the context untouched.
"""
import numpy as np
import pytest
import torch

import paper_2609_18935_amd as tu
from gpu_cases import DEV

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _pair(L, Hkv, D, n_layers, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    ks = [torch.randn(L, Hkv, D, generator=g, device=DEV).to(torch.bfloat16) for _ in range(n_layers)]
    vs = [torch.randn(L, Hkv, D, generator=g, device=DEV).to(torch.bfloat16) for _ in range(n_layers)]
    return ks, vs


def _ctx(L):
    ctx = tu.Context(L, device=DEV)
    ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
    ctx.set_metadata([(0, L)], L)
    return ctx


@pytest.mark.parametrize("call", [
    # (rows, kv heads, head dim, layers, removed ranges, pass an index list)
    [(20000, 2, 256, 3, [(100, 900), (5000, 5001), (19000, 20000)], True),
     (3000, 1, 64, 1, [(0, 10), (2500, 2600)], False)],
])
def test_noalloc_equals_compact_kv(call):
    for i, (L, Hkv, D, n_layers, ranges, with_index) in enumerate(call):
        print(f"[case] call {i}: L={L} Hkv={Hkv} D={D} layers={n_layers} ranges={ranges} index={with_index}",
              flush=True)
        ranges = np.asarray(ranges, dtype=np.int64)
        ks, vs = _pair(L, Hkv, D, n_layers, seed=100 + i)
        ks2, vs2 = [k.clone() for k in ks], [v.clone() for v in vs]
        ctx, ctx2 = _ctx(L), _ctx(L)
        src = torch.full((L,), -1, dtype=torch.int32, device=DEV)
        src2 = torch.full((L,), -1, dtype=torch.int32, device=DEV) if with_index else None
        status = torch.full((256,), 0xFF, dtype=torch.uint8, device=DEV)   # stale bytes
        tu.compact_kv(ctx, ks, vs, ranges, src_index=src)
        tu.compact_kv_noalloc(ctx2, ks2, vs2, ranges, src_index=src2, status=status)
        torch.cuda.synchronize()
        n = ctx.len
        assert (ctx2.len, ctx2.next_pos, ctx2.intervals(), ctx2.vt_rows) == (n, ctx.next_pos, ctx.intervals(),
                                                                              ctx.vt_rows)
        assert torch.equal(ctx2.pos[:n], ctx.pos[:n])
        for l in range(n_layers):
            assert torch.equal(ks2[l][:n], ks[l][:n]), f"call {i} layer {l}: K"
            assert torch.equal(vs2[l][:n], vs[l][:n]), f"call {i} layer {l}: V"
        if with_index:
            assert torch.equal(src2[:n], src[:n])
        assert tu.workspace_faults(status) == 0


def test_noalloc_reports_device_checks_and_refuses_oversized_calls():
    L = 4096
    print(f"[case] mislabelled row, then an oversized call: L={L}", flush=True)
    ks, vs = _pair(L, 2, 64, 1, seed=7)
    ctx = _ctx(L)
    ctx.pos[1000] = 5000                     # the device label disagrees with the host's runs
    status = torch.zeros(256, dtype=torch.uint8, device=DEV)
    tu.compact_kv_noalloc(ctx, ks, vs, np.array([[900, 1100]]), status=status)
    assert tu.workspace_faults(status) == tu.TU_FAULT_POSITIONS
    # a context too long for the fixed scratch: refused before any launch, nothing changed
    big = 3_000_000
    ctx = tu.Context(big, device=DEV)
    ctx.set_metadata([(0, big)], big)
    k1 = torch.zeros(1, 2, 64, dtype=torch.bfloat16, device=DEV)   # never read: the call is refused first
    before = (ctx.len, ctx.intervals(), ctx.next_pos)
    with pytest.raises(tu.TailUpdateError) as ei:
        tu.compact_kv_noalloc(ctx, [k1], [k1], np.array([[10, 20]]))
    assert ei.value.code == -4 and "fixed scratch" in str(ei.value)
    assert (ctx.len, ctx.intervals(), ctx.next_pos) == before
