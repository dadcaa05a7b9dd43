"""GPU parity of degenerate stack updates through the C ABI (MI355X only).

One update_layer_stack call over four contexts at once, each a degenerate case:
  * removals and no tail (pure deletion: caches compacted, recurrent state and
    cursor unchanged, no output rows);
  * every live row removed, then a tail (attention over the tail only);
  * a tail and no removals (ordinary continuation);
  * an empty context (fresh prefill from position 0).
Each context is checked against the float64 oracle on its own.

Also the device-side check of the compaction: position labels that disagree with
the host's live runs set the device's sticky fault word, which the host reads and
clears; correct updates leave it clear.
"""
import numpy as np
import pytest
import torch

import synth
import paper_2609_18935_amd as tu
from gpu_cases import (AttnCase, DeltaCase, DEV, assert_bf16_close_bits, assert_close, bits_of, to_dev_bf16)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _ctx_for(case):
    ctx = tu.Context(max(case.capacity, 1), device=DEV)
    if case.L_old:
        ctx.pos[: case.L_old] = torch.from_numpy(case.positions.astype(np.int32)).to(DEV)
    ctx.set_metadata([(0, case.L_old)] if case.L_old else [], case.L_old)
    return ctx


def test_degenerate_contexts_in_one_call():
    a = synth.AttnShape(16, 2, 256)
    d = synth.DeltaShape(16, 32, 128, 128, 64)
    specs = [  # (L_old, ranges, T)
        (1500, np.array([[100, 300], [1400, 1500]]), 0),
        (700, np.array([[0, 700]]), 90),
        (1200, np.zeros((0, 2), np.int64), 33),
        (0, np.zeros((0, 2), np.int64), 65),
    ]
    print(f"[case] four contexts: {[(L, r.tolist(), T) for L, r, T in specs]}", flush=True)
    acs = [AttnCase(a, 40, 1, 0, L, T, char=c) for c, (L, _, T) in enumerate(specs)]
    dcs = [DeltaCase(d, 40, 1, 1, T, char=c) for c, (_, _, T) in enumerate(specs)]
    ctxs = [_ctx_for(ac) for ac in acs]
    Ts = [T for _, _, T in specs]
    off = np.concatenate([[0], np.cumsum(Ts)])
    cat = lambda xs: to_dev_bf16(np.concatenate(xs))
    a_out = torch.full((int(off[-1]), a.n_q_heads, a.head_dim), float("nan"), dtype=torch.float32, device=DEV)
    d_out = torch.full((int(off[-1]), d.n_v_heads, d.d_v), float("nan"), dtype=torch.float32, device=DEV)
    srcs = [torch.full((max(1, L),), -1, dtype=torch.int32, device=DEV) for L, _, _ in specs]
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, cat([c.q_t for c in acs]), cat([c.k_t for c in acs]),
                         cat([c.v_t for c in acs]), a_out, k_cache=[c.k_cache for c in acs],
                         v_cache=[c.v_cache for c in acs]),
              tu.LayerIO(tu.TU_LAYER_DELTA, cat([c.q_b for c in dcs]), cat([c.k_b for c in dcs]),
                         cat([c.v_b for c in dcs]), d_out, state=[c.state for c in dcs],
                         beta=torch.from_numpy(np.concatenate([c.beta for c in dcs])).to(DEV),
                         g=torch.from_numpy(np.concatenate([c.g for c in dcs])).to(DEV))]
    up = tu.update_layer_stack(ctxs, [r for _, r, _ in specs], Ts, layers,
                               tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta),
                               tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk), src_index=srcs)
    torch.cuda.synchronize()
    for c, ((L, ranges, T), ac, dc, ctx) in enumerate(zip(specs, acs, dcs, ctxs)):
        ref = ac.oracle(ranges, L)
        n = len(ref["pos"])
        what = f"context {c} (L_old {L}, removed {int(np.sum(ranges[:, 1] - ranges[:, 0]))}, T {T})"
        assert ctx.len == n and ctx.next_pos == L + T, what
        assert np.array_equal(srcs[c][: ref["L_keep"]].cpu().numpy(), ref["src_index"]), what
        assert np.array_equal(ctx.pos[:n].cpu().numpy(), ref["pos"]), what
        assert np.array_equal(bits_of(ac.v_cache[:n]), ref["v_cache"]), what
        assert_bf16_close_bits(bits_of(ac.k_cache[:n]), ref["k_cache"], f"{what}: K cache")
        runs = synth.append_interval(synth.subtract_ranges([(0, L)] if L else [], ranges), L, T)
        assert ctx.intervals() == runs, what
        o_ref, S_ref = dc.oracle()
        if T == 0:
            assert np.array_equal(dc.state.cpu().numpy(), dc.S0), f"{what}: state must not change"
            continue
        assert_close(a_out[int(off[c]): int(off[c + 1])].cpu().numpy(), ref["out"], f"{what}: attention")
        assert_close(d_out[int(off[c]): int(off[c + 1])].cpu().numpy(), o_ref, f"{what}: delta out")
        assert_close(dc.state.cpu().numpy(), S_ref, f"{what}: delta state")
    assert tu.workspace_faults(up.workspace) == 0, "an update of consistent contexts raised a device fault"


def test_device_fault_on_mislabelled_positions():
    """The host says rows 0..4095 hold positions 0..4095; the device labels row 1000 with
    5000 instead. Removing positions [900, 1100) removes rows 900..1099 by the host's
    spans, but the row labelled 5000 lies in no range: the scan flags the disagreement
    in the call's status word. The move still follows the host's spans (every access in
    bounds). A second call on a workspace whose status word holds stale bits (and
    another workspace untouched meanwhile) starts from a clear word."""
    L = 4096
    _say = lambda m: print(f"[case] {m}", flush=True)
    _say("mislabelled row 1000 of 4096, remove [900, 1100)")
    k = torch.randn(L, 2, 64, device=DEV).to(torch.bfloat16)
    v = torch.randn_like(k)
    k0, v0 = k.clone(), v.clone()
    ctx = tu.Context(L, device=DEV)
    labels = torch.arange(L, dtype=torch.int32, device=DEV)
    labels[1000] = 5000
    ctx.pos[:L] = labels
    ctx.set_metadata([(0, L)], L)
    nbytes = tu.lib().compact_kv_workspace_size(L, 1, 2, 64)
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device=DEV)   # stale bits everywhere
    other = torch.zeros_like(ws)
    tu.compact_kv(ctx, [k], [v], np.array([[900, 1100]]), workspace=ws)
    assert tu.workspace_faults(ws) == tu.TU_FAULT_POSITIONS
    assert tu.workspace_faults(other) == 0      # another workspace is never touched
    keep = torch.cat([torch.arange(900), torch.arange(1100, L)]).to(DEV)
    assert ctx.len == L - 200
    assert torch.equal(k[: L - 200], k0[keep]) and torch.equal(v[: L - 200], v0[keep])
    assert torch.equal(ctx.pos[: L - 200], labels[keep])
    # the same removal with consistent labels raises nothing, on the same workspace
    k, v = k0.clone(), v0.clone()
    ctx = tu.Context(L, device=DEV)
    ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
    ctx.set_metadata([(0, L)], L)
    tu.compact_kv(ctx, [k], [v], np.array([[900, 1100]]), workspace=ws)
    assert tu.workspace_faults(ws) == 0
    assert torch.equal(k[: L - 200], k0[keep])


def test_all_tails_empty():
    """Pure deletion in every context of a call: caches compacted, states, outputs and
    cursors untouched, no attention or delta launch needed."""
    a = synth.AttnShape(16, 2, 256)
    d = synth.DeltaShape(16, 32, 128, 128, 64)
    specs = [(2000, np.array([[10, 50], [1900, 2000]])), (900, np.array([[0, 300]]))]
    print(f"[case] all tails empty: {[(L, r.tolist()) for L, r in specs]}", flush=True)
    acs = [AttnCase(a, 41, 1, 0, L, 0, char=c) for c, (L, _) in enumerate(specs)]
    dcs = [DeltaCase(d, 41, 1, 1, 0, char=c) for c in range(len(specs))]
    ctxs = [_ctx_for(ac) for ac in acs]
    empty = lambda *s: torch.empty(s, dtype=torch.bfloat16, device=DEV)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, empty(0, 16, 256), empty(0, 2, 256), empty(0, 2, 256),
                         torch.empty((0, 16, 256), dtype=torch.float32, device=DEV),
                         k_cache=[c.k_cache for c in acs], v_cache=[c.v_cache for c in acs]),
              tu.LayerIO(tu.TU_LAYER_DELTA, empty(0, 16, 128), empty(0, 16, 128), empty(0, 32, 128),
                         torch.empty((0, 32, 128), dtype=torch.float32, device=DEV), state=[c.state for c in dcs],
                         beta=torch.empty((0, 32), dtype=torch.float32, device=DEV),
                         g=torch.empty((0, 32), dtype=torch.float32, device=DEV))]
    up = tu.update_layer_stack(ctxs, [r for _, r in specs], [0, 0], layers,
                               tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta),
                               tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk))
    torch.cuda.synchronize()
    for (L, ranges), ac, dc, ctx in zip(specs, acs, dcs, ctxs):
        ref = ac.oracle(ranges, L)
        n = len(ref["pos"])
        assert ctx.len == n and ctx.next_pos == L
        assert np.array_equal(ctx.pos[:n].cpu().numpy(), ref["pos"])
        assert np.array_equal(bits_of(ac.v_cache[:n]), ref["v_cache"])
        assert np.array_equal(bits_of(ac.k_cache[:n]), ref["k_cache"])
        assert np.array_equal(dc.state.cpu().numpy(), dc.S0)
    assert tu.workspace_faults(up.workspace) == 0
