"""GPU tests of the persistent V^T copy and of the f16 range guard (MI355X only).

V^T copy: an update that refreshes each attention layer's V^T copy from the first row
that moved must give exactly the results of an update that packs every row into the
workspace (the same f16 tiles reach the attention kernel), across removals early and
late in the cache, delimiter rows removed after the prefill, an update without
removals, and the standalone compact / prefill / commit calls; both are checked
against the float64 oracle chained over the rounds.

Range: the attention values and several delta-rule operands are rounded to f16. Values
up to the largest bf16 below 2^16 must still match the oracle (the bar scales with the
inputs' magnitude); larger ones set TU_FAULT_RANGE in the call's status word. Strong
decay (g = 1e-3) and gates of exactly 0 must stay finite and match the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import DEV, DeltaCase, assert_bf16_close_bits, assert_close, bits_of, errors, to_dev_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _say(msg):
    print(f"[case] {msg}", flush=True)


A = synth.AttnShape(16, 2, 256)


def _ap():
    return tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta, A.softmax_scale)


def _ctx(L, cap):
    ctx = tu.Context(cap, device=DEV)
    ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
    ctx.set_metadata([(0, L)] if L else [], L)
    return ctx


# rounds: (removal ranges, tail length, post-prefill ranges relative to the cursor)
ROUNDS = [
    (np.array([[1000, 1200]]), 130, None),
    (np.array([[2900, 2950]]), 70, np.array([[0, 5]])),
    (np.zeros((0, 2), np.int64), 64, None),
    (np.array([[5, 40], [3100, 3120]]), 1, None),
]


def test_vt_copy_matches_workspace_path_over_rounds():
    L0, n_layers = 3000, 2
    cap = L0 + sum(T for _, T, _ in ROUNDS)
    _say(f"V^T copies vs workspace packing: L0={L0}, {n_layers} attention layers, rounds "
         f"{[(r.tolist(), T) for r, T, _ in ROUNDS]}")
    host = [synth.gen_attn_cache(11, 1, l, L0, A) for l in range(n_layers)]
    caches = {}
    for arm in ("copy", "workspace"):
        kv = []
        for kb, vb in host:
            kc = np.zeros((cap, A.n_kv_heads, A.head_dim), np.uint16)
            vc = np.zeros_like(kc)
            kc[:L0], vc[:L0] = kb, vb
            kv.append((to_dev_bf16(kc), to_dev_bf16(vc)))
        caches[arm] = kv
    ctxs = {"copy": _ctx(L0, cap), "workspace": _ctx(L0, cap)}
    vts = [tu.new_vt_cache(cap, A.n_kv_heads, A.head_dim, DEV) for _ in range(n_layers)]
    ws = tu.refresh_vt_cache(ctxs["copy"], [v for _, v in caches["copy"]], vts)
    assert tu.workspace_faults(ws) == 0 and ctxs["copy"].vt_rows == L0
    # oracle state, chained over the rounds
    pos = np.arange(L0)
    kbs = [kb for kb, _ in host]
    vbs = [vb for _, vb in host]
    for ri, (ranges, T, post_rel) in enumerate(ROUNDS):
        cursor = ctxs["copy"].next_pos
        post = None if post_rel is None else post_rel + cursor
        tails = [synth.gen_attn_tail(11, 1, l, T, A, rnd=ri) for l in range(n_layers)]
        outs = {}
        for arm in ("copy", "workspace"):
            layers = []
            outs[arm] = []
            for l, (q, k, v) in enumerate(tails):
                o = torch.full((T, A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
                outs[arm].append(o)
                layers.append(tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), o,
                                         k_cache=[caches[arm][l][0]], v_cache=[caches[arm][l][1]],
                                         vt_cache=[vts[l]] if arm == "copy" else None))
            up = tu.update_layer_stack([ctxs[arm]], [ranges], [T], layers, _ap(),
                                       post_ranges=None if post is None else [post])
            torch.cuda.synchronize()
            assert tu.workspace_faults(up.workspace) == 0, f"round {ri} {arm}: device check"
        c, w = ctxs["copy"], ctxs["workspace"]
        assert (c.len, c.next_pos, c.intervals()) == (w.len, w.next_pos, w.intervals()), f"round {ri}: metadata"
        # the copies are current up to the tail's end, or up to the first delimiter row the
        # post-prefill removal moved
        want_vt = c.len
        if post is not None:
            removed_post = int(np.sum(post_rel[:, 1] - post_rel[:, 0]))
            want_vt = c.len - T + removed_post + int(post_rel[0][0])
        assert c.vt_rows == want_vt, f"round {ri}: vt_rows {c.vt_rows}, expected {want_vt}"
        n = c.len
        assert torch.equal(c.pos[:n], w.pos[:n])
        for l in range(n_layers):
            assert torch.equal(outs["copy"][l], outs["workspace"][l]), f"round {ri} layer {l}: outputs differ"
            assert torch.equal(caches["copy"][l][0][:n], caches["workspace"][l][0][:n])
            assert torch.equal(caches["copy"][l][1][:n], caches["workspace"][l][1][:n])
            q, k, v = tails[l]
            ref = oracle.attention_layer_update(pos, kbs[l], vbs[l], ranges, cursor, q, k, v, A.rdim, A.rope_theta,
                                                A.softmax_scale, live=pos, post_ranges=post)
            assert np.array_equal(c.pos[:n].cpu().numpy(), ref["pos"])
            assert_bf16_close_bits(bits_of(caches["copy"][l][0][:n]), ref["k_cache"], f"round {ri} layer {l}: K")
            assert np.array_equal(bits_of(caches["copy"][l][1][:n]), ref["v_cache"])
            assert_close(outs["copy"][l].cpu().numpy(), ref["out"], f"round {ri} layer {l}: attention")
            kbs[l], vbs[l] = ref["k_cache"], ref["v_cache"]
        pos = ref["pos"]


def test_vt_copy_standalone_calls():
    """compact_kv lowers vt_rows to the first removed row, tail_prefill_attention with a
    copy refreshes from there, commit_tail raises vt_rows to len; the result equals the
    workspace-packed call bit for bit."""
    L0, T = 2500, 200
    ranges = np.array([[700, 900]])
    _say(f"standalone V^T copy: L0={L0} ranges={ranges.tolist()} T={T}")
    kb, vb = synth.gen_attn_cache(12, 1, 0, L0, A)
    q, k, v = synth.gen_attn_tail(12, 1, 0, T, A)
    outs = []
    for use_copy in (True, False):
        kc = np.zeros((L0 + T, A.n_kv_heads, A.head_dim), np.uint16)
        vc = np.zeros_like(kc)
        kc[:L0], vc[:L0] = kb, vb
        kd, vd = to_dev_bf16(kc), to_dev_bf16(vc)
        ctx = _ctx(L0, L0 + T)
        vt = None
        if use_copy:
            vt = tu.new_vt_cache(L0 + T, A.n_kv_heads, A.head_dim, DEV)
            tu.refresh_vt_cache(ctx, [vd], [vt])
        ws = tu.compact_kv(ctx, [kd], [vd], ranges)
        assert tu.workspace_faults(ws) == 0
        if use_copy:
            assert ctx.vt_rows == 700
        o = torch.full((T, A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
        ws = tu.tail_prefill_attention(ctx, kd, vd, _ap(), to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), o,
                                       vt_cache=vt)
        assert tu.workspace_faults(ws) == 0
        tu.commit_tail(ctx, T)
        assert ctx.vt_rows == ctx.len == L0 - 200 + T
        torch.cuda.synchronize()
        outs.append(o)
    assert torch.equal(outs[0], outs[1])
    ref = oracle.attention_layer_update(np.arange(L0), kb, vb, ranges, L0, q, k, v, A.rdim, A.rope_theta,
                                        A.softmax_scale)
    assert_close(outs[0].cpu().numpy(), ref["out"], "standalone V^T copy: attention")


# ----------------------------------------------------------------------------- f16 range

def _scaled_bf16(x):
    """float64 -> bf16 bits (nearest even via float32), for inputs of any magnitude."""
    return synth.to_bf16_bits(np.asarray(x, np.float64))


BF16_BELOW_2_16 = 65280.0   # the largest bf16 value below 2^16 (f16's largest finite is 65504)


@pytest.mark.parametrize("scale", [1.0e4, 6.0e4])
def test_attention_large_values_within_f16(scale):
    """Values of magnitude up to 65,280 (clipped N(0, scale^2)) match the oracle; the bar is
    relative to the outputs' magnitude (mean-rel 1e-3, max-abs 2e-2 of max |ref|)."""
    L0, T = 1500, 96
    ranges = np.array([[200, 260]])
    _say(f"attention with |v| up to {min(4 * scale, BF16_BELOW_2_16):.0f}: L0={L0} T={T}")
    rng = np.random.default_rng(31)
    kb, _ = synth.gen_attn_cache(13, 1, 0, L0, A)
    q, k, _ = synth.gen_attn_tail(13, 1, 0, T, A)
    vb = _scaled_bf16(np.clip(rng.standard_normal((L0, A.n_kv_heads, A.head_dim)) * scale, -BF16_BELOW_2_16,
                              BF16_BELOW_2_16))
    v = _scaled_bf16(np.clip(rng.standard_normal((T, A.n_kv_heads, A.head_dim)) * scale, -BF16_BELOW_2_16,
                             BF16_BELOW_2_16))
    kc = np.zeros((L0 + T, A.n_kv_heads, A.head_dim), np.uint16)
    vc = np.zeros_like(kc)
    kc[:L0], vc[:L0] = kb, vb
    kd, vd = to_dev_bf16(kc), to_dev_bf16(vc)
    ctx = _ctx(L0, L0 + T)
    o = torch.empty((T, A.n_q_heads, A.head_dim), dtype=torch.float32, device=DEV)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), o, k_cache=[kd],
                         v_cache=[vd])]
    up = tu.update_layer_stack([ctx], [ranges], [T], layers, _ap())
    torch.cuda.synchronize()
    assert tu.workspace_faults(up.workspace) == 0
    ref = oracle.attention_layer_update(np.arange(L0), kb, vb, ranges, L0, q, k, v, A.rdim, A.rope_theta,
                                        A.softmax_scale)
    got = o.cpu().numpy()
    assert np.all(np.isfinite(got))
    ma, mr = errors(got, ref["out"])
    top = float(np.abs(ref["out"]).max())
    print(f"[parity] |v| scale {scale:g}: max_abs={ma:.3e} (of max |ref| {top:.3e}) mean_rel={mr:.3e}", flush=True)
    assert mr <= 1e-3 and ma <= 2e-2 * top


@pytest.mark.parametrize("where", ["cache", "tail"])
def test_attention_values_beyond_f16_are_flagged(where):
    """A value of magnitude 1e5 in a surviving cache row, or in the tail, has no f16
    counterpart: the call reports TU_FAULT_RANGE in its status word."""
    L0, T = 800, 40
    _say(f"attention value 1e5 in the {where}: L0={L0} T={T}")
    kb, vb = synth.gen_attn_cache(14, 1, 0, L0, A)
    q, k, v = synth.gen_attn_tail(14, 1, 0, T, A)
    big = _scaled_bf16(np.array([1.0e5]))[0]
    if where == "cache":
        vb = vb.copy()
        vb[500, 1, 17] = big
    else:
        v = v.copy()
        v[3, 0, 200] = big
    kc = np.zeros((L0 + T, A.n_kv_heads, A.head_dim), np.uint16)
    vc = np.zeros_like(kc)
    kc[:L0], vc[:L0] = kb, vb
    ctx = _ctx(L0, L0 + T)
    o = torch.empty((T, A.n_q_heads, A.head_dim), dtype=torch.float32, device=DEV)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), o,
                         k_cache=[to_dev_bf16(kc)], v_cache=[to_dev_bf16(vc)])]
    up = tu.update_layer_stack([ctx], [np.array([[10, 20]])], [T], layers, _ap())
    assert tu.workspace_faults(up.workspace) & tu.TU_FAULT_RANGE


D1 = synth.CONFIGS[1].delta


def _delta_run(case, p):
    ws = tu.delta_rule_continue(case.state, case.q, case.k, case.v, case.beta_d, case.g_d, p, case.out)
    torch.cuda.synchronize()
    return tu.workspace_faults(ws)


def _dp(shape):
    return tu.delta_params(shape.n_k_heads, shape.n_v_heads, shape.d_k, shape.d_v, shape.chunk, shape.scale)


def test_delta_strong_decay_and_zero_gates():
    """g = 1e-3 on every token (the cumulative decay over a 64-token chunk is 1e-192, far
    below fp32) and g = 0 on every seventh token: outputs and state stay finite and match
    the per-token oracle."""
    shape = synth.DeltaShape(4, 8, 128, 128, 64)
    T = 300
    _say(f"delta strong decay g=1e-3, zero gates every 7th token: T={T} Hk=4 Hv=8")
    case = DeltaCase(shape, 15, 1, 1, T)
    g = np.full_like(case.g, 1e-3)
    g[::7] = 0.0
    case.g = g
    case.g_d = torch.from_numpy(g).to(DEV)
    assert _delta_run(case, _dp(shape)) == 0
    o_ref, S_ref = case.oracle()
    got_o, got_S = case.out.cpu().numpy(), case.state.cpu().numpy()
    assert np.all(np.isfinite(got_o)) and np.all(np.isfinite(got_S))
    assert_close(got_o, o_ref, "strong decay: delta out")
    assert_close(got_S, S_ref, "strong decay: delta state")


def test_delta_large_values():
    """Values scaled by 1e3 (state entries of the same order) match the oracle with the
    relative bar and raise no flag; values scaled by 1e5 overflow f16 operands and set
    TU_FAULT_RANGE."""
    shape = synth.DeltaShape(2, 4, 128, 128, 64)
    T = 150
    for scale, ok in ((1.0e3, True), (1.0e5, False)):
        _say(f"delta with v scaled by {scale:g}: T={T}")
        case = DeltaCase(shape, 16, 1, 1, T)
        v = synth.bf16_bits_to_f32(case.v_b).astype(np.float64) * scale
        case.v_b = _scaled_bf16(v)
        case.v = to_dev_bf16(case.v_b)
        case.S0 = case.S0 * np.float32(scale)
        case.state = torch.from_numpy(case.S0.copy()).to(DEV)
        faults = _delta_run(case, _dp(shape))
        if not ok:
            assert faults & tu.TU_FAULT_RANGE
            continue
        assert faults == 0
        o_ref, S_ref = case.oracle()
        for got, ref, what in ((case.out.cpu().numpy(), o_ref, "out"), (case.state.cpu().numpy(), S_ref, "state")):
            ma, mr = errors(got, ref)
            top = float(np.abs(ref).max())
            print(f"[parity] delta x{scale:g} {what}: max_abs={ma:.3e} (of {top:.3e}) mean_rel={mr:.3e}", flush=True)
            assert mr <= 1e-3 and ma <= 2e-2 * top
