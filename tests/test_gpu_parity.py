"""GPU parity of the HIP path against the float64 oracle (MI355X only).

Every call goes through the C ABI (libtailupdate.so) via the ctypes binding.
Inputs are the seeded synthetic workloads of `synth`; each test prints the case
it runs before the GPU work so a failure names it.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import (AttnCase, DeltaCase, DEV, assert_bf16_close_bits, assert_close, bits_of, errors,
                       to_dev_bf16)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _ctx_for(case: AttnCase):
    ctx = tu.Context(case.capacity, device=DEV)
    ctx.pos[: case.L_old] = torch.from_numpy(case.positions.astype(np.int32)).to(DEV)
    iv = []
    for p in case.positions.tolist():
        if iv and iv[-1][1] == p:
            iv[-1] = (iv[-1][0], p + 1)
        else:
            iv.append((p, p + 1))
    ctx.set_metadata(iv, int(case.positions[-1]) + 1 if case.L_old else 0)
    return ctx


# ----------------------------------------------------------------------------- compaction

@pytest.mark.parametrize("cfg", [0, 1, 4])
def test_compaction_bit_exact(cfg):
    sc = synth.make_scenario(cfg, seed=0)
    r = sc.chars[0].rounds[0]
    shape = sc.cfg.attn
    n_layers = 3 if cfg == 4 else 1
    _say(f"compaction cfg{cfg} L_old={r.L_old} ranges={r.ranges.tolist()} layers={n_layers}")
    cases = [AttnCase(shape, 0, cfg, 4 * l + 3, r.L_old, 0, capacity=r.L_old) for l in range(n_layers)]
    ctx = _ctx_for(cases[0])
    src = torch.full((r.L_old,), -1, dtype=torch.int32, device=DEV)
    tu.compact_kv(ctx, [c.k_cache for c in cases], [c.v_cache for c in cases], r.ranges, src_index=src)
    torch.cuda.synchronize()
    want_src, want_pos = oracle.compact(np.arange(r.L_old), r.ranges)
    n = len(want_src)
    assert ctx.len == n and ctx.next_pos == r.cursor
    assert np.array_equal(src[:n].cpu().numpy(), want_src)
    assert np.array_equal(ctx.pos[:n].cpu().numpy(), want_pos)
    for c in cases:
        assert np.array_equal(bits_of(c.k_cache[:n]), c.k_bits[want_src])
        assert np.array_equal(bits_of(c.v_cache[:n]), c.v_bits[want_src])
    assert ctx.intervals() == synth.subtract_ranges(r.intervals, r.ranges)


@pytest.mark.parametrize("name,L,ranges", [
    ("front", 3000, [(0, 700)]),
    ("back", 3000, [(2900, 3000)]),
    ("adjacent", 3000, [(100, 200), (200, 300), (2999, 3000)]),
    ("everything", 500, [(0, 500)]),
    ("many_small", 20000, [(i * 150 + 7, i * 150 + 9) for i in range(128)]),
    ("none", 1000, []),
])
def test_compaction_edge_cases(name, L, ranges):
    shape = synth.AttnShape(2, 1, 64)      # 128-byte rows: many rows per stripe
    _say(f"compaction edge {name} L={L} n_ranges={len(ranges)}")
    case = AttnCase(shape, 1, 0, 1, L, 0, capacity=L)
    ctx = _ctx_for(case)
    src = torch.full((L,), -1, dtype=torch.int32, device=DEV)
    tu.compact_kv(ctx, [case.k_cache], [case.v_cache], np.asarray(ranges, dtype=np.int64).reshape(-1, 2),
                  src_index=src)
    torch.cuda.synchronize()
    want_src, want_pos = oracle.compact(np.arange(L), ranges)
    n = len(want_src)
    assert ctx.len == n
    assert np.array_equal(src[:n].cpu().numpy(), want_src)
    assert np.array_equal(ctx.pos[:n].cpu().numpy(), want_pos)
    assert np.array_equal(bits_of(case.k_cache[:n]), case.k_bits[want_src])
    assert np.array_equal(bits_of(case.v_cache[:n]), case.v_bits[want_src])


# ----------------------------------------------------------------------------- attention

def _attn_update(case, ctx, ranges, params, src=None):
    tu.compact_kv(ctx, [case.k_cache], [case.v_cache], ranges, src_index=src)
    tu.tail_prefill_attention(ctx, case.k_cache, case.v_cache, params, case.q, case.k, case.v, case.out,
                              q_hat=case.q_hat)
    torch.cuda.synchronize()


@pytest.mark.parametrize("cfg", [0, 1])
def test_attention_update_parity(cfg):
    sc = synth.make_scenario(cfg, seed=0)
    r = sc.chars[0].rounds[0]
    s = sc.cfg.attn
    _say(f"attention cfg{cfg} L_old={r.L_old} L_keep={r.L_keep} T={r.T}")
    case = AttnCase(s, 0, cfg, 0, r.L_old, r.T)
    ctx = _ctx_for(case)
    p = tu.attn_params(s.n_q_heads, s.n_kv_heads, s.head_dim, s.rdim, s.rope_theta, s.softmax_scale)
    _attn_update(case, ctx, r.ranges, p)
    ref = case.oracle(r.ranges, r.cursor)
    assert_bf16_close_bits(bits_of(case.q_hat), ref["q_hat"], f"cfg{cfg} rotated q")
    N = r.L_keep + r.T
    assert_bf16_close_bits(bits_of(case.k_cache[:N]), ref["k_cache"], f"cfg{cfg} K cache")
    assert np.array_equal(bits_of(case.v_cache[:N]), ref["v_cache"])
    assert np.array_equal(ctx.pos[:N].cpu().numpy(), ref["pos"])
    assert_close(case.out.cpu().numpy(), ref["out"], f"cfg{cfg} attention out")


@pytest.mark.parametrize("L_keep,T,splits", [(0, 1, 0), (0, 77, 0), (5, 1, 0), (300, 17, 1), (1000, 200, 3),
                                             (4000, 64, 0), (2000, 511, 7), (32768, 1, 0), (32768, 8, 0),
                                             (3000, 40, 12), (4000, 64, 24), (300, 17, 40)])
def test_attention_shapes(L_keep, T, splits):
    s = synth.CONFIGS[1].attn
    _say(f"attention shape L_keep={L_keep} T={T} splits={splits}")
    case = AttnCase(s, 3, 1, 0, L_keep, T)
    ctx = _ctx_for(case)
    p = tu.attn_params(s.n_q_heads, s.n_kv_heads, s.head_dim, s.rdim, s.rope_theta, s.softmax_scale, kv_splits=splits)
    _attn_update(case, ctx, np.zeros((0, 2), np.int64), p)
    ref = case.oracle(np.zeros((0, 2), np.int64), L_keep)
    assert_close(case.out.cpu().numpy(), ref["out"], f"L_keep={L_keep} T={T} splits={splits}")


@pytest.mark.parametrize("Hq,Hkv,D,rdim,L_keep,T,splits", [(8, 2, 128, 128, 700, 45, 0), (4, 4, 128, 64, 300, 130, 2),
                                                        (16, 2, 64, 64, 1500, 33, 0), (6, 2, 256, 192, 900, 70, 3)])
def test_attention_head_dims(Hq, Hkv, D, rdim, L_keep, T, splits):
    # every compiled head size, group sizes 1..8 and a partial rotary dimension
    s = synth.AttnShape(n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, rotary_dim=rdim)
    _say(f"attention Hq={Hq} Hkv={Hkv} D={D} rdim={rdim} L_keep={L_keep} T={T} splits={splits}")
    case = AttnCase(s, 5, 1, 0, L_keep, T)
    ctx = _ctx_for(case)
    p = tu.attn_params(Hq, Hkv, D, rdim, s.rope_theta, s.softmax_scale, kv_splits=splits)
    _attn_update(case, ctx, np.zeros((0, 2), np.int64), p)
    ref = case.oracle(np.zeros((0, 2), np.int64), L_keep)
    assert_bf16_close_bits(bits_of(case.q_hat), ref["q_hat"], f"D={D} rotated q")
    assert_close(case.out.cpu().numpy(), ref["out"], f"Hq={Hq} Hkv={Hkv} D={D} rdim={rdim}")


def test_attention_splits_agree():
    s = synth.CONFIGS[1].attn
    _say("attention split counts 1 vs 4 vs auto on cfg1 shapes")
    outs = []
    for splits in (1, 4, 0):
        case = AttnCase(s, 0, 1, 0, 8192, 512)
        ctx = _ctx_for(case)
        p = tu.attn_params(s.n_q_heads, s.n_kv_heads, s.head_dim, kv_splits=splits)
        _attn_update(case, ctx, np.zeros((0, 2), np.int64), p)
        outs.append(case.out.cpu().numpy())
    assert_close(outs[1], outs[0], "splits 4 vs 1")
    assert_close(outs[2], outs[0], "splits auto vs 1")


def test_attention_large_positions():
    # true-tail cursor of the paper's placement case (Section 6.3): 479,547
    s = synth.CONFIGS[1].attn
    pos = np.concatenate([np.arange(0, 2000), np.arange(470000, 477547)])
    _say("attention at cursor 479547")
    case = AttnCase(s, 4, 1, 0, len(pos), 300, positions=pos)
    ctx = _ctx_for(case)
    ctx.set_metadata([(0, 2000), (470000, 477547)], 479547)
    p = tu.attn_params(s.n_q_heads, s.n_kv_heads, s.head_dim, s.rdim, s.rope_theta, s.softmax_scale)
    ranges = np.array([[100, 228], [471000, 471300]])
    _attn_update(case, ctx, ranges, p)
    ref = case.oracle(ranges, 479547)
    assert_bf16_close_bits(bits_of(case.q_hat), ref["q_hat"], "rotated q at 479547")
    assert_close(case.out.cpu().numpy(), ref["out"], "attention at 479547")


# ----------------------------------------------------------------------------- delta rule

@pytest.mark.parametrize("cfg", [0, 1])
def test_delta_parity(cfg):
    sc = synth.make_scenario(cfg, seed=0)
    T = sc.chars[0].rounds[0].T
    d = sc.cfg.delta
    _say(f"delta cfg{cfg} T={T} chunk={d.chunk}")
    case = DeltaCase(d, 0, cfg, 1, T)
    p = tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk, d.scale)
    tu.delta_rule_continue(case.state, case.q, case.k, case.v, case.beta_d, case.g_d, p, case.out)
    torch.cuda.synchronize()
    o_ref, S_ref = case.oracle()
    assert_close(case.out.cpu().numpy(), o_ref, f"cfg{cfg} delta out")
    assert_close(case.state.cpu().numpy(), S_ref, f"cfg{cfg} delta state")


@pytest.mark.parametrize("d,chunk,T,hk,hv", [(128, 64, 100, 2, 4), (128, 64, 1, 2, 4), (128, 32, 70, 1, 2),
                                             (128, 16, 33, 1, 1), (64, 64, 129, 2, 2), (64, 16, 50, 1, 2),
                                             (64, 32, 45, 2, 4)])
def test_delta_shapes(d, chunk, T, hk, hv):
    shape = synth.DeltaShape(hk, hv, d, d, chunk)
    _say(f"delta shape d={d} chunk={chunk} T={T} Hk={hk} Hv={hv}")
    case = DeltaCase(shape, 5, 9, 0, T)
    p = tu.delta_params(hk, hv, d, d, chunk, shape.scale)
    tu.delta_rule_continue(case.state, case.q, case.k, case.v, case.beta_d, case.g_d, p, case.out)
    torch.cuda.synchronize()
    o_ref, S_ref = case.oracle()
    assert_close(case.out.cpu().numpy(), o_ref, f"delta d={d} C={chunk} T={T} out")
    assert_close(case.state.cpu().numpy(), S_ref, f"delta d={d} C={chunk} T={T} state")


def test_delta_continuation_equals_one_pass():
    d = synth.CONFIGS[1].delta
    _say("delta 3 calls (200+57+255) vs oracle one pass")
    case = DeltaCase(d, 6, 1, 1, 512)
    p = tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk, d.scale)
    for a, b in [(0, 200), (200, 257), (257, 512)]:
        out = torch.empty((b - a, d.n_v_heads, d.d_v), dtype=torch.float32, device=DEV)
        tu.delta_rule_continue(case.state, case.q[a:b], case.k[a:b], case.v[a:b], case.beta_d[a:b], case.g_d[a:b], p,
                               out)
        case.out[a:b] = out
    torch.cuda.synchronize()
    o_ref, S_ref = case.oracle()
    assert_close(case.out.cpu().numpy(), o_ref, "split delta out")
    assert_close(case.state.cpu().numpy(), S_ref, "split delta state")


# ----------------------------------------------------------------------------- stack update

def _stack_case(cfg, seed=0, char=0, rnd=0, plan_round=None, cases=None):
    sc = synth.make_scenario(cfg, seed=seed)
    r = plan_round if plan_round is not None else sc.chars[char].rounds[rnd]
    return sc, r


def test_stack_update_cfg1_matches_oracle_and_commits():
    sc, r = _stack_case(1)
    a, d = sc.cfg.attn, sc.cfg.delta
    _say(f"stack cfg1 [attn, delta] L_old={r.L_old} T={r.T}")
    ac = AttnCase(a, 0, 1, 0, r.L_old, r.T)
    dc = DeltaCase(d, 0, 1, 1, r.T)
    ctx = _ctx_for(ac)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, ac.q, ac.k, ac.v, ac.out, k_cache=[ac.k_cache], v_cache=[ac.v_cache]),
              tu.LayerIO(tu.TU_LAYER_DELTA, dc.q, dc.k, dc.v, dc.out, state=[dc.state], beta=dc.beta_d, g=dc.g_d)]
    src = torch.full((r.L_old,), -1, dtype=torch.int32, device=DEV)
    tu.update_layer_stack([ctx], [r.ranges], [r.T], layers,
                          tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta),
                          tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk), src_index=[src])
    torch.cuda.synchronize()
    ref = ac.oracle(r.ranges, r.cursor)
    assert np.array_equal(src[: r.L_keep].cpu().numpy(), ref["src_index"])
    assert_close(ac.out.cpu().numpy(), ref["out"], "stack attention out")
    o_ref, S_ref = dc.oracle()
    assert_close(dc.out.cpu().numpy(), o_ref, "stack delta out")
    assert_close(dc.state.cpu().numpy(), S_ref, "stack delta state")
    assert ctx.len == r.L_keep + r.T and ctx.next_pos == r.cursor + r.T
    assert ctx.intervals() == synth.append_interval(synth.subtract_ranges(r.intervals, r.ranges), r.cursor, r.T)


def test_stack_update_removes_delimiters_after_prefill():
    # Section 4.1: an 11-token opening wrapper and a 3-token closing one are prefilled
    # with the replacement, then their rows leave every attention cache
    sc, r = _stack_case(1)
    a, d = sc.cfg.attn, sc.cfg.delta
    post = np.array([[r.cursor, r.cursor + 11], [r.cursor + r.T - 3, r.cursor + r.T]])
    _say(f"stack cfg1 with post-prefill removal of {post.tolist()}")
    ac = AttnCase(a, 0, 1, 0, r.L_old, r.T)
    dc = DeltaCase(d, 0, 1, 1, r.T)
    ctx = _ctx_for(ac)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, ac.q, ac.k, ac.v, ac.out, k_cache=[ac.k_cache], v_cache=[ac.v_cache]),
              tu.LayerIO(tu.TU_LAYER_DELTA, dc.q, dc.k, dc.v, dc.out, state=[dc.state], beta=dc.beta_d, g=dc.g_d)]
    tu.update_layer_stack([ctx], [r.ranges], [r.T], layers,
                          tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta),
                          tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk), post_ranges=[post])
    torch.cuda.synchronize()
    ref = ac.oracle(r.ranges, r.cursor, post_ranges=post)
    n = r.L_keep + r.T - 14
    assert ctx.len == n and ctx.next_pos == r.cursor + r.T
    assert_close(ac.out.cpu().numpy(), ref["out"], "attention out of every tail row")
    assert np.array_equal(ctx.pos[:n].cpu().numpy(), ref["pos"])
    assert np.array_equal(bits_of(ac.v_cache[:n]), ref["v_cache"])
    assert_bf16_close_bits(bits_of(ac.k_cache[:n]), ref["k_cache"], "retained K cache")
    o_ref, S_ref = dc.oracle()
    assert_close(dc.state.cpu().numpy(), S_ref, "delta state keeps the delimiters' influence")
    iv = synth.append_interval(synth.subtract_ranges(r.intervals, r.ranges), r.cursor, r.T)
    assert ctx.intervals() == synth.subtract_ranges(iv, post)


def test_stack_is_deterministic():
    sc, r = _stack_case(1)
    a, d = sc.cfg.attn, sc.cfg.delta
    _say("stack cfg1 run twice, bit-identical")
    res = []
    for _ in range(2):
        ac = AttnCase(a, 0, 1, 0, r.L_old, r.T)
        dc = DeltaCase(d, 0, 1, 1, r.T)
        ctx = _ctx_for(ac)
        layers = [tu.LayerIO(tu.TU_LAYER_ATTN, ac.q, ac.k, ac.v, ac.out, k_cache=[ac.k_cache], v_cache=[ac.v_cache]),
                  tu.LayerIO(tu.TU_LAYER_DELTA, dc.q, dc.k, dc.v, dc.out, state=[dc.state], beta=dc.beta_d,
                             g=dc.g_d)]
        tu.update_layer_stack([ctx], [r.ranges], [r.T], layers, tu.attn_params(16, 2, 256),
                              tu.delta_params(16, 32, 128, 128, 64))
        torch.cuda.synchronize()
        res.append((ac.out.cpu().numpy().copy(), dc.out.cpu().numpy().copy(), dc.state.cpu().numpy().copy(),
                    bits_of(ac.k_cache)))
    for x, y in zip(res[0], res[1]):
        assert np.array_equal(x, y)


# ----------------------------------------------------------------------------- short convolution

def _conv_run(st_bits, x_bits, w_bits, act):
    st = to_dev_bf16(st_bits) if st_bits.shape[0] else None
    x = to_dev_bf16(x_bits)
    w = to_dev_bf16(w_bits)
    out = torch.full(x.shape, float("nan"), dtype=torch.bfloat16, device=DEV)
    tu.short_conv_continue(st, x, w, out, activation=act)
    torch.cuda.synchronize()
    return bits_of(out), (bits_of(st) if st is not None else st_bits)


@pytest.mark.parametrize("W,C,T,act", [(4, 2048, 512, "silu"), (4, 4096, 2048, "silu"), (4, 4096, 37, "silu"),
                                       (3, 8, 1, "none"), (4, 64, 2, "silu"), (1, 32, 19, "silu"),
                                       (8, 264, 100, "none"), (2, 16, 300, "silu"), (4, 8192, 17, "none")])
def test_short_conv_parity(W, C, T, act):
    _say(f"short conv W={W} C={C} T={T} act={act}")
    st, x, w = synth.gen_conv_inputs(11, T, C, W)
    ref_y, _, ref_state = oracle.short_conv_continue(st, x, w, activation=act)
    y, state = _conv_run(st, x, w, act)
    assert_bf16_close_bits(y, ref_y, f"conv W={W} C={C} T={T} out")
    assert np.array_equal(state, ref_state), "carried state must be the last input rows, bit for bit"


def test_short_conv_continuation_is_split_invariant():
    W, C, T = 4, 1024, 200
    _say("short conv split into calls of 0, 1, 2, 61 and 136 tokens vs one call")
    st, x, w = synth.gen_conv_inputs(12, T, C, W)
    y_all, s_all = _conv_run(st, x, w, "silu")
    parts, s = [], st
    for a, b in [(0, 0), (0, 1), (1, 3), (3, 64), (64, 200)]:
        y, s = _conv_run(s, x[a:b], w, "silu")
        parts.append(y)
    assert np.array_equal(np.concatenate(parts), y_all)
    assert np.array_equal(s, s_all)
    ref_y, _, ref_s = oracle.short_conv_continue(st, x, w)
    assert_bf16_close_bits(y_all, ref_y, "conv one call vs oracle")
    assert np.array_equal(s_all, ref_s)


def test_short_conv_batch_matches_single_calls():
    # q, k, v of two contexts with ragged tails (one empty) in one call
    _say("short conv batch of 6 tensors (C 2048/2048/4096, T 300 and 0 and 5)")
    W = 4
    specs = [(2048, 300), (2048, 300), (4096, 300), (2048, 0), (2048, 5), (4096, 5)]
    items, refs = [], []
    for i, (C, T) in enumerate(specs):
        st, x, w = synth.gen_conv_inputs(13, T, C, W, layer=i)
        refs.append(oracle.short_conv_continue(st, x, w))
        items.append((to_dev_bf16(st), to_dev_bf16(x), to_dev_bf16(w),
                      torch.full((T, C), float("nan"), dtype=torch.bfloat16, device=DEV)))
    tu.short_conv_continue_batch(items)
    torch.cuda.synchronize()
    for (st, x, w, out), (ref_y, _, ref_s), (C, T) in zip(items, refs, specs):
        assert_bf16_close_bits(bits_of(out), ref_y, f"batch conv C={C} T={T}")
        assert np.array_equal(bits_of(st), ref_s)


def test_stack_equals_per_layer_calls():
    """One update_layer_stack call over two attention and two delta layers gives, bit for
    bit, what the separate entry points give layer by layer on copies of the same state
    (compact_kv over both attention layers' caches, tail_prefill_attention per layer,
    commit_tail, delta_rule_continue per layer): the stack only batches and orders them.
    The key-range split count is forced: left to the library it follows the launch's
    size, which differs between one layer and two, and with it the rounding."""
    a = synth.CONFIGS[1].attn
    d = synth.CONFIGS[1].delta
    L, T = 3000, 200
    ranges = np.array([[400, 528], [2000, 2064]])
    _say(f"stack vs per-layer calls: L {L}, ranges {ranges.tolist()}, T {T}")
    ap = tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta, a.softmax_scale,
                        kv_splits=3)
    dp = tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk, d.scale)
    caches, tails, states, dins = [], [], [], []
    for layer in range(2):
        kb, vb = synth.gen_attn_cache(7, 1, layer, L, a)
        kc = np.zeros((L + T, a.n_kv_heads, a.head_dim), np.uint16)
        vc = np.zeros_like(kc)
        kc[:L], vc[:L] = kb, vb
        caches.append((kc, vc))
        tails.append([to_dev_bf16(x) for x in synth.gen_attn_tail(7, 1, layer, T, a)])
        states.append(synth.gen_delta_state(7, 1, 2 + layer, d))
        q, k, v, beta, g = synth.gen_delta_inputs(7, 1, 2 + layer, T, d)
        dins.append((to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), torch.from_numpy(beta).to(DEV),
                     torch.from_numpy(g).to(DEV)))

    def fresh():
        ctx = tu.Context(L + T, device=DEV)
        ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
        ctx.set_metadata([(0, L)], L)
        kv = [(to_dev_bf16(kc), to_dev_bf16(vc)) for kc, vc in caches]
        st = [torch.from_numpy(S.copy()).to(DEV) for S in states]
        ao = [torch.full((T, a.n_q_heads, a.head_dim), float("nan"), dtype=torch.float32, device=DEV)
              for _ in range(2)]
        do = [torch.full((T, d.n_v_heads, d.d_v), float("nan"), dtype=torch.float32, device=DEV) for _ in range(2)]
        return ctx, kv, st, ao, do

    # the stack: attention, delta, attention, delta
    c1, kv1, st1, ao1, do1 = fresh()
    layers = []
    for i in range(2):
        q, k, v = tails[i]
        layers.append(tu.LayerIO(tu.TU_LAYER_ATTN, q, k, v, ao1[i], k_cache=[kv1[i][0]], v_cache=[kv1[i][1]]))
        dq, dk, dv, beta, g = dins[i]
        layers.append(tu.LayerIO(tu.TU_LAYER_DELTA, dq, dk, dv, do1[i], state=[st1[i]], beta=beta, g=g))
    tu.update_layer_stack([c1], [ranges], [T], layers, ap, dp)
    # the same through the separate entry points
    c2, kv2, st2, ao2, do2 = fresh()
    tu.compact_kv(c2, [k for k, _ in kv2], [v for _, v in kv2], ranges)
    for i in range(2):
        q, k, v = tails[i]
        tu.tail_prefill_attention(c2, kv2[i][0], kv2[i][1], ap, q, k, v, ao2[i])
    tu.commit_tail(c2, T)
    for i in range(2):
        dq, dk, dv, beta, g = dins[i]
        tu.delta_rule_continue(st2[i], dq, dk, dv, beta, g, dp, do2[i])
    torch.cuda.synchronize()
    assert c1.len == c2.len and c1.next_pos == c2.next_pos and c1.intervals() == c2.intervals()
    n = c1.len
    assert torch.equal(c1.pos[:n], c2.pos[:n])
    for i in range(2):
        assert torch.equal(kv1[i][0][:n], kv2[i][0][:n]) and torch.equal(kv1[i][1][:n], kv2[i][1][:n]), f"layer {i} cache"
        assert torch.equal(ao1[i], ao2[i]), f"layer {i} attention output"
        assert torch.equal(do1[i], do2[i]) and torch.equal(st1[i], st2[i]), f"layer {i} delta output and state"


def test_stack_of_many_delta_layers_equals_per_layer_calls():
    """A stack of 50 delta layers (no attention layer) takes two delta launches that reuse
    one workspace region (at most 48 (layer, context) items per launch); every layer's
    output and state must equal, bit for bit, a separate delta_rule_continue call on a
    copy of its state. T = 100 gives a ragged second chunk."""
    d = synth.CONFIGS[1].delta
    n_layers, T, L = 50, 100, 256
    _say(f"stack of {n_layers} delta layers, T {T}")
    dp = tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk, d.scale)
    states, dins = [], []
    for layer in range(n_layers):
        states.append(synth.gen_delta_state(9, 1, layer, d))
        q, k, v, beta, g = synth.gen_delta_inputs(9, 1, layer, T, d)
        dins.append((to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), torch.from_numpy(beta).to(DEV),
                     torch.from_numpy(g).to(DEV)))
    ctx = tu.Context(L + T, device=DEV)
    ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
    ctx.set_metadata([(0, L)], L)
    st1 = [torch.from_numpy(S.copy()).to(DEV) for S in states]
    st2 = [torch.from_numpy(S.copy()).to(DEV) for S in states]
    do1 = [torch.full((T, d.n_v_heads, d.d_v), float("nan"), dtype=torch.float32, device=DEV) for _ in range(n_layers)]
    do2 = [torch.full_like(x, float("nan")) for x in do1]
    layers = [tu.LayerIO(tu.TU_LAYER_DELTA, *dins[i][:3], do1[i], state=[st1[i]], beta=dins[i][3], g=dins[i][4])
              for i in range(n_layers)]
    ap = tu.attn_params(16, 2, 256)
    tu.update_layer_stack([ctx], [np.zeros((0, 2), np.int64)], [T], layers, ap, dp)
    for i in range(n_layers):
        dq, dk, dv, beta, g = dins[i]
        tu.delta_rule_continue(st2[i], dq, dk, dv, beta, g, dp, do2[i])
    torch.cuda.synchronize()
    for i in range(n_layers):
        assert torch.equal(do1[i], do2[i]) and torch.equal(st1[i], st2[i]), f"layer {i} delta output and state"
