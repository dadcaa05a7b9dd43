"""GPU parity of whole workloads at their full sizes (MI355X only).

Each test drives update_layer_stack through the C ABI exactly as the benchmark
does (default key-range splitting) on one of the seeded workloads and checks it
against the float64 oracle:
  * compaction indices, positions and moved cache rows bit for bit, appended
    rotated keys within one bf16 ulp;
  * attention outputs on sampled tail rows (the oracle computes each row on its own);
  * delta-rule outputs and states on sampled heads (heads are independent, so the
    oracle runs on the sub-shape of the sampled key heads and their value heads);
  * the committed metadata (length, live intervals, cursor).

Workloads: eight maintenance rounds carried over a 32K-token context (one
attention + one delta layer of 16q/2kv x 256 and 16k/32v x 128); a population of
32 contexts of 4K-16K surviving rows with ragged tails in one call; the 48-layer
stack (12 attention + 36 delta layers) on a 64K-token context with a 2048-token
tail. Plus the zero-removal identity on the device: a maintained update without
removals equals a fresh prefill of the whole sequence.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import (DEV, assert_bf16_close_bits, assert_close, bits_of, delta_oracle_heads, sample_rows,
                       to_dev_bf16)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _ap(a):
    return tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta, a.softmax_scale)


def _dp(d):
    return tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk, d.scale)


def _dev_cache(bits, cap):
    L = bits.shape[0]
    host = np.zeros((cap,) + bits.shape[1:], np.uint16)
    host[:L] = bits
    return to_dev_bf16(host)


def _nan(shape):
    return torch.full(shape, float("nan"), dtype=torch.float32, device=DEV)


def _check_attention_layer(ctx, kc, vc, ref, out, rows, what):
    n = len(ref["pos"])
    assert ctx.len == n, f"{what}: live length"
    assert np.array_equal(ctx.pos[:n].cpu().numpy(), ref["pos"]), f"{what}: positions"
    assert np.array_equal(bits_of(vc[:n]), ref["v_cache"]), f"{what}: V cache rows"
    assert_bf16_close_bits(bits_of(kc[:n]), ref["k_cache"], f"{what}: K cache rows")
    if len(rows):
        assert_close(out[torch.from_numpy(rows).to(DEV)].cpu().numpy(), ref["out"], f"{what}: attention rows {len(rows)}")


# ----------------------------------------------------------------------------- 8 rounds over a 32K context

@pytest.mark.timeout(900)
def test_long_lived_context_eight_rounds():
    """Eight scripted maintenance rounds from a 32,768-token context: every round removes
    1-4 records of 64-256 tokens at seeded positions and appends 256-1024 tail tokens; the
    compacted KV, the delta state and the cursor carry from round to round."""
    sc = synth.make_scenario(2, seed=0)
    a, d = sc.cfg.attn, sc.cfg.delta
    plan = sc.chars[0]
    L0 = plan.L_initial
    cap = max([L0] + [r.L_keep + r.T for r in plan.rounds])
    _say(f"32K context, {len(plan.rounds)} rounds, capacity {cap}, tails {[r.T for r in plan.rounds]}")
    kb, vb = synth.gen_attn_cache(0, 2, 0, L0, a)
    kc, vc = _dev_cache(kb, cap), _dev_cache(vb, cap)
    ctx = tu.Context(cap, device=DEV)
    ctx.pos[:L0] = torch.arange(L0, dtype=torch.int32, device=DEV)
    ctx.set_metadata(synth.initial_intervals(L0), L0)
    S0 = synth.gen_delta_state(0, 2, 1, d)
    state = torch.from_numpy(S0.copy()).to(DEV)
    key_heads = [0, 5, d.n_k_heads - 1]
    # the oracle's own chain: cache, positions, cursor, state of the sampled heads
    pos_h, k_h, v_h, cursor = np.arange(L0, dtype=np.int64), kb, vb, L0
    S_h = S0.astype(np.float64).copy()
    all_inputs = []
    for ri, r in enumerate(plan.rounds):
        assert r.cursor == cursor and r.L_old == len(pos_h)
        q, k, v = synth.gen_attn_tail(0, 2, 0, r.T, a, rnd=ri)
        dq, dk, dv, beta, g = synth.gen_delta_inputs(0, 2, 1, r.T, d, rnd=ri)
        all_inputs.append((dq, dk, dv, beta, g))
        a_out = _nan((r.T, a.n_q_heads, a.head_dim))
        d_out = _nan((r.T, d.n_v_heads, d.d_v))
        src = torch.full((cap,), -1, dtype=torch.int32, device=DEV)
        layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), a_out,
                             k_cache=[kc], v_cache=[vc]),
                  tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(dq), to_dev_bf16(dk), to_dev_bf16(dv), d_out,
                             state=[state], beta=torch.from_numpy(beta).to(DEV), g=torch.from_numpy(g).to(DEV))]
        _say(f"round {ri}: L_old {r.L_old}, ranges {r.ranges.tolist()}, T {r.T}, cursor {r.cursor}")
        tu.update_layer_stack([ctx], [r.ranges], [r.T], layers, _ap(a), _dp(d), src_index=[src])
        torch.cuda.synchronize()
        rows = sample_rows(r.T, 12, seed=100 + ri)
        ref = oracle.attention_layer_update(pos_h, k_h, v_h, r.ranges, cursor, q, k, v, a.rdim, a.rope_theta,
                                            a.softmax_scale, live=pos_h.tolist(), rows=rows)
        assert np.array_equal(src[: ref["L_keep"]].cpu().numpy(), ref["src_index"]), f"round {ri}: src_index"
        _check_attention_layer(ctx, kc, vc, ref, a_out, rows, f"round {ri}")
        assert ctx.next_pos == cursor + r.T
        assert ctx.intervals() == synth.append_interval(synth.subtract_ranges(r.intervals, r.ranges), r.cursor, r.T)
        vh, o_ref, S_ref = delta_oracle_heads(S_h, dq, dk, dv, beta, g, d.scale, key_heads)
        assert_close(d_out[:, torch.from_numpy(vh).to(DEV)].cpu().numpy(), o_ref, f"round {ri}: delta out")
        assert_close(state[torch.from_numpy(vh).to(DEV)].cpu().numpy(), S_ref, f"round {ri}: delta state")
        S_h[vh] = S_ref
        pos_h, k_h, v_h, cursor = ref["pos"], ref["k_cache"], ref["v_cache"], ref["cursor"]
    # removals never touch the recurrent state: the state after the rounds equals one
    # uninterrupted pass over the concatenated tails
    cat = [np.concatenate([x[i] for x in all_inputs]) for i in range(5)]
    one = torch.from_numpy(S0.copy()).to(DEV)
    o_one = _nan((cat[0].shape[0], d.n_v_heads, d.d_v))
    _say(f"one delta pass over all {cat[0].shape[0]} tail tokens")
    tu.delta_rule_continue(one, to_dev_bf16(cat[0]), to_dev_bf16(cat[1]), to_dev_bf16(cat[2]),
                           torch.from_numpy(cat[3]).to(DEV), torch.from_numpy(cat[4]).to(DEV), _dp(d), o_one)
    torch.cuda.synchronize()
    vh_t = torch.from_numpy(vh).to(DEV)
    assert_close(one[vh_t].cpu().numpy(), S_h[vh], "one pass vs the oracle's rounds")
    assert_close(state.cpu().numpy(), one.cpu().numpy().astype(np.float64), "rounds vs one pass, every head")


# ----------------------------------------------------------------------------- 32 contexts in one call

@pytest.mark.timeout(900)
def test_population_batch_of_32_contexts():
    """32 contexts with 4K-16K surviving rows, 0-4 removed 64-token records each and
    tails of 128-512 tokens, updated together in one call (packed ragged tails, one
    index list per context)."""
    sc = synth.make_scenario(3, seed=0)
    a, d = sc.cfg.attn, sc.cfg.delta
    rs = [ch.rounds[0] for ch in sc.chars]
    Ts = [r.T for r in rs]
    off = np.concatenate([[0], np.cumsum(Ts)])
    _say(f"32 contexts: L_keep {min(r.L_keep for r in rs)}-{max(r.L_keep for r in rs)}, "
         f"T {min(Ts)}-{max(Ts)}, removed records {[len(r.ranges) for r in rs]}")
    t0 = time.time()
    host, ctxs, kcs, vcs, srcs, states = [], [], [], [], [], []
    qs, ks, vs, dqs, dks, dvs, bs, gs = [], [], [], [], [], [], [], []
    for c, r in enumerate(rs):
        cap = max(r.L_old, r.L_keep + r.T)
        kb, vb = synth.gen_attn_cache(0, 3, 0, r.L_old, a, char=c)
        q, k, v = synth.gen_attn_tail(0, 3, 0, r.T, a, char=c)
        S0 = synth.gen_delta_state(0, 3, 1, d, char=c)
        dq, dk, dv, beta, g = synth.gen_delta_inputs(0, 3, 1, r.T, d, char=c)
        host.append((kb, vb, q, k, v, S0, dq, dk, dv, beta, g))
        kcs.append(_dev_cache(kb, cap))
        vcs.append(_dev_cache(vb, cap))
        ctx = tu.Context(cap, device=DEV)
        ctx.pos[: r.L_old] = torch.arange(r.L_old, dtype=torch.int32, device=DEV)
        ctx.set_metadata(r.intervals, r.cursor)
        ctxs.append(ctx)
        srcs.append(torch.full((cap,), -1, dtype=torch.int32, device=DEV))
        states.append(torch.from_numpy(S0.copy()).to(DEV))
        for lst, x in zip((qs, ks, vs, dqs, dks, dvs, bs, gs), (q, k, v, dq, dk, dv, beta, g)):
            lst.append(x)
    _say(f"inputs drawn in {time.time() - t0:.1f} s")
    a_out = _nan((int(off[-1]), a.n_q_heads, a.head_dim))
    d_out = _nan((int(off[-1]), d.n_v_heads, d.d_v))
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(np.concatenate(qs)), to_dev_bf16(np.concatenate(ks)),
                         to_dev_bf16(np.concatenate(vs)), a_out, k_cache=kcs, v_cache=vcs),
              tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(np.concatenate(dqs)), to_dev_bf16(np.concatenate(dks)),
                         to_dev_bf16(np.concatenate(dvs)), d_out, state=states,
                         beta=torch.from_numpy(np.concatenate(bs)).to(DEV),
                         g=torch.from_numpy(np.concatenate(gs)).to(DEV))]
    tu.update_layer_stack(ctxs, [r.ranges for r in rs], Ts, layers, _ap(a), _dp(d), src_index=srcs)
    torch.cuda.synchronize()
    for c, r in enumerate(rs):
        kb, vb, q, k, v, S0, dq, dk, dv, beta, g = host[c]
        _say(f"context {c}: L_old {r.L_old}, L_keep {r.L_keep}, T {r.T}")
        rows = sample_rows(r.T, 6, seed=200 + c)
        ref = oracle.attention_layer_update(np.arange(r.L_old), kb, vb, r.ranges, r.cursor, q, k, v, a.rdim,
                                            a.rope_theta, a.softmax_scale, rows=rows)
        assert np.array_equal(srcs[c][: r.L_keep].cpu().numpy(), ref["src_index"]), f"context {c}: src_index"
        out_c = a_out[int(off[c]): int(off[c + 1])]
        _check_attention_layer(ctxs[c], kcs[c], vcs[c], ref, out_c, rows, f"context {c}")
        assert ctxs[c].next_pos == r.cursor + r.T
        assert ctxs[c].intervals() == synth.append_interval(synth.subtract_ranges(r.intervals, r.ranges),
                                                            r.cursor, r.T)
        vh, o_ref, S_ref = delta_oracle_heads(S0, dq, dk, dv, beta, g, d.scale, [c % d.n_k_heads])
        vh_t = torch.from_numpy(vh).to(DEV)
        assert_close(d_out[int(off[c]): int(off[c + 1])][:, vh_t].cpu().numpy(), o_ref, f"context {c}: delta out")
        assert_close(states[c][vh_t].cpu().numpy(), S_ref, f"context {c}: delta state")


# ----------------------------------------------------------------------------- 48-layer stack, 64K context

@pytest.mark.timeout(900)
def test_full_depth_stack_64k():
    """48 layers (attention at every fourth layer, gated delta rule elsewhere) on a
    65,536-token context: 8 records of 256 tokens removed, 2048 tail tokens."""
    sc = synth.make_scenario(4, seed=0)
    cfg, a, d = sc.cfg, sc.cfg.attn, sc.cfg.delta
    r = sc.chars[0].rounds[0]
    kinds = cfg.layer_kinds()
    cap = max(r.L_old, r.L_keep + r.T)
    _say(f"48 layers ({kinds.count('attn')} attention), L_old {r.L_old}, L_keep {r.L_keep}, T {r.T}")
    t0 = time.time()
    ctx = tu.Context(cap, device=DEV)
    ctx.pos[: r.L_old] = torch.arange(r.L_old, dtype=torch.int32, device=DEV)
    ctx.set_metadata(r.intervals, r.cursor)
    src = torch.full((cap,), -1, dtype=torch.int32, device=DEV)
    layers, host = [], []
    for l, kind in enumerate(kinds):
        if kind == "attn":
            kb, vb = synth.gen_attn_cache(0, 4, l, r.L_old, a)
            q, k, v = synth.gen_attn_tail(0, 4, l, r.T, a)
            kc, vc = _dev_cache(kb, cap), _dev_cache(vb, cap)
            out = _nan((r.T, a.n_q_heads, a.head_dim))
            layers.append(tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), out,
                                     k_cache=[kc], v_cache=[vc]))
            host.append(("attn", kb, vb, q, k, v, kc, vc, out))
        else:
            S0 = synth.gen_delta_state(0, 4, l, d)
            dq, dk, dv, beta, g = synth.gen_delta_inputs(0, 4, l, r.T, d)
            st = torch.from_numpy(S0.copy()).to(DEV)
            out = _nan((r.T, d.n_v_heads, d.d_v))
            layers.append(tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(dq), to_dev_bf16(dk), to_dev_bf16(dv), out,
                                     state=[st], beta=torch.from_numpy(beta).to(DEV), g=torch.from_numpy(g).to(DEV)))
            host.append(("delta", S0, dq, dk, dv, beta, g, st, out))
        if l % 12 == 11:
            _say(f"layers 0..{l} drawn ({time.time() - t0:.1f} s)")
    tu.update_layer_stack([ctx], [r.ranges], [r.T], layers, _ap(a), _dp(d), src_index=[src])
    torch.cuda.synchronize()
    _say("stack update done; checking every layer")
    want_src, _ = oracle.compact(np.arange(r.L_old), r.ranges)
    assert np.array_equal(src[: r.L_keep].cpu().numpy(), want_src)
    assert ctx.len == r.L_keep + r.T and ctx.next_pos == r.cursor + r.T
    assert ctx.intervals() == synth.append_interval(synth.subtract_ranges(r.intervals, r.ranges), r.cursor, r.T)
    first_attn, last_attn = kinds.index("attn"), len(kinds) - 1 - kinds[::-1].index("attn")
    for l, h in enumerate(host):
        if h[0] == "attn":
            _, kb, vb, q, k, v, kc, vc, out = h
            rows = sample_rows(r.T, 8 if l in (first_attn, last_attn) else 2, seed=300 + l)
            ref = oracle.attention_layer_update(np.arange(r.L_old), kb, vb, r.ranges, r.cursor, q, k, v, a.rdim,
                                                a.rope_theta, a.softmax_scale, rows=rows)
            _check_attention_layer(ctx, kc, vc, ref, out, rows, f"layer {l} (attention)")
        else:
            _, S0, dq, dk, dv, beta, g, st, out = h
            vh, o_ref, S_ref = delta_oracle_heads(S0, dq, dk, dv, beta, g, d.scale, [l % d.n_k_heads])
            vh_t = torch.from_numpy(vh).to(DEV)
            assert_close(out[:, vh_t].cpu().numpy(), o_ref, f"layer {l} (delta): out")
            assert_close(st[vh_t].cpu().numpy(), S_ref, f"layer {l} (delta): state")


# ----------------------------------------------------------------------------- zero removals = prefill

def test_zero_removals_equal_fresh_prefill():
    """Without removals the maintained update is the tail of an ordinary prefill: prefill
    N0 tokens into an empty context, then update with no ranges and T more tokens; the
    tail's attention rows and the final delta state equal those of one prefill of all
    N0 + T tokens (each checked against the oracle, and the two against each other)."""
    a = synth.AttnShape(16, 2, 256)
    d = synth.DeltaShape(16, 32, 128, 128, 64)
    N0, T = 1500, 200
    N = N0 + T
    _say(f"prefill {N0} then update T={T} with no removals vs one prefill of {N}")
    q, k, v = synth.gen_attn_tail(5, 1, 0, N, a)
    S0 = np.zeros((d.n_v_heads, d.d_v, d.d_k), np.float32)
    dq, dk, dv, beta, g = synth.gen_delta_inputs(5, 1, 1, N, d)

    def run(parts):
        kc = torch.zeros((N, a.n_kv_heads, a.head_dim), dtype=torch.bfloat16, device=DEV)
        vc = torch.zeros_like(kc)
        ctx = tu.Context(N, device=DEV)
        ctx.set_metadata([], 0)
        st = torch.zeros((d.n_v_heads, d.d_v, d.d_k), dtype=torch.float32, device=DEV)
        outs = []
        for (s, e) in parts:
            ao = _nan((e - s, a.n_q_heads, a.head_dim))
            do = _nan((e - s, d.n_v_heads, d.d_v))
            layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q[s:e]), to_dev_bf16(k[s:e]), to_dev_bf16(v[s:e]),
                                 ao, k_cache=[kc], v_cache=[vc]),
                      tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(dq[s:e]), to_dev_bf16(dk[s:e]), to_dev_bf16(dv[s:e]),
                                 do, state=[st], beta=torch.from_numpy(beta[s:e]).to(DEV),
                                 g=torch.from_numpy(g[s:e]).to(DEV))]
            tu.update_layer_stack([ctx], [np.zeros((0, 2), np.int64)], [e - s], layers, _ap(a), _dp(d))
            outs.append((ao, do))
        torch.cuda.synchronize()
        assert ctx.len == N and ctx.next_pos == N and ctx.intervals() == [(0, N)]
        return outs, st, kc, vc

    (_, (ao2, do2)), st2, kc2, vc2 = run([(0, N0), (N0, N)])
    ((ao1, do1),), st1, kc1, vc1 = run([(0, N)])
    rows = sample_rows(T, 16, seed=7)
    ref_out, ref_k = oracle.refill_attention(q, k, v, a.rdim, a.rope_theta, a.softmax_scale, rows=N0 + rows)
    rows_t = torch.from_numpy(rows).to(DEV)
    assert_close(ao2[rows_t].cpu().numpy(), ref_out, "maintained tail vs oracle prefill")
    assert_close(ao1[N0 + rows_t].cpu().numpy(), ref_out, "device prefill vs oracle prefill")
    assert_close(ao2.cpu().numpy(), ao1[N0:].cpu().numpy().astype(np.float64), "maintained tail vs device prefill")
    assert np.array_equal(bits_of(kc1), bits_of(kc2)) and np.array_equal(bits_of(vc1), bits_of(vc2))
    assert_bf16_close_bits(bits_of(kc2), ref_k, "cache keys vs oracle prefill")
    vh, o_ref, S_ref = delta_oracle_heads(S0, dq, dk, dv, beta, g, d.scale, [0, 9])
    vh_t = torch.from_numpy(vh).to(DEV)
    assert_close(st2[vh_t].cpu().numpy(), S_ref, "maintained state vs oracle one pass")
    assert_close(do2[:, vh_t].cpu().numpy(), o_ref[N0:], "maintained delta tail vs oracle")
    assert_close(st2.cpu().numpy(), st1.cpu().numpy().astype(np.float64), "maintained state vs device one pass")


def test_paper_shaped_revision_trace():
    """Revisions shaped like the paper's measured trace (records in 10K-position slots,
    one or two whole records replaced per revision at fresh slots past the cursor, framing
    delimiters prefilled and removed again), carried over four revisions of one context
    with one attention and one delta layer; every revision checked against the oracle
    chained from the previous one."""
    A, D = synth.CONFIGS[1].attn, synth.CONFIGS[1].delta
    tr = synth.make_paper_trace(seed=5, head=700, n_records=10, record_len=(330, 450), n_revisions=4,
                                m_range=(214, 362), index=201)
    L0 = len(tr.positions)
    cap = max([L0] + [r.L_old + r.T for r in tr.revisions])
    k_bits, v_bits = synth.gen_attn_cache(5, 201, 0, L0, A)
    S = synth.gen_delta_state(5, 201, 1, D).astype(np.float64)
    kc, vc = _dev_cache(k_bits, cap), _dev_cache(v_bits, cap)
    state = torch.from_numpy(S.astype(np.float32)).to(DEV)
    ctx = tu.Context(cap, device=DEV)
    ctx.pos[:L0] = torch.from_numpy(tr.positions.astype(np.int32)).to(DEV)
    ctx.set_metadata(tr.intervals, tr.cursor)
    pos, kb, vb = tr.positions.copy(), k_bits, v_bits
    for ri, rv in enumerate(tr.revisions):
        _say(f"revision {ri}: remove {rv.ranges.tolist()}, tail runs {rv.runs}, framing {rv.post.tolist()}, T {rv.T}")
        assert ctx.len == rv.L_old and ctx.next_pos == rv.cursor
        q, k, v = synth.gen_attn_tail(5, 201, 0, rv.T, A, rnd=ri)
        dq, dk, dv, beta, g = synth.gen_delta_inputs(5, 201, 1, rv.T, D, rnd=ri)
        a_out = torch.full((rv.T, A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
        d_out = torch.full((rv.T, D.n_v_heads, D.d_v), float("nan"), dtype=torch.float32, device=DEV)
        layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), a_out, k_cache=[kc],
                             v_cache=[vc]),
                  tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(dq), to_dev_bf16(dk), to_dev_bf16(dv), d_out,
                             state=[state], beta=torch.from_numpy(beta).to(DEV), g=torch.from_numpy(g).to(DEV))]
        up = tu.update_layer_stack([ctx], [rv.ranges], [rv.T], layers, _ap(A), _dp(D), post_ranges=[rv.post],
                              placement=["slot"], place_runs=[rv.runs])
        torch.cuda.synchronize()
        tail_pos = np.concatenate([np.arange(a, b) for a, b in rv.runs])
        ref = oracle.attention_layer_update(pos, kb, vb, rv.ranges, rv.cursor, q, k, v, A.rdim, A.rope_theta,
                                            A.softmax_scale, live=pos, post_ranges=rv.post,
                                            placement="slot", tail_positions=tail_pos)
        n = len(ref["pos"])
        assert ctx.len == n and ctx.next_pos == rv.cursor_after
        assert np.array_equal(ctx.pos[:n].cpu().numpy(), ref["pos"])
        assert np.array_equal(bits_of(vc[:n]), ref["v_cache"])
        assert_bf16_close_bits(bits_of(kc[:n]), ref["k_cache"], f"revision {ri}: K cache")
        assert_close(a_out.cpu().numpy(), ref["out"], f"revision {ri}: attention")
        o_ref, S = oracle.delta_layer_update(S, dq, dk, dv, beta, g, D.scale)
        assert_close(d_out.cpu().numpy(), o_ref, f"revision {ri}: delta out")
        assert_close(state.cpu().numpy(), S, f"revision {ri}: delta state")
        pos, kb, vb = ref["pos"], ref["k_cache"], ref["v_cache"]
        assert tu.workspace_faults(up.workspace) == 0, f"revision {ri}: device check"

