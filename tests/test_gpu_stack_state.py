"""Stack updates with several small attention layers, and state continuity (MI355X only).

Pooled layers: attention layers whose own workgroups cannot fill the chip share one set of
launches (up to 32 (layer, context) items each, later launches reusing the same workspace).
Four such layers over nine contexts (36 items, two launches), with the library's own key
splits, each checked against the float64 oracle.

Continuity (paper Section 4.1: the context is the state (A_t, R_t, p_t)): an update, a
snapshot of the whole state (metadata, positions, caches, V^T copies, recurrent states), a
restore into fresh buffers, and the next update there equal the same two updates run
without interruption, bit for bit; both match the oracle chained over the two updates.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import DEV, assert_bf16_close_bits, assert_close, bits_of, sample_rows, to_dev_bf16

pytestmark = pytest.mark.gpu

A = synth.AttnShape(16, 2, 256)
D = synth.DeltaShape(2, 4, 64, 64, 32)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _ap(splits=0):
    return tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta, A.softmax_scale,
                          kv_splits=splits)


def _dp():
    return tu.delta_params(D.n_k_heads, D.n_v_heads, D.d_k, D.d_v, D.chunk, D.scale)


def test_pooled_small_attention_layers_many_contexts():
    rng = np.random.default_rng(77)
    n_ctx, n_attn = 9, 4
    specs = []
    for c in range(n_ctx):
        L = int(rng.integers(300, 2001))
        iv = synth.initial_intervals(L)
        ranges = synth.draw_records(rng, iv, int(rng.integers(0, 3)), (5, 120))
        specs.append((L, ranges, int(rng.integers(20, 61))))
    print(f"[case] {n_attn} attention layers + 1 delta layer, {n_ctx} contexts "
          f"{[(L, r.tolist(), T) for L, r, T in specs]}, automatic splits", flush=True)
    Ts = [T for _, _, T in specs]
    off = np.concatenate([[0], np.cumsum(Ts)]).astype(int)
    ctxs = []
    for L, _, T in specs:
        ctx = tu.Context(L + T, device=DEV)
        ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
        ctx.set_metadata(synth.initial_intervals(L), L)
        ctxs.append(ctx)
    layers, host = [], []
    for l in range(n_attn):
        per = []
        kcs, vcs = [], []
        for c, (L, _, T) in enumerate(specs):
            kb, vb = synth.gen_attn_cache(21, 400, l, L, A, char=c)
            kc = np.zeros((L + T, A.n_kv_heads, A.head_dim), np.uint16)
            vc = np.zeros_like(kc)
            kc[:L], vc[:L] = kb, vb
            kcs.append(to_dev_bf16(kc))
            vcs.append(to_dev_bf16(vc))
            per.append((kb, vb) + synth.gen_attn_tail(21, 400, l, T, A, char=c))
        out = torch.full((off[-1], A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
        cat = lambda i: to_dev_bf16(np.concatenate([p[i] for p in per]))
        layers.append(tu.LayerIO(tu.TU_LAYER_ATTN, cat(2), cat(3), cat(4), out, k_cache=kcs, v_cache=vcs))
        host.append((per, kcs, vcs, out))
    dh = [synth.gen_delta_inputs(21, 400, 9, T, D, char=c) for c, T in enumerate(Ts)]
    S0 = [synth.gen_delta_state(21, 400, 9, D, char=c) for c in range(n_ctx)]
    states = [torch.from_numpy(s.copy()).to(DEV) for s in S0]
    d_out = torch.full((off[-1], D.n_v_heads, D.d_v), float("nan"), dtype=torch.float32, device=DEV)
    layers.append(tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(np.concatenate([h[0] for h in dh])),
                             to_dev_bf16(np.concatenate([h[1] for h in dh])),
                             to_dev_bf16(np.concatenate([h[2] for h in dh])), d_out, state=states,
                             beta=torch.from_numpy(np.concatenate([h[3] for h in dh])).to(DEV),
                             g=torch.from_numpy(np.concatenate([h[4] for h in dh])).to(DEV)))
    up = tu.update_layer_stack(ctxs, [r for _, r, _ in specs], Ts, layers, _ap(), _dp())
    torch.cuda.synchronize()
    assert tu.workspace_faults(up.workspace) == 0
    for l, (per, kcs, vcs, out) in enumerate(host):
        for c, ((L, ranges, T), (kb, vb, q, k, v)) in enumerate(zip(specs, per)):
            what = f"layer {l} context {c} (L {L}, T {T})"
            rows = sample_rows(T, 10, seed=100 * l + c)
            ref = oracle.attention_layer_update(np.arange(L), kb, vb, ranges, L, q, k, v, A.rdim, A.rope_theta,
                                                A.softmax_scale, rows=rows)
            n = len(ref["pos"])
            assert ctxs[c].len == n and ctxs[c].next_pos == L + T, what
            assert np.array_equal(ctxs[c].pos[:n].cpu().numpy(), ref["pos"]), what
            assert np.array_equal(bits_of(vcs[c][:n]), ref["v_cache"]), what
            assert_bf16_close_bits(bits_of(kcs[c][:n]), ref["k_cache"], f"{what}: K cache")
            got = out[off[c]: off[c + 1]][torch.from_numpy(rows).to(DEV)].cpu().numpy()
            assert_close(got, ref["out"], f"{what}: attention rows")
    for c, T in enumerate(Ts):
        o_ref, S_ref = oracle.delta_layer_update(S0[c].astype(np.float64), *dh[c][:3], dh[c][3], dh[c][4], D.scale)
        assert_close(d_out[off[c]: off[c + 1]].cpu().numpy(), o_ref, f"context {c}: delta out")
        assert_close(states[c].cpu().numpy(), S_ref, f"context {c}: delta state")


class _State:
    """One context with an attention layer (caches + V^T copy) and a delta layer."""

    def __init__(self, L0, cap, seed):
        self.ctx = tu.Context(cap, device=DEV)
        self.ctx.pos[:L0] = torch.arange(L0, dtype=torch.int32, device=DEV)
        self.ctx.set_metadata([(0, L0)], L0)
        kb, vb = synth.gen_attn_cache(seed, 401, 0, L0, A)
        kc = np.zeros((cap, A.n_kv_heads, A.head_dim), np.uint16)
        vc = np.zeros_like(kc)
        kc[:L0], vc[:L0] = kb, vb
        self.k, self.v = to_dev_bf16(kc), to_dev_bf16(vc)
        self.vt = tu.new_vt_cache(cap, A.n_kv_heads, A.head_dim, DEV)
        tu.refresh_vt_cache(self.ctx, [self.v], [self.vt])
        self.S0 = synth.gen_delta_state(seed, 401, 1, D)
        self.S = torch.from_numpy(self.S0.copy()).to(DEV)
        self.host = (kb, vb)

    def snapshot(self):
        return (self.ctx.snapshot(), self.k.clone(), self.v.clone(), self.vt.clone(), self.S.clone())

    @classmethod
    def restored(cls, snap, cap):
        st = cls.__new__(cls)
        meta, k, v, vt, S = snap
        st.ctx = tu.Context(cap, device=DEV)
        st.ctx.restore(meta)
        st.k, st.v, st.vt, st.S = k.clone(), v.clone(), vt.clone(), S.clone()
        return st

    def update(self, ranges, T, seed, rnd):
        q, k, v = synth.gen_attn_tail(seed, 401, 0, T, A, rnd=rnd)
        dq, dk, dv, beta, g = synth.gen_delta_inputs(seed, 401, 1, T, D, rnd=rnd)
        ao = torch.empty((T, A.n_q_heads, A.head_dim), dtype=torch.float32, device=DEV)
        do = torch.empty((T, D.n_v_heads, D.d_v), dtype=torch.float32, device=DEV)
        layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), ao, k_cache=[self.k],
                             v_cache=[self.v], vt_cache=[self.vt]),
                  tu.LayerIO(tu.TU_LAYER_DELTA, to_dev_bf16(dq), to_dev_bf16(dk), to_dev_bf16(dv), do, state=[self.S],
                             beta=torch.from_numpy(beta).to(DEV), g=torch.from_numpy(g).to(DEV))]
        up = tu.update_layer_stack([self.ctx], [ranges], [T], layers, _ap(), _dp())
        torch.cuda.synchronize()
        assert tu.workspace_faults(up.workspace) == 0
        return ao, do, (q, k, v), (dq, dk, dv, beta, g)


def test_snapshot_restore_continue_equals_uninterrupted():
    L0, seed = 1800, 5
    rounds = [(np.array([[300, 420]]), 150), (np.array([[1000, 1010], [1850, 1900]]), 90)]
    cap = L0 + sum(T for _, T in rounds)
    print(f"[case] update, snapshot, restore, update: L0={L0} rounds={[(r.tolist(), T) for r, T in rounds]}",
          flush=True)
    a = _State(L0, cap, seed)
    a.update(rounds[0][0], rounds[0][1], seed, 0)
    snap = a.snapshot()
    ao1, do1, _, _ = a.update(rounds[1][0], rounds[1][1], seed, 1)          # uninterrupted
    b = _State.restored(snap, cap)
    ao2, do2, at, dt = b.update(rounds[1][0], rounds[1][1], seed, 1)        # after the restore
    assert (b.ctx.len, b.ctx.next_pos, b.ctx.intervals(), b.ctx.vt_rows) == \
        (a.ctx.len, a.ctx.next_pos, a.ctx.intervals(), a.ctx.vt_rows)
    n = a.ctx.len
    assert torch.equal(ao1, ao2) and torch.equal(do1, do2)
    assert torch.equal(a.S, b.S) and torch.equal(a.ctx.pos[:n], b.ctx.pos[:n])
    assert torch.equal(a.k[:n], b.k[:n]) and torch.equal(a.v[:n], b.v[:n])
    # and both are the oracle's two updates
    kb, vb = a.host
    q0, k0, v0 = synth.gen_attn_tail(seed, 401, 0, rounds[0][1], A, rnd=0)
    r1 = oracle.attention_layer_update(np.arange(L0), kb, vb, rounds[0][0], L0, q0, k0, v0, A.rdim, A.rope_theta,
                                       A.softmax_scale)
    r2 = oracle.attention_layer_update(r1["pos"], r1["k_cache"], r1["v_cache"], rounds[1][0], r1["cursor"], *at,
                                       A.rdim, A.rope_theta, A.softmax_scale, live=r1["pos"])
    assert_close(ao2.cpu().numpy(), r2["out"], "restored update: attention")
    d0 = synth.gen_delta_inputs(seed, 401, 1, rounds[0][1], D, rnd=0)
    _, S1 = oracle.delta_layer_update(a.S0.astype(np.float64), *d0[:3], d0[3], d0[4], D.scale)
    o2, S2 = oracle.delta_layer_update(S1, *dt[:3], dt[3], dt[4], D.scale)
    assert_close(do2.cpu().numpy(), o2, "restored update: delta out")
    assert_close(b.S.cpu().numpy(), S2, "restored update: delta state")
