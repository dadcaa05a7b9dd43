"""Seeded randomized GPU parity of stack updates through the C ABI (MI355X only).

Each of 48 trials draws one update_layer_stack call: 1-6 contexts of 0-6,000 live rows with
0-3 removed records each and 0-700 tail tokens, one attention layer of a drawn shape
(head dims 64, 128, 256; group sizes 4 and 8) and one small delta layer, and either the
library's own key-range splits or a forced count. The draws cover single- and
multi-context launches (the wave-aware split count and the die table), merges over 1 to
64 splits, empty contexts and empty tails. Every context is checked against the float64
oracle: positions, V rows bit for bit, K rows within one bf16 ulp, sampled attention rows,
delta outputs and state.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import DEV, assert_bf16_close_bits, assert_close, bits_of, sample_rows, to_dev_bf16

pytestmark = pytest.mark.gpu

SHAPES = [synth.AttnShape(16, 2, 256), synth.AttnShape(8, 2, 128), synth.AttnShape(4, 1, 64)]
DSHAPE = synth.DeltaShape(2, 4, 64, 64, 32)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


@pytest.mark.parametrize("trial", range(48))
def test_random_stack_update(trial):
    rng = np.random.default_rng(9000 + trial)
    A = SHAPES[trial % len(SHAPES)]
    n_ctx = int(rng.integers(1, 7))
    splits = int(rng.choice([0, 0, 0, 3, 17, 64]))
    specs = []
    for c in range(n_ctx):
        L = int(rng.choice([0, int(rng.integers(1, 6001))], p=[0.15, 0.85]))
        iv = synth.initial_intervals(L) if L else []
        n_rec = int(rng.integers(0, 4)) if L > 400 else 0
        # records of up to 300 rows, shorter where n_rec of them would not fit
        ranges = (synth.draw_records(rng, iv, n_rec, (1, min(300, L // (n_rec + 1)))) if n_rec
                  else np.zeros((0, 2), np.int64))
        T = int(rng.choice([0, int(rng.integers(1, 701))], p=[0.15, 0.85]))
        specs.append((L, ranges, T))
    if all(T == 0 for _, _, T in specs):
        specs[0] = (specs[0][0], specs[0][1], 5)
    print(f"[case] trial {trial}: shape {A}, splits {splits}, contexts "
          f"{[(L, r.tolist(), T) for L, r, T in specs]}", flush=True)
    ctxs, kcs, vcs, host, states = [], [], [], [], []
    for c, (L, ranges, T) in enumerate(specs):
        cap = max(1, L + T)
        kb, vb = synth.gen_attn_cache(trial, 300, 0, L, A, char=c)
        kc = np.zeros((cap, A.n_kv_heads, A.head_dim), np.uint16)
        vc = np.zeros_like(kc)
        kc[:L], vc[:L] = kb, vb
        kcs.append(to_dev_bf16(kc))
        vcs.append(to_dev_bf16(vc))
        ctx = tu.Context(cap, device=DEV)
        if L:
            ctx.pos[:L] = torch.arange(L, dtype=torch.int32, device=DEV)
        ctx.set_metadata(synth.initial_intervals(L) if L else [], L)
        ctxs.append(ctx)
        S0 = synth.gen_delta_state(trial, 300, 1, DSHAPE, char=c)
        states.append((S0, torch.from_numpy(S0.copy()).to(DEV)))
        q, k, v = synth.gen_attn_tail(trial, 300, 0, T, A, char=c)
        dq, dk, dv, beta, g = synth.gen_delta_inputs(trial, 300, 1, T, DSHAPE, char=c)
        host.append((kb, vb, q, k, v, dq, dk, dv, beta, g))
    Ts = [T for _, _, T in specs]
    off = np.concatenate([[0], np.cumsum(Ts)]).astype(int)
    cat = lambda i: to_dev_bf16(np.concatenate([h[i] for h in host]))
    a_out = torch.full((off[-1], A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
    d_out = torch.full((off[-1], DSHAPE.n_v_heads, DSHAPE.d_v), float("nan"), dtype=torch.float32, device=DEV)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, cat(2), cat(3), cat(4), a_out, k_cache=kcs, v_cache=vcs),
              tu.LayerIO(tu.TU_LAYER_DELTA, cat(5), cat(6), cat(7), d_out, state=[s for _, s in states],
                         beta=torch.from_numpy(np.concatenate([h[8] for h in host])).to(DEV),
                         g=torch.from_numpy(np.concatenate([h[9] for h in host])).to(DEV))]
    ap = tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta, A.softmax_scale,
                        kv_splits=splits)
    dp = tu.delta_params(DSHAPE.n_k_heads, DSHAPE.n_v_heads, DSHAPE.d_k, DSHAPE.d_v, DSHAPE.chunk, DSHAPE.scale)
    up = tu.update_layer_stack(ctxs, [r for _, r, _ in specs], Ts, layers, ap, dp)
    torch.cuda.synchronize()
    for c, ((L, ranges, T), (kb, vb, q, k, v, dq, dk, dv, beta, g)) in enumerate(zip(specs, host)):
        what = f"trial {trial} context {c} (L {L}, removed {int(np.sum(ranges[:, 1] - ranges[:, 0]))}, T {T})"
        rows = sample_rows(T, 8, seed=trial * 10 + c)
        ref = oracle.attention_layer_update(np.arange(L), kb, vb, ranges, L, q, k, v, A.rdim, A.rope_theta,
                                            A.softmax_scale, rows=rows)
        n = len(ref["pos"])
        assert ctxs[c].len == n and ctxs[c].next_pos == L + T, what
        assert np.array_equal(ctxs[c].pos[:n].cpu().numpy(), ref["pos"]), what
        assert np.array_equal(bits_of(vcs[c][:n]), ref["v_cache"]), what
        assert_bf16_close_bits(bits_of(kcs[c][:n]), ref["k_cache"], f"{what}: K cache")
        if T:
            got = a_out[off[c]: off[c + 1]][torch.from_numpy(rows).to(DEV)].cpu().numpy()
            assert_close(got, ref["out"], f"{what}: attention rows")
        o_ref, S_ref = oracle.delta_layer_update(states[c][0].astype(np.float64), dq, dk, dv, beta, g, DSHAPE.scale)
        if T:
            assert_close(d_out[off[c]: off[c + 1]].cpu().numpy(), o_ref, f"{what}: delta out")
        assert_close(states[c][1].cpu().numpy(), S_ref, f"{what}: delta state")
    assert tu.workspace_faults(up.workspace) == 0
