"""GPU parity of the attention diagnostics (paper Section 5.3, Appendix C) through the
C ABI against the oracle: the float32 reference-softmax probe of the last eight rows
of a context after an update (rows in position order, and after a slot-preserving
update, in work order), averaged over two layers; memory-group and boundary-window
masses with the effective group count; total variation between two distributions,
with and without a row map, over several reduction blocks.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import DEV, assert_close, to_dev_bf16

pytestmark = pytest.mark.gpu

A = synth.AttnShape(16, 2, 256)
TIGHT = 2e-5   # fp32 softmax and sums against the oracle's float32 reference, relative


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _params():
    return tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta)


def _updated_layer(seed, layer, L_old, ranges, T, placement="tail", runs=None):
    """One attention layer of one context after an update, on the device and in the oracle."""
    cap = L_old + T
    kb, vb = synth.gen_attn_cache(seed, 1, layer, L_old, A)
    q, k, v = synth.gen_attn_tail(seed, 1, layer, T, A)
    kc = np.zeros((cap, A.n_kv_heads, A.head_dim), np.uint16)
    vc = np.zeros_like(kc)
    kc[:L_old], vc[:L_old] = kb, vb
    kc_d, vc_d = to_dev_bf16(kc), to_dev_bf16(vc)
    ctx = tu.Context(cap, device=DEV)
    ctx.pos[:L_old] = torch.arange(L_old, dtype=torch.int32, device=DEV)
    ctx.set_metadata([(0, L_old)], L_old)
    out = torch.empty((T, A.n_q_heads, A.head_dim), dtype=torch.float32, device=DEV)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), out,
                         k_cache=[kc_d], v_cache=[vc_d])]
    tu.update_layer_stack([ctx], [ranges], [T], layers, _params(), placement=[placement], place_runs=[runs])
    torch.cuda.synchronize()
    tail_pos = None if runs is None else np.concatenate([np.arange(a, b) for a, b in runs])
    ref = oracle.attention_layer_update(np.arange(L_old), kb, vb, ranges, L_old, q, k, v, A.rdim, A.rope_theta,
                                        A.softmax_scale, rows=np.zeros(0, np.int64), placement=placement,
                                        tail_positions=tail_pos)
    return ctx, kc_d, q, ref


def _oracle_probe(q, ref, n=8):
    return oracle.probe_distribution(q[-n:], ref["pos"][-n:], ref["k_cache"], A.rdim, A.rope_theta, A.softmax_scale)


def _close(got, want, what):
    assert_close(got, want, what)
    rel = np.abs(got - want).sum() / np.abs(want).sum()
    assert rel <= TIGHT, f"{what}: {rel:.3e} above the float32 agreement {TIGHT:.0e}"


@pytest.mark.parametrize("placement", ["tail", "slot"])
def test_probe_distribution_two_layers(placement):
    ranges = np.array([[400, 528], [1500, 1628]])
    runs = [(400, 528), (1500, 1628), (9000, 9044)] if placement == "slot" else None
    _say(f"probe of the last 8 rows, two layers, placement {placement}")
    p_dev, p_ref = None, np.zeros(0)
    for layer in (0, 4):
        ctx, kc, q, ref = _updated_layer(30, layer, 2600, ranges, 300, placement, runs)
        if p_dev is None:
            p_dev = torch.zeros(ctx.len, dtype=torch.float32, device=DEV)
            p_ref = np.zeros(ctx.len)
        tu.attention_probe(ctx, kc, _params(), to_dev_bf16(q[-8:]), p_dev, weight=0.5)
        p_ref += 0.5 * _oracle_probe(q, ref)
    torch.cuda.synchronize()
    got = p_dev.cpu().numpy().astype(np.float64)
    assert abs(got.sum() - 1.0) < 1e-4
    _close(got, p_ref, f"probe distribution ({placement})")


@pytest.mark.parametrize("hq,hkv,d,rdim,n,L", [
    (8, 4, 128, 64, 5, 1000),     # 10 rows per KV head: one ragged row tile
    (16, 1, 64, 64, 8, 333),      # 128 rows: four row tiles, two tasks per wave
    (4, 4, 256, 256, 1, 64),      # one row per KV head, one key tile
    (8, 2, 64, 32, 5, 5),         # every row a probe row: the first sees only row 0
    (16, 2, 128, 128, 10, 700),   # 80 rows per KV head: three row tiles, one wave idle
])
def test_probe_shapes(hq, hkv, d, rdim, n, L):
    """Other head shapes on a context with a hole in its positions, keys and queries
    scaled so that the softmax rows are peaked."""
    _say(f"probe shape Hq={hq} Hkv={hkv} D={d} rotary={rdim} n={n} len={L}")
    rng = np.random.default_rng(50 + d + n)
    k = synth.to_bf16_bits(rng.normal(0.0, 2.0, (L, hkv, d)))
    q = synth.to_bf16_bits(rng.normal(0.0, 2.0, (n, hq, d)))
    cut = L // 3
    pos = np.concatenate([np.arange(cut), np.arange(cut + 700, cut + 700 + L - cut)])
    ctx = tu.Context(L, device=DEV)
    ctx.pos[:L] = torch.from_numpy(pos.astype(np.int32)).to(DEV)
    ctx.set_metadata([(0, cut), (cut + 700, int(pos[-1]) + 1)], int(pos[-1]) + 1)
    p = tu.attn_params(hq, hkv, d, rdim, 1.0e6)
    got = torch.zeros(L, dtype=torch.float32, device=DEV)
    tu.attention_probe(ctx, to_dev_bf16(k), p, to_dev_bf16(q), got)
    torch.cuda.synchronize()
    want = oracle.probe_distribution(q, pos[-n:], k, rdim, 1.0e6, d ** -0.5)
    got = got.cpu().numpy().astype(np.float64)
    assert abs(got.sum() - 1.0) < 1e-4
    _close(got, want, f"probe distribution Hq={hq} Hkv={hkv} D={d} n={n}")


@pytest.mark.parametrize("trial", range(12))
def test_probe_random(trial):
    """Seeded draws of the probe's shape: KV heads 1-4, group size 1-16 (at most 128 rows
    per KV head), head dim 64-256 with full or half rotary, 1-16 probe rows, contexts of
    up to 3,000 rows in 1-4 live runs, queries and keys of scale 0.5-3."""
    rng = np.random.default_rng(7000 + trial)
    d = int(rng.choice([64, 128, 256]))
    rdim = int(rng.choice([d, d // 2]))
    hkv = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 4, 8, 16]))
    n = int(rng.integers(1, min(16, 128 // G) + 1))
    L = int(rng.integers(n, 3001))
    runs = int(rng.integers(1, 5))
    cuts = np.sort(rng.choice(np.arange(1, L), size=min(runs - 1, L - 1), replace=False)) if L > 1 else []
    sizes = np.diff(np.concatenate([[0], cuts, [L]])).astype(int)
    pos, iv, at = [], [], 0
    for r, sz in enumerate(sizes):
        at += int(rng.integers(0 if r == 0 else 1, 5000))   # a hole before the run (runs never touch)
        pos.append(np.arange(at, at + sz))
        iv.append((at, at + int(sz)))
        at += int(sz)
    pos = np.concatenate(pos).astype(np.int64)
    sc = float(rng.uniform(0.5, 3.0))
    _say(f"probe trial {trial}: Hq={hkv * G} Hkv={hkv} D={d} rotary={rdim} n={n} len={L} runs={len(iv)}")
    k = synth.to_bf16_bits(rng.normal(0.0, sc, (L, hkv, d)))
    q = synth.to_bf16_bits(rng.normal(0.0, sc, (n, hkv * G, d)))
    ctx = tu.Context(L, device=DEV)
    ctx.pos[:L] = torch.from_numpy(pos.astype(np.int32)).to(DEV)
    ctx.set_metadata(iv, at)
    got = torch.zeros(L, dtype=torch.float32, device=DEV)
    tu.attention_probe(ctx, to_dev_bf16(k), tu.attn_params(hkv * G, hkv, d, rdim, 1.0e6), to_dev_bf16(q), got)
    torch.cuda.synchronize()
    want = oracle.probe_distribution(q, pos[-n:], k, rdim, 1.0e6, d ** -0.5)
    got = got.cpu().numpy().astype(np.float64)
    assert abs(got.sum() - 1.0) < 1e-4
    _close(got, want, f"probe distribution, trial {trial}")


def test_probe_long_context():
    """100,003 rows at the 16/2 x 256 attention shape, 8 probe rows: 3,126 (KV head,
    key tile) items, several per workgroup of the streaming passes, so the prefetch of
    the next tile and the walk over items run, with a ragged last tile."""
    rng = np.random.default_rng(62)
    L, hq, hkv, d, n = 100_003, 16, 2, 256, 8
    _say(f"probe over {L} rows, Hq={hq} Hkv={hkv} D={d} n={n}")
    k = synth.to_bf16_bits(rng.normal(0.0, 1.5, (L, hkv, d)))
    q = synth.to_bf16_bits(rng.normal(0.0, 1.5, (n, hq, d)))
    pos = np.concatenate([np.arange(40_000), np.arange(40_500, 40_500 + L - 40_000)]).astype(np.int64)
    ctx = tu.Context(L, device=DEV)
    ctx.pos[:L] = torch.from_numpy(pos.astype(np.int32)).to(DEV)
    ctx.set_metadata([(0, 40_000), (40_500, int(pos[-1]) + 1)], int(pos[-1]) + 1)
    got = torch.zeros(L, dtype=torch.float32, device=DEV)
    tu.attention_probe(ctx, to_dev_bf16(k), tu.attn_params(hq, hkv, d, d, 1.0e7), to_dev_bf16(q), got)
    torch.cuda.synchronize()
    want = oracle.probe_distribution(q, pos[-n:], k, d, 1.0e7, d ** -0.5)
    got = got.cpu().numpy().astype(np.float64)
    assert abs(got.sum() - 1.0) < 1e-4
    _close(got, want, "probe distribution, 100,003 rows")


def test_group_masses_and_summary():
    ranges = np.array([[100, 228]])
    ctx, kc, q, ref = _updated_layer(31, 0, 3000, ranges, 200)
    p_dev = torch.zeros(ctx.len, dtype=torch.float32, device=DEV)
    tu.attention_probe(ctx, kc, _params(), to_dev_bf16(q[-8:]), p_dev)
    p_ref = _oracle_probe(q, ref)
    # 600 records of 5 positions each plus one holding the removed range and the tail
    groups = [(5 * g, 5 * g + 5) for g in range(600)] + [(3000, 3200)]
    _say(f"group masses of {len(groups)} groups (several launches of 256)")
    mass, win, summary = tu.attention_group_mass(ctx, p_dev, groups, window=3)
    torch.cuda.synchronize()
    m_ref, w_ref = oracle.group_masses(p_ref, ref["pos"], groups, window=3)
    _close(mass.cpu().numpy().astype(np.float64), m_ref, "group masses")
    _close(win.cpu().numpy().astype(np.float64), w_ref, "boundary-window masses")
    s_ref = np.array(oracle.group_summary(m_ref, w_ref))
    _close(summary.cpu().numpy().astype(np.float64), s_ref, "memory mass, effective count, window share")
    assert float(mass[20:26].sum()) == 0.0      # groups of removed positions hold no rows


def test_group_masses_many_workgroups():
    """300,001 rows in shuffled position order (every group-mass workgroup takes several
    rounds, the launch its maximum number of workgroups), 300 groups over part of the
    positions (two launches of groups), window 5: against the
    oracle, and the same bits on a second call."""
    rng = np.random.default_rng(60)
    n = 300_001
    pos = rng.permutation(n).astype(np.int64) + 7          # one live run, rows in shuffled order
    ctx = tu.Context(n, device=DEV)
    ctx.pos[:n] = torch.from_numpy(pos.astype(np.int32)).to(DEV)
    ctx.set_metadata([(7, n + 7)], n + 7)
    x = rng.random(n)
    x = (x / x.sum()).astype(np.float32)
    cuts = np.sort(rng.choice(np.arange(0, n + 20), size=600, replace=False))
    groups = [(int(cuts[2 * g]), int(cuts[2 * g + 1])) for g in range(300)]
    _say(f"group masses of {len(groups)} groups over {n} shuffled rows")
    p_dev = torch.from_numpy(x).to(DEV)
    mass, win, summary = tu.attention_group_mass(ctx, p_dev, groups, window=5)
    mass2, win2, summary2 = tu.attention_group_mass(ctx, p_dev, groups, window=5)
    torch.cuda.synchronize()
    m_ref, w_ref = oracle.group_masses(x, pos, groups, window=5)
    _close(mass.cpu().numpy().astype(np.float64), m_ref, "group masses, many workgroups")
    _close(win.cpu().numpy().astype(np.float64), w_ref, "boundary-window masses, many workgroups")
    s_ref = np.array(oracle.group_summary(m_ref, w_ref))
    _close(summary.cpu().numpy().astype(np.float64), s_ref, "summary, many workgroups")
    assert torch.equal(mass, mass2) and torch.equal(win, win2) and torch.equal(summary, summary2)


def test_group_masses_edge_cases():
    """Window 0 (no boundary window), a group over the hole in the positions (no row), a
    group past the last position, and rows in no group (memory mass below 1)."""
    rng = np.random.default_rng(61)
    n = 700
    pos = np.concatenate([np.arange(300), np.arange(900, 1300)]).astype(np.int64)
    ctx = tu.Context(n, device=DEV)
    ctx.pos[:n] = torch.from_numpy(pos.astype(np.int32)).to(DEV)
    ctx.set_metadata([(0, 300), (900, 1300)], 1300)
    x = rng.random(n)
    x = (x / x.sum()).astype(np.float32)
    groups = [(10, 120), (300, 900), (905, 1000), (1000, 1250), (1300, 1400)]
    p_dev = torch.from_numpy(x).to(DEV)
    mass, win, summary = tu.attention_group_mass(ctx, p_dev, groups, window=0)
    torch.cuda.synchronize()
    m_ref, w_ref = oracle.group_masses(x, pos, groups, window=0)
    _close(mass.cpu().numpy().astype(np.float64), m_ref, "group masses, edge cases")
    assert float(mass[1]) == 0.0 and float(mass[4]) == 0.0
    assert float(win.abs().sum()) == 0.0 and float(summary[2]) == 0.0
    s_ref = np.array(oracle.group_summary(m_ref, w_ref))
    assert s_ref[0] < 0.95
    _close(summary.cpu().numpy().astype(np.float64), s_ref, "summary, edge cases")


def test_total_variation():
    ranges = np.array([[700, 828]])
    ctx_a, kc_a, q_a, ref_a = _updated_layer(32, 0, 2400, ranges, 150)
    ctx_b, kc_b, q_b, ref_b = _updated_layer(32, 8, 2400, ranges, 150)
    pa = torch.zeros(ctx_a.len, dtype=torch.float32, device=DEV)
    pb = torch.zeros(ctx_b.len, dtype=torch.float32, device=DEV)
    tu.attention_probe(ctx_a, kc_a, _params(), to_dev_bf16(q_a[-8:]), pa)
    tu.attention_probe(ctx_b, kc_b, _params(), to_dev_bf16(q_b[-8:]), pb)
    ra, rb = _oracle_probe(q_a, ref_a), _oracle_probe(q_b, ref_b)
    tv = tu.attention_tv_distance(pa, pb)
    perm = np.random.default_rng(3).permutation(ctx_a.len)
    pb_perm = torch.empty_like(pb)
    pb_perm[torch.from_numpy(perm).to(DEV)] = pb                  # row j of pb sits at perm[j]
    tv_map = tu.attention_tv_distance(pa, pb_perm, torch.from_numpy(perm.astype(np.int32)).to(DEV))
    torch.cuda.synchronize()
    want = oracle.tv_distance(ra, rb)
    _say(f"total variation {float(tv[0]):.6f} (oracle {want:.6f})")
    assert abs(float(tv[0]) - want) <= TIGHT * want
    assert float(tv_map[0]) == float(tv[0])
    # many reduction blocks: random distributions over 300,001 rows
    rng = np.random.default_rng(4)
    x, y = rng.random(300_001), rng.random(300_001)
    x, y = (x / x.sum()).astype(np.float32), (y / y.sum()).astype(np.float32)
    big = tu.attention_tv_distance(torch.from_numpy(x).to(DEV), torch.from_numpy(y).to(DEV))
    torch.cuda.synchronize()
    want = oracle.tv_distance(x, y)
    assert abs(float(big[0]) - want) <= 1e-6 * want
