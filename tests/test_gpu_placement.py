"""GPU parity of the placement variants (paper Section 5.2, compared in Section 6.3)
and of key relocation, through the C ABI, against the float64 oracle.

  * slot-preserving: the replacement is rotated at the removed records' positions
    (plus a free range) while computed after every surviving row; rows keep those
    positions, so the cache is no longer in position order;
  * a later true-tail update of that context: compaction by position over rows in
    work order;
  * tail-and-relocate: computed at the true tail, then the stored keys are rotated
    to the slot and relabelled, with maintenance delimiters removed by their final
    positions;
  * relocate_keys on its own, with a move whose positions sit in two runs.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2609_18935_amd as tu
from gpu_cases import DEV, assert_bf16_close_bits, assert_close, bits_of, to_dev_bf16

pytestmark = pytest.mark.gpu

A = synth.AttnShape(16, 2, 256)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tu.lib()


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _runs_of(positions):
    out = []
    for p in np.asarray(positions).tolist():
        if out and out[-1][1] == p:
            out[-1] = (out[-1][0], p + 1)
        else:
            out.append((p, p + 1))
    return out


class Ctx:
    """A context on the device with its host-side oracle twin."""

    def __init__(self, seed, L_old, cap, layer=0):
        self.k_h, self.v_h = synth.gen_attn_cache(seed, 1, layer, L_old, A)
        self.pos_h = np.arange(L_old, dtype=np.int64)
        self.cursor = L_old
        kc = np.zeros((cap, A.n_kv_heads, A.head_dim), np.uint16)
        vc = np.zeros_like(kc)
        kc[:L_old], vc[:L_old] = self.k_h, self.v_h
        self.kc, self.vc = to_dev_bf16(kc), to_dev_bf16(vc)
        self.ctx = tu.Context(cap, device=DEV)
        self.ctx.pos[:L_old] = torch.arange(L_old, dtype=torch.int32, device=DEV)
        self.ctx.set_metadata([(0, L_old)], L_old)

    def update(self, seed, rnd, T, ranges, placement="tail", runs=None, post=None):
        q, k, v = synth.gen_attn_tail(seed, 1, 0, T, A, rnd=rnd)
        out = torch.full((T, A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
        layers = [tu.LayerIO(tu.TU_LAYER_ATTN, to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), out,
                             k_cache=[self.kc], v_cache=[self.vc])]
        tu.update_layer_stack([self.ctx], [ranges], [T], layers,
                              tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta),
                              post_ranges=[post], placement=[placement], place_runs=[runs])
        torch.cuda.synchronize()
        tail_pos = None if runs is None else np.concatenate([np.arange(a, b) for a, b in runs])
        ref = oracle.attention_layer_update(self.pos_h, self.k_h, self.v_h, ranges, self.cursor, q, k, v, A.rdim,
                                            A.rope_theta, A.softmax_scale, live=self.pos_h.tolist(),
                                            post_ranges=post, placement=placement, tail_positions=tail_pos)
        self.pos_h, self.k_h, self.v_h, self.cursor = ref["pos"], ref["k_cache"], ref["v_cache"], ref["cursor"]
        return out, ref

    def check(self, what):
        n = len(self.pos_h)
        assert self.ctx.len == n, f"{what}: length"
        assert self.ctx.next_pos == self.cursor, f"{what}: cursor"
        assert np.array_equal(self.ctx.pos[:n].cpu().numpy(), self.pos_h), f"{what}: positions"
        assert self.ctx.intervals() == _runs_of(self.pos_h), f"{what}: live runs"
        assert np.array_equal(bits_of(self.vc[:n]), self.v_h), f"{what}: V cache"
        assert_bf16_close_bits(bits_of(self.kc[:n]), self.k_h, f"{what}: K cache")


def test_slot_placement_then_true_tail_update():
    c = Ctx(21, 3000, 3600)
    ranges = np.array([[700, 828], [2100, 2228]])
    runs = [(700, 828), (2100, 2228), (4000, 4044)]      # the two slots, then a free range
    _say(f"slot placement: ranges {ranges.tolist()}, runs {runs}, T 300")
    out, ref = c.update(21, 0, 300, ranges, "slot", runs)
    assert_close(out.cpu().numpy(), ref["out"], "slot-placed attention")
    c.check("after slot placement")
    assert c.ctx.next_pos == 4044
    # a true-tail update of the same context: its rows are no longer in position order;
    # one range takes slot-placed rows (at the end of the cache), one a surviving run
    # and one a range whose positions sit in two runs that are not row-adjacent
    ranges2 = np.array([[690, 720], [1500, 1564], [2200, 2250]])
    _say(f"true-tail update after it: ranges {ranges2.tolist()}, T 200")
    out2, ref2 = c.update(21, 1, 200, ranges2)
    assert_close(out2.cpu().numpy(), ref2["out"], "true-tail attention over work-ordered rows")
    c.check("after the true-tail update")


def test_relocate_placement_with_delimiters():
    c = Ctx(22, 2500, 3200)
    ranges = np.array([[300, 556], [1800, 1900]])
    runs = [(300, 556), (1800, 1900), (9000, 9044)]      # T = 400
    post = np.array([[300, 311], [9041, 9044]])          # delimiters, by their final positions
    _say(f"tail-and-relocate: ranges {ranges.tolist()}, runs {runs}, post {post.tolist()}")
    out, ref = c.update(22, 0, 400, ranges, "relocate", runs, post)
    assert_close(out.cpu().numpy(), ref["out"], "attention computed at the true tail")
    c.check("after relocation")
    assert c.ctx.next_pos == 9044
    out2, ref2 = c.update(22, 1, 64, np.array([[1000, 1010], [9000, 9020]]))
    assert_close(out2.cpu().numpy(), ref2["out"], "true-tail attention after a relocation")
    c.check("after the next update")


def test_relocate_keys_standalone():
    c = Ctx(23, 1200, 1400)
    out, ref = c.update(23, 0, 100, np.array([[200, 264]]), "slot", [(200, 264), (5000, 5036)])
    c.check("slot placement")
    # rows (row order): positions 0..199, 264..1199, 200..263, 5000..5035; move positions
    # 190..209 (two runs, rows not adjacent) to 7000 and the slot-placed 5000..5035 to 3000
    moves = np.array([[190, 210, 7000], [5000, 5036, 3000]])
    _say(f"relocate_keys {moves.tolist()}")
    tu.relocate_keys(c.ctx, [c.kc], tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta),
                     moves)
    torch.cuda.synchronize()
    c.pos_h, c.k_h = oracle.relocate_keys(c.pos_h, c.k_h, moves, A.rdim, A.rope_theta)
    c.cursor = max(c.cursor, 7020)
    c.check("after relocate_keys")


def test_three_placements_in_one_call():
    """One stack call over three contexts, one per placement (true tail, slot-preserving,
    tail-and-relocate with delimiters): the launch carries several contexts' position runs
    and places their attention work through the die table; each context is checked
    against its own oracle chain."""
    specs = [  # (seed, L_old, cap, T, ranges, placement, runs, post)
        (31, 2200, 2800, 250, np.array([[100, 300]]), "tail", None, None),
        (32, 3100, 3800, 330, np.array([[500, 628], [2900, 3000]]), "slot",
         [(500, 628), (2900, 3000), (7000, 7102)], None),
        (33, 1800, 2400, 180, np.array([[1000, 1100]]), "relocate", [(1000, 1100), (8000, 8080)],
         np.array([[1000, 1007], [8075, 8080]])),
    ]
    _say(f"three placements in one call: {[(s[1], s[5], s[3]) for s in specs]}")
    cs = [Ctx(seed, L, cap) for seed, L, cap, *_ in specs]
    qkv = [synth.gen_attn_tail(seed, 1, 0, T, A, rnd=0) for seed, _, _, T, *_ in specs]
    Ts = [s[3] for s in specs]
    off = np.concatenate([[0], np.cumsum(Ts)]).astype(int)
    cat = lambda i: to_dev_bf16(np.concatenate([x[i] for x in qkv]))
    out = torch.full((off[-1], A.n_q_heads, A.head_dim), float("nan"), dtype=torch.float32, device=DEV)
    layers = [tu.LayerIO(tu.TU_LAYER_ATTN, cat(0), cat(1), cat(2), out, k_cache=[c.kc for c in cs],
                         v_cache=[c.vc for c in cs])]
    tu.update_layer_stack([c.ctx for c in cs], [s[4] for s in specs], Ts, layers,
                          tu.attn_params(A.n_q_heads, A.n_kv_heads, A.head_dim, A.rdim, A.rope_theta),
                          post_ranges=[s[7] for s in specs], placement=[s[5] for s in specs],
                          place_runs=[s[6] for s in specs])
    torch.cuda.synchronize()
    for i, (c, (seed, L, cap, T, ranges, placement, runs, post), (q, k, v)) in enumerate(zip(cs, specs, qkv)):
        tail_pos = None if runs is None else np.concatenate([np.arange(a, b) for a, b in runs])
        ref = oracle.attention_layer_update(c.pos_h, c.k_h, c.v_h, ranges, c.cursor, q, k, v, A.rdim, A.rope_theta,
                                            A.softmax_scale, live=c.pos_h.tolist(), post_ranges=post,
                                            placement=placement, tail_positions=tail_pos)
        c.pos_h, c.k_h, c.v_h, c.cursor = ref["pos"], ref["k_cache"], ref["v_cache"], ref["cursor"]
        assert_close(out[off[i]: off[i + 1]].cpu().numpy(), ref["out"], f"context {i} ({placement}) attention")
        c.check(f"context {i} ({placement})")
