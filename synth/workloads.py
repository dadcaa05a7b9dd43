"""Workload shapes and seeded input draws for the true-tail update.

The five workloads mirror the maintenance settings the paper describes
(Section 5.1: one character with a long cached prefix; Section 6.6 and
Appendix B: eight scripted revision rounds that remove records and append
replacements at the tail), at the sizes of the five benchmark configurations:

  0  tiny attention + delta pair (L_old 256, 4 runs of 4 removed, T 32)
  1  single-character refresh (L_keep 8192, 3 x 128 removed, T 512)
  2  long-lived character, 8 rounds from a 32K context
  3  population batch of 32 characters (L_keep U[4096,16384], T U[128,512])
  4  48-layer hybrid stack (12 attention + 36 delta), 64K context, T 2048

Value distributions (all draws float64, then rounded once to float32 and,
for bf16 tensors, once more from float32 to bf16 round-to-nearest-even):
  q, k, v          ~ N(0, 1)
  delta-rule k     L2-normalised per (token, head)
  beta             = sigmoid(N(0, 1))
  g (decay gate)   = exp(-softplus(N(-4, 1)))
  carried state S  ~ N(0, 0.1^2)

Cached attention keys are drawn directly as N(0,1) bf16 rows: a rotary
position rotation maps an isotropic Gaussian vector to an isotropic Gaussian
vector, so rotated and unrotated cached keys have the same distribution.

Every tensor has its own generator, seeded with
``[seed, cfg, layer, tensor_id, round, char]``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

# tensor ids for sub-seeding
T_KCACHE, T_VCACHE, T_Q, T_K, T_V, T_BETA, T_G, T_STATE, T_PLAN, T_CONV_X, T_CONV_STATE, T_CONV_W = range(12)


@dataclass(frozen=True)
class AttnShape:
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float = 1.0e7
    rotary_dim: Optional[int] = None  # None -> head_dim

    @property
    def rdim(self) -> int:
        return self.head_dim if self.rotary_dim is None else self.rotary_dim

    @property
    def softmax_scale(self) -> float:
        return float(self.head_dim) ** -0.5


@dataclass(frozen=True)
class DeltaShape:
    n_k_heads: int
    n_v_heads: int
    d_k: int
    d_v: int
    chunk: int

    @property
    def scale(self) -> float:
        return float(self.d_k) ** -0.5


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    attn: AttnShape
    delta: DeltaShape
    n_layers: int            # total layers of the stack
    attn_every: int          # layer l is attention iff l % attn_every == attn_every - 1
    n_chars: int
    n_rounds: int
    # per-character prefix: either a fixed L_old, or fixed/drawn L_keep
    L_old: Optional[int] = None
    L_keep: Optional[int] = None
    L_keep_range: Optional[Tuple[int, int]] = None
    # records removed per round
    n_records: Tuple[int, int] = (0, 0)       # inclusive range
    record_len: Tuple[int, int] = (0, 0)      # inclusive range
    # tail tokens per round
    tail: Tuple[int, int] = (0, 0)            # inclusive range

    def layer_kinds(self) -> List[str]:
        if self.n_layers == 2:
            return ["attn", "delta"]
        return ["attn" if (l % self.attn_every) == self.attn_every - 1 else "delta"
                for l in range(self.n_layers)]


_A1 = AttnShape(16, 2, 256)
_D1 = DeltaShape(16, 32, 128, 128, 64)

CONFIGS = {
    0: Config(0, "tiny attention+delta pair", AttnShape(2, 1, 64), DeltaShape(2, 2, 64, 64, 16),
              n_layers=2, attn_every=2, n_chars=1, n_rounds=1, L_old=256,
              n_records=(4, 4), record_len=(4, 4), tail=(32, 32)),
    1: Config(1, "single-character refresh", _A1, _D1, n_layers=2, attn_every=2,
              n_chars=1, n_rounds=1, L_keep=8192, n_records=(3, 3), record_len=(128, 128),
              tail=(512, 512)),
    2: Config(2, "long-lived character, 8 maintenance rounds", _A1, _D1, n_layers=2,
              attn_every=2, n_chars=1, n_rounds=8, L_old=32768, n_records=(1, 4),
              record_len=(64, 256), tail=(256, 1024)),
    3: Config(3, "population batch of 32 characters", _A1, _D1, n_layers=2, attn_every=2,
              n_chars=32, n_rounds=1, L_keep_range=(4096, 16384), n_records=(0, 4),
              record_len=(64, 64), tail=(128, 512)),
    4: Config(4, "48-layer hybrid stack, 64K context", _A1, _D1, n_layers=48, attn_every=4,
              n_chars=1, n_rounds=1, L_old=65536, n_records=(8, 8), record_len=(256, 256),
              tail=(2048, 2048)),
}


# Tail-length sweep at a 32K surviving context (one 64-token record removed): short tails
# are decode-like and bound by reading the cache, long ones by the attention products.
T_SWEEP = (1, 8, 32, 128, 512, 2048)


def t_sweep_config(T: int) -> Config:
    return Config(100 + T_SWEEP.index(T), f"tail sweep, T = {T} at 32K surviving rows", _A1, _D1, n_layers=2,
                  attn_every=2, n_chars=1, n_rounds=1, L_keep=32768, n_records=(1, 1), record_len=(64, 64),
                  tail=(T, T))


def sub_rng(seed: int, cfg: int, layer: int, tensor_id: int, rnd: int = 0, char: int = 0):
    return np.random.default_rng([int(seed), int(cfg), int(layer), int(tensor_id), int(rnd), int(char)])


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64/float32 array -> bf16 bit patterns (uint16), rounded once from float32."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _normal(rng, shape, mean=0.0, std=1.0):
    return rng.normal(mean, std, size=shape)


# ----------------------------------------------------------------------------- tensors

def gen_attn_cache(seed: int, cfg: int, layer: int, L: int, shape: AttnShape, char: int = 0):
    """Cached (already rotated) K and V rows, bf16 bits, [L][Hkv][D]."""
    hk = (L, shape.n_kv_heads, shape.head_dim)
    k = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_KCACHE, 0, char), hk))
    v = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_VCACHE, 0, char), hk))
    return k, v


def gen_attn_tail(seed: int, cfg: int, layer: int, T: int, shape: AttnShape, rnd: int = 0,
                  char: int = 0):
    """Pre-rotation tail q [T][Hq][D], k, v [T][Hkv][D] as bf16 bits."""
    q = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_Q, rnd, char),
                             (T, shape.n_q_heads, shape.head_dim)))
    k = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_K, rnd, char),
                             (T, shape.n_kv_heads, shape.head_dim)))
    v = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_V, rnd, char),
                             (T, shape.n_kv_heads, shape.head_dim)))
    return q, k, v


def gen_delta_state(seed: int, cfg: int, layer: int, shape: DeltaShape, char: int = 0):
    """Carried fp32 state S [Hv][d_v][d_k] ~ N(0, 0.1^2)."""
    s = _normal(sub_rng(seed, cfg, layer, T_STATE, 0, char), (shape.n_v_heads, shape.d_v, shape.d_k),
                std=0.1)
    return s.astype(np.float32)


def gen_delta_inputs(seed: int, cfg: int, layer: int, T: int, shape: DeltaShape, rnd: int = 0,
                     char: int = 0):
    """Tail inputs of one gated delta-rule layer.

    q, k: bf16 bits [T][Hk][d_k] (k L2-normalised per token and head before rounding);
    v: bf16 bits [T][Hv][d_v]; beta, g: float32 [T][Hv].
    """
    q = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_Q, rnd, char), (T, shape.n_k_heads, shape.d_k)))
    kr = _normal(sub_rng(seed, cfg, layer, T_K, rnd, char), (T, shape.n_k_heads, shape.d_k))
    nrm = np.sqrt(np.sum(kr * kr, axis=-1, keepdims=True))
    k = to_bf16_bits(kr / np.maximum(nrm, 1e-30))
    v = to_bf16_bits(_normal(sub_rng(seed, cfg, layer, T_V, rnd, char), (T, shape.n_v_heads, shape.d_v)))
    b = _normal(sub_rng(seed, cfg, layer, T_BETA, rnd, char), (T, shape.n_v_heads))
    beta = (1.0 / (1.0 + np.exp(-b))).astype(np.float32)
    a = _normal(sub_rng(seed, cfg, layer, T_G, rnd, char), (T, shape.n_v_heads), mean=-4.0)
    softplus = np.log1p(np.exp(-np.abs(a))) + np.maximum(a, 0.0)
    g = np.exp(-softplus).astype(np.float32)
    return q, k, v, beta, g


# ----------------------------------------------------------------------------- records

def gen_conv_inputs(seed: int, T: int, channels: int, width: int, layer: int = 0, rnd: int = 0, char: int = 0):
    """Short-convolution inputs of one projected tensor (bf16 bits):
    x [T][channels] ~ N(0, 1) (pre-convolution projections), the carried rows
    [width-1][channels] ~ N(0, 1) (earlier inputs of the same tensor), weights
    [channels][width] ~ N(0, 1/width)."""
    x = to_bf16_bits(_normal(sub_rng(seed, 0, layer, T_CONV_X, rnd, char), (T, channels)))
    st = to_bf16_bits(_normal(sub_rng(seed, 0, layer, T_CONV_STATE, 0, char), (width - 1, channels)))
    w = to_bf16_bits(_normal(sub_rng(seed, 0, layer, T_CONV_W, 0, char), (channels, width), std=width ** -0.5))
    return st, x, w


def initial_intervals(L_old: int) -> List[Tuple[int, int]]:
    return [(0, int(L_old))] if L_old > 0 else []


def subtract_ranges(intervals: Sequence[Tuple[int, int]], ranges) -> List[Tuple[int, int]]:
    """Live position intervals after removing half-open position ranges (bookkeeping)."""
    out: List[Tuple[int, int]] = []
    rs = sorted((int(a), int(b)) for a, b in ranges)
    for (s, e) in intervals:
        cur = s
        for (a, b) in rs:
            if b <= cur or a >= e:
                continue
            if a > cur:
                out.append((cur, a))
            cur = max(cur, b)
        if cur < e:
            out.append((cur, e))
    return out


def append_interval(intervals: List[Tuple[int, int]], begin: int, T: int) -> List[Tuple[int, int]]:
    out = list(intervals)
    if T <= 0:
        return out
    if out and out[-1][1] == begin:
        out[-1] = (out[-1][0], begin + T)
    else:
        out.append((begin, begin + T))
    return out


def draw_records(rng, intervals: Sequence[Tuple[int, int]], n: int, len_range: Tuple[int, int],
                 max_tries: int = 100000) -> np.ndarray:
    """Draw n removal records: runs of live positions with no hole inside.

    Draw order: for each record, its length (inclusive range), then its start,
    uniform over [min live, max live end - len], rejected until the run lies in
    one live interval and does not overlap an earlier record. Returns int64 [n, 2]
    half-open position ranges sorted by start.
    """
    if n == 0:
        return np.zeros((0, 2), dtype=np.int64)
    lo = intervals[0][0]
    hi = intervals[-1][1]
    chosen: List[Tuple[int, int]] = []
    for _ in range(n):
        ln = int(rng.integers(len_range[0], len_range[1] + 1))
        for _try in range(max_tries):
            a = int(rng.integers(lo, hi - ln + 1))
            b = a + ln
            inside = any(s <= a and b <= e for (s, e) in intervals)
            clash = any(not (b <= c or a >= d) for (c, d) in chosen)
            if inside and not clash:
                chosen.append((a, b))
                break
        else:
            raise RuntimeError("could not place a record")
    chosen.sort()
    return np.asarray(chosen, dtype=np.int64).reshape(-1, 2)


# ----------------------------------------------------------------------------- scenarios

@dataclass
class Round:
    ranges: np.ndarray     # int64 [n, 2] removal ranges in position space
    T: int                 # tail tokens appended at the cursor
    cursor: int            # cursor (next position id) before the round
    L_old: int             # live rows before the removal
    L_keep: int            # live rows after the removal
    intervals: List[Tuple[int, int]] = field(default_factory=list)  # live intervals before


@dataclass
class CharacterPlan:
    L_initial: int
    rounds: List[Round]


@dataclass
class Scenario:
    cfg: Config
    seed: int
    chars: List[CharacterPlan]


def make_scenario(cfg_index: int, seed: int = 0, n_rounds: Optional[int] = None,
                  n_chars: Optional[int] = None, cfg: Optional[Config] = None) -> Scenario:
    """Removal ranges and tail lengths for every character and round of a workload
    (CONFIGS[cfg_index], or `cfg` when given, whose index then seeds the draws)."""
    if cfg is None:
        cfg = CONFIGS[cfg_index]
    cfg_index = cfg.index
    R = cfg.n_rounds if n_rounds is None else n_rounds
    C = cfg.n_chars if n_chars is None else n_chars
    chars: List[CharacterPlan] = []
    for ch in range(C):
        rng = sub_rng(seed, cfg_index, 0, T_PLAN, 0, ch)
        # the first round's record count and lengths fix L_old when L_keep is given
        if cfg.L_old is not None:
            L0 = cfg.L_old
            first_n = None
        else:
            L_keep = cfg.L_keep if cfg.L_keep is not None else int(
                rng.integers(cfg.L_keep_range[0], cfg.L_keep_range[1] + 1))
            first_n = int(rng.integers(cfg.n_records[0], cfg.n_records[1] + 1))
            # record lengths are fixed-size for the L_keep-specified configs
            assert cfg.record_len[0] == cfg.record_len[1]
            L0 = L_keep + first_n * cfg.record_len[0]
        intervals = initial_intervals(L0)
        cursor = L0
        live = L0
        rounds: List[Round] = []
        for r in range(R):
            n = first_n if (r == 0 and first_n is not None) else int(
                rng.integers(cfg.n_records[0], cfg.n_records[1] + 1))
            ranges = draw_records(rng, intervals, n, cfg.record_len)
            T = int(rng.integers(cfg.tail[0], cfg.tail[1] + 1))
            removed = int(np.sum(ranges[:, 1] - ranges[:, 0])) if len(ranges) else 0
            rounds.append(Round(ranges=ranges, T=T, cursor=cursor, L_old=live,
                                L_keep=live - removed, intervals=list(intervals)))
            intervals = append_interval(subtract_ranges(intervals, ranges), cursor, T)
            live = live - removed + T
            cursor += T
        chars.append(CharacterPlan(L_initial=L0, rounds=rounds))
    return Scenario(cfg=cfg, seed=seed, chars=chars)


# ----------------------------------------------------------------------------- paper-shaped trace

@dataclass
class Revision:
    ranges: np.ndarray                 # int64 [n, 2] position ranges of the records removed
    runs: List[Tuple[int, int]]        # tail positions as runs, in tail order (framing included)
    post: np.ndarray                   # int64 [k, 2] framing positions removed after the tail
    T: int                             # tail tokens: replacement records + framing
    m: int                             # replacement-record tokens
    cursor: int                        # next position id before the revision
    cursor_after: int                  # after it (one past the highest position in use)
    L_old: int                         # live rows before
    intervals: List[Tuple[int, int]]   # live position runs (row order) before


@dataclass
class PaperTrace:
    positions: np.ndarray              # int64 [L0] position of every initial row (row order)
    intervals: List[Tuple[int, int]]   # initial live runs
    cursor: int
    revisions: List[Revision]
    interval: int


def make_paper_trace(seed: int = 0, head: int = 1699, n_records: int = 26, record_len=(330, 450),
                     interval: int = 10000, n_revisions: int = 8, m_range=(214, 362), framing=(5, 6),
                     index: int = 200) -> PaperTrace:
    """A revision trace shaped like the paper's measured one (Sections 5.2 and 6.6, Table 1): a common
    head at positions [0, head), then records of about 390 tokens, record k at the start
    of its own `interval`-position slot (logical positions, not occupied rows); every
    revision removes one or two whole records and appends as many replacement records
    (m tokens in all) at fresh slots past the cursor (the next slot boundary at or above
    it), framed by `framing` delimiter tokens that are removed again after the tail is
    processed. The cursor then is one past the highest position in use.

    Draw order per revision: the number of records removed (1 or 2), which live records
    (uniform, without replacement), m (inclusive range), the split of m over the new
    records (uniform cut). Positions of the tail: the opening delimiters and the first
    record share the first fresh slot, each further record takes the next slot, the
    closing delimiters follow the last record."""
    rng = sub_rng(seed, index, 0, T_PLAN)
    lens = rng.integers(record_len[0], record_len[1] + 1, size=n_records)
    recs = [(interval * (k + 1), interval * (k + 1) + int(lens[k])) for k in range(n_records)]
    positions = np.concatenate([np.arange(head)] + [np.arange(a, b) for a, b in recs]).astype(np.int64)
    intervals = [(0, head)] + list(recs)
    initial = list(intervals)
    cursor = interval * (n_records + 1)
    live = len(positions)
    revisions: List[Revision] = []
    for _ in range(n_revisions):
        n = int(rng.integers(1, 3))
        pick = sorted(int(i) for i in rng.choice(len(recs), size=n, replace=False))
        gone = [recs[i] for i in pick]
        m = int(rng.integers(m_range[0], m_range[1] + 1))
        cuts = sorted(int(c) for c in rng.integers(1, m, size=n - 1)) if n > 1 else []
        new_lens = [b - a for a, b in zip([0] + cuts, cuts + [m])]
        runs, new_recs, post = [], [], []
        base = -(-cursor // interval) * interval      # the next free slot boundary
        for j, ln in enumerate(new_lens):
            a = base + interval * j
            lead = framing[0] if j == 0 else 0
            trail = framing[1] if j == n - 1 else 0
            runs.append((a, a + lead + ln + trail))
            new_recs.append((a + lead, a + lead + ln))
            if lead:
                post.append((a, a + lead))
            if trail:
                post.append((a + lead + ln, a + lead + ln + trail))
        T = m + framing[0] + framing[1]
        cursor_after = runs[-1][1]                     # one past the highest position in use
        ranges = np.asarray(sorted(gone), dtype=np.int64).reshape(-1, 2)
        revisions.append(Revision(ranges=ranges, runs=runs, post=np.asarray(post, dtype=np.int64).reshape(-1, 2),
                                  T=T, m=m, cursor=cursor, cursor_after=cursor_after, L_old=live,
                                  intervals=list(intervals)))
        intervals = subtract_ranges(intervals, ranges) + list(new_recs)
        recs = [r for i, r in enumerate(recs) if i not in pick] + new_recs
        live = live - sum(b - a for a, b in gone) + m
        cursor = cursor_after
    return PaperTrace(positions=positions, intervals=initial, cursor=interval * (n_records + 1),
                      revisions=revisions, interval=interval)
