"""Helpers of the GPU parity tests: seeded cases on the device, oracle references
and the error metrics of the acceptance bar.

Bar (floating point): max-abs <= 2e-2 and mean-rel = sum|x - r| / sum|r| <= 1e-3
per tensor. Bit-exact for compaction indices and moved rows; appended rotated
keys within one bf16 ulp of the oracle on at most 0.1% of the elements.
"""
import numpy as np
import torch

import oracle
import synth

MAX_ABS = 2e-2
MEAN_REL = 1e-3
DEV = "cuda:0"


def to_dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def bits_of(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def errors(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = np.abs(x - ref)
    return float(d.max()) if d.size else 0.0, float(d.sum() / max(np.abs(ref).sum(), 1e-300))


def assert_close(x, ref, what=""):
    ma, mr = errors(x, ref)
    print(f"[parity] {what}: max_abs={ma:.3e} mean_rel={mr:.3e}", flush=True)
    assert ma <= MAX_ABS and mr <= MEAN_REL, f"{what}: max_abs {ma:.3e} mean_rel {mr:.3e}"


def assert_bf16_close_bits(got_bits, want_bits, what="", max_frac=1e-3):
    got = got_bits.astype(np.int32)
    want = want_bits.astype(np.int32)
    diff = np.abs(got - want)
    n_off = int(np.count_nonzero(diff))
    print(f"[parity] {what}: {n_off} of {diff.size} bf16 values differ (max {int(diff.max()) if diff.size else 0} ulp)",
          flush=True)
    assert diff.max(initial=0) <= 1, f"{what}: difference above one bf16 ulp"
    assert n_off <= max_frac * diff.size, f"{what}: too many 1-ulp differences"


class AttnCase:
    """One attention layer of one context: synthetic cache + tail, on host and device."""

    def __init__(self, shape: synth.AttnShape, seed, cfg, layer, L_old, T, capacity=None, char=0, rnd=0,
                 positions=None):
        self.shape = shape
        self.L_old, self.T = L_old, T
        self.capacity = capacity if capacity is not None else L_old + T
        self.k_bits, self.v_bits = synth.gen_attn_cache(seed, cfg, layer, L_old, shape, char)
        self.q_t, self.k_t, self.v_t = synth.gen_attn_tail(seed, cfg, layer, T, shape, rnd, char)
        self.positions = np.arange(L_old, dtype=np.int64) if positions is None else np.asarray(positions)
        Hkv, D = shape.n_kv_heads, shape.head_dim
        kc = np.zeros((self.capacity, Hkv, D), np.uint16)
        vc = np.zeros((self.capacity, Hkv, D), np.uint16)
        kc[:L_old] = self.k_bits
        vc[:L_old] = self.v_bits
        self.k_cache = to_dev_bf16(kc)
        self.v_cache = to_dev_bf16(vc)
        self.q = to_dev_bf16(self.q_t)
        self.k = to_dev_bf16(self.k_t)
        self.v = to_dev_bf16(self.v_t)
        self.out = torch.full((T, shape.n_q_heads, D), float("nan"), dtype=torch.float32, device=DEV)
        self.q_hat = torch.zeros((T, shape.n_q_heads, D), dtype=torch.bfloat16, device=DEV)

    def oracle(self, ranges, cursor, rows=None, post_ranges=None):
        s = self.shape
        return oracle.attention_layer_update(self.positions, self.k_bits, self.v_bits, ranges, cursor, self.q_t,
                                             self.k_t, self.v_t, s.rdim, s.rope_theta, s.softmax_scale, rows=rows,
                                             post_ranges=post_ranges)


class DeltaCase:
    def __init__(self, shape: synth.DeltaShape, seed, cfg, layer, T, char=0, rnd=0, state=None):
        self.shape = shape
        self.T = T
        self.S0 = synth.gen_delta_state(seed, cfg, layer, shape, char) if state is None else state
        self.q_b, self.k_b, self.v_b, self.beta, self.g = synth.gen_delta_inputs(seed, cfg, layer, T, shape, rnd, char)
        self.state = torch.from_numpy(self.S0.copy()).to(DEV)
        self.q = to_dev_bf16(self.q_b)
        self.k = to_dev_bf16(self.k_b)
        self.v = to_dev_bf16(self.v_b)
        self.beta_d = torch.from_numpy(self.beta).to(DEV)
        self.g_d = torch.from_numpy(self.g).to(DEV)
        self.out = torch.full((T, shape.n_v_heads, shape.d_v), float("nan"), dtype=torch.float32, device=DEV)

    def oracle(self):
        return oracle.delta_layer_update(self.S0.astype(np.float64), self.q_b, self.k_b, self.v_b, self.beta,
                                         self.g, self.shape.scale)


def delta_oracle_heads(S0, q_b, k_b, v_b, beta, g, scale, key_heads):
    """The per-token oracle restricted to some key heads and the value heads that read
    them (heads are independent, so this is the full oracle on a sub-shape).

    Returns (value head indices, o [T, n, d_v], S [n, d_v, d_k])."""
    Hk = q_b.shape[1]
    Hv = v_b.shape[1]
    G = Hv // Hk
    kh = np.asarray(key_heads, dtype=np.int64)
    vh = (kh[:, None] * G + np.arange(G)[None, :]).reshape(-1)
    o, S = oracle.delta_layer_update(np.asarray(S0, np.float64)[vh], q_b[:, kh], k_b[:, kh], v_b[:, vh],
                                     beta[:, vh], g[:, vh], scale)
    return vh, o, S


def sample_rows(T, n, seed):
    """Tail rows checked at full sizes: both ends, the middle and a seeded sample."""
    if T <= 0:
        return np.zeros(0, np.int64)
    fixed = [0, 1, T // 2, T - 2, T - 1]
    rng = np.random.default_rng(seed)
    extra = rng.integers(0, T, size=max(0, n - len(fixed)))
    return np.unique(np.clip(np.concatenate([fixed, extra]), 0, T - 1)).astype(np.int64)
