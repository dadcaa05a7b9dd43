#!/usr/bin/env python3
"""Benchmark of the true-tail update of a hybrid layer stack on one MI355X.

A step is one whole update (paper Section 4.1, Eq. 1-3) of the workload's
contexts: range verification, KV compaction of every attention layer, then in
layer order tail attention (RoPE append + causal GQA over surviving + new KV)
or gated delta-rule continuation from the carried state; metadata commit. Each
step runs on its own pristine copy of the contexts (caches, states, positions),
prepared before the timed region, so the K timed steps run back to back between
two device synchronisations.

The headline workload is the 48-layer hybrid stack (12 attention + 36 delta-rule
layers) on a 65,536-token context: 8 records of 256 tokens removed, 2,048 tail
tokens appended. Printed: one JSON line with tail tokens/s, the speedup over a
full refill of the same final context through the same kernels, the roofline
fraction of the dominant kernel (its duration measured with HIP events on its
stream, in a second pass over the same steps, and its HBM traffic from the
committed counter passes), the whole step against its roofline
(stack_roofline), per-stage fractions, and the CPU oracle timed on this host.
extra_rows adds: the other workloads (single refresh at 8K, eight rounds over a
32K context with the refill speedup after every round, 32 contexts in one call),
delimiter removal after prefill, the slot-preserving and tail-and-relocate
placements, the attention diagnostics, the short-convolution continuation, the
paper-shaped revision trace through the 48-layer stack and the tail-length sweep
at 32K rows.

    python bench.py [--config 4] [--steps 20] [--warmup 3] [--gpus 1] [--extra-configs 1,2,3]
                    [--no-refill] [--no-cpu-baseline] [--no-peaks] [--no-t-sweep] [--no-paper-trace]
                    [--only-update]
    python bench.py --calibrate-copy 256            # counter calibration (a plain device copy)
    python bench.py --config N --summarize-profile DIR   # rocprofv3 outputs -> profiles/ (CPU)
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# every attention layer keeps a persistent V^T copy beside its caches (refreshed from the
# first row that moved); --no-vt-copy packs every row into the workspace on every call
VT_COPIES = True
MFMA16_PEAK_TFLOPS = 2500.0
METRIC = "tail-update tokens/s (hybrid layer stack) + speedup vs full refill; % roofline"


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, choices=[0, 1, 2, 3, 4],
                    help="headline workload (default 4: the 48-layer hybrid stack at 64K)")
    ap.add_argument("--extra-configs", default="1,2,3",
                    help="comma-separated workloads also measured (update, refill speedup, stage fractions)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--refill-steps", type=int, default=5)
    ap.add_argument("--no-refill", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0)
    ap.add_argument("--kv-splits", type=int, default=0)
    ap.add_argument("--no-peaks", action="store_true", help="skip the copy and GEMM rate measurements")
    ap.add_argument("--no-t-sweep", action="store_true", help="skip the tail-length sweep at 32K rows")
    ap.add_argument("--no-paper-trace", action="store_true", help="skip the paper-shaped revision trace")
    ap.add_argument("--no-vt-copy", action="store_true",
                    help="no persistent V^T copies: every update packs all value rows into the workspace")
    ap.add_argument("--only-update", action="store_true",
                    help="time the headline update and its profiled pass only (for counter passes)")
    ap.add_argument("--only-diagnostics", action="store_true",
                    help="only the attention diagnostics on the workload (probe, group masses, total variation), "
                         "one JSON line, then exit (for profiling the probe kernels)")
    ap.add_argument("--calibrate-copy", type=int, metavar="MIB", default=0,
                    help="only copy a MIB-sized device buffer 5 times (calibrates HBM counters), then exit")
    ap.add_argument("--summarize-diagnostics", metavar="DIR", default=None,
                    help="CPU only: turn the rocprofv3 outputs of the --only-diagnostics passes under DIR into "
                         "profiles/attention_diagnostics_config<N>.md, then exit")
    ap.add_argument("--summarize-profile", metavar="DIR", default=None,
                    help="CPU only: turn the rocprofv3 outputs under DIR (trace/, calib_*/, pmc_*/) into "
                         "profiles/update_stack_config<N>.md and profiles/traffic_config<N>.json, then exit")
    return ap.parse_args()


# ----------------------------------------------------------------------------- device inputs

class DevRng:
    """Seeded device-side draws with the workload's value distributions."""

    def __init__(self, seed, device):
        import torch
        self.torch = torch
        self.g = torch.Generator(device=device)
        self.g.manual_seed(int(seed))
        self.dev = device

    def normal(self, shape, std=1.0, mean=0.0, dtype=None):
        t = self.torch.randn(*shape, generator=self.g, device=self.dev, dtype=self.torch.float32)
        if std != 1.0 or mean != 0.0:
            t = t * std + mean
        return t if dtype is None else t.to(dtype)

    def bf16(self, shape):
        return self.normal(shape).to(self.torch.bfloat16)

    def unit_bf16(self, shape):
        t = self.normal(shape)
        return (t / t.norm(dim=-1, keepdim=True)).to(self.torch.bfloat16)

    def beta(self, shape):
        return self.torch.sigmoid(self.normal(shape))

    def gate(self, shape):
        return self.torch.exp(-self.torch.nn.functional.softplus(self.normal(shape, mean=-4.0)))


def attach_vt_copies(tu, layers, chars, device):
    """A V^T copy beside every attention layer's cache of every context, brought up to date
    with the pristine rows (part of the pristine state each step copies)."""
    import torch
    if not VT_COPIES:
        return
    for L in layers:
        if L["kind"] != "attn":
            continue
        L["vts"] = []
        for (k, v), c in zip(L["caches"], chars):
            vt = tu.new_vt_cache(c["cap"], v.shape[1], v.shape[2], device)
            ctx = tu.Context(c["cap"], device=device)
            ctx.set_metadata(c["intervals"], c["cursor"])
            tu.refresh_vt_cache(ctx, [v], [vt])
            L["vts"].append(vt)
    torch.cuda.synchronize()


def build_workload(cfg, seed, device, tu=None):
    """Per-context plans plus pristine device buffers and packed tail inputs of every round.

    chars[c]: the context's initial state (L_old, intervals, cursor) and capacity;
    rounds[r]: per context the removal ranges, tail length and surviving rows of round
    r, and per layer that round's packed tail inputs."""
    import torch
    import synth
    sc = synth.make_scenario(cfg.index, seed=seed, cfg=cfg)
    rng = DevRng(seed * 1000 + cfg.index, device)
    a, d = cfg.attn, cfg.delta
    kinds = cfg.layer_kinds()
    chars = []
    for ch in sc.chars:
        r0 = ch.rounds[0]
        cap = max([r0.L_old] + [r.L_keep + r.T for r in ch.rounds])
        chars.append({"L_old": r0.L_old, "cursor": r0.cursor, "intervals": r0.intervals, "cap": cap})
    rounds = []
    for ri in range(len(sc.chars[0].rounds)):
        rr = [ch.rounds[ri] for ch in sc.chars]
        sumT = sum(r.T for r in rr)
        inputs = []
        for kind in kinds:
            if kind == "attn":
                inputs.append({"q": rng.bf16((sumT, a.n_q_heads, a.head_dim)),
                               "k": rng.bf16((sumT, a.n_kv_heads, a.head_dim)),
                               "v": rng.bf16((sumT, a.n_kv_heads, a.head_dim)),
                               "out": torch.empty((sumT, a.n_q_heads, a.head_dim), dtype=torch.float32,
                                                  device=device)})
            else:
                inputs.append({"q": rng.bf16((sumT, d.n_k_heads, d.d_k)),
                               "k": rng.unit_bf16((sumT, d.n_k_heads, d.d_k)),
                               "v": rng.bf16((sumT, d.n_v_heads, d.d_v)),
                               "beta": rng.beta((sumT, d.n_v_heads)), "g": rng.gate((sumT, d.n_v_heads)),
                               "out": torch.empty((sumT, d.n_v_heads, d.d_v), dtype=torch.float32, device=device)})
        rounds.append({"ranges": [r.ranges for r in rr], "T": [r.T for r in rr], "L_keep": [r.L_keep for r in rr],
                       "L_old": [r.L_old for r in rr], "cursor": [r.cursor for r in rr],
                       "intervals": [r.intervals for r in rr], "inputs": inputs})
    layers = []
    for kind in kinds:
        if kind == "attn":
            layers.append({"kind": "attn",
                           "caches": [(rng.bf16((c["cap"], a.n_kv_heads, a.head_dim)),
                                       rng.bf16((c["cap"], a.n_kv_heads, a.head_dim))) for c in chars]})
        else:
            layers.append({"kind": "delta",
                           "states": [rng.normal((d.n_v_heads, d.d_v, d.d_k), std=0.1) for _ in chars]})
    if tu is not None:
        attach_vt_copies(tu, layers, chars, device)
    return sc, chars, rounds, layers, rng


def make_copy(tu, chars, layers, device, pristine=True):
    """A fresh set of contexts/caches/states equal to the pristine workload."""
    import torch
    ctxs = []
    for c in chars:
        ctx = tu.Context(c["cap"], device=device)
        ctx.pos[: c["L_old"]] = torch.arange(c["L_old"], dtype=torch.int32, device=device)
        ctx.set_metadata(c["intervals"], c["cursor"], vt_rows=c["L_old"] if VT_COPIES else 0)
        ctxs.append(ctx)
    own = []
    for L in layers:
        if L["kind"] == "attn":
            o = {"caches": [(k.clone(), v.clone()) for (k, v) in L["caches"]]}
            if "vts" in L:
                o["vts"] = [vt.clone() for vt in L["vts"]]
            own.append(o)
        else:
            own.append({"states": [s.clone() for s in L["states"]]})
    return ctxs, own


def stack_update(tu, ctxs, own, layers, inputs, ranges, tails, attn_p, delta_p, post=None, placement=None,
                 place_runs=None):
    ios = []
    for L, O, src in zip(layers, own, inputs):
        if L["kind"] == "attn":
            ios.append(tu.LayerIO(tu.TU_LAYER_ATTN, src["q"], src["k"], src["v"], src["out"],
                                  k_cache=[k for (k, _) in O["caches"]], v_cache=[v for (_, v) in O["caches"]],
                                  vt_cache=O.get("vts")))
        else:
            ios.append(tu.LayerIO(tu.TU_LAYER_DELTA, src["q"], src["k"], src["v"], src["out"], state=O["states"],
                                  beta=src["beta"], g=src["g"]))
    return tu.StackUpdate(ctxs, ranges, tails, ios, attn_p, delta_p, post_ranges=post, placement=placement,
                          place_runs=place_runs)


def round_updates(tu, ctxs, own, layers, rounds, attn_p, delta_p, post=None, arm=None, place=None):
    """The prepared calls of one step: every round of the workload, in order, on one copy."""
    return [stack_update(tu, ctxs, own, layers, R["inputs"], R["ranges"], R["T"], attn_p, delta_p,
                         post=None if post is None else post(R),
                         placement=None if arm is None else [arm] * len(R["T"]),
                         place_runs=None if place is None else place(R)) for R in rounds]


def layers_of_kind(layers, rounds, kind):
    """The workload restricted to its layers of one kind (each round's inputs likewise)."""
    keep = [i for i, L in enumerate(layers) if L["kind"] == kind]
    rounds_k = [dict(R, inputs=[R["inputs"][i] for i in keep]) for R in rounds]
    return [layers[i] for i in keep], rounds_k


def paths_alone_row(tu, cfg, m, attn_p, delta_p, dev, W, K):
    """The update with only its delta layers, and with only its attention layers, on
    pristine copies of the same workload: in the full update the two run side by side and
    take turns on whole CUs, so the delta kernels' own durations there include waiting for
    CUs the attention workgroups hold."""
    import torch
    chars, rounds, layers = m["chars"], m["rounds"], m["layers"]
    kinds = cfg.layer_kinds()
    row = {}
    for kind in ("delta", "attn"):
        if not kinds.count(kind):
            continue
        lk, rk = layers_of_kind(layers, rounds, kind)
        copies = [make_copy(tu, chars, lk, dev) for _ in range(W + 2 * K)]
        ups = [round_updates(tu, ctxs, own, lk, rk, attn_p, delta_p) for (ctxs, own) in copies]
        ws = torch.empty(max(1, max(u.workspace_size() for u in ups[0])), dtype=torch.uint8, device=dev)
        for i in range(W):
            run_step(ups[i], ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(W, W + K):
            run_step(ups[i], ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / K
        tu.profile_enable(True)
        for i in range(W + K, W + 2 * K):
            run_step(ups[i], ws)
        prof = tu.profile_collect()
        tu.profile_enable(False)
        kern = {n: round(t / K, 5) for n, (c, t) in prof.items()}
        if kind == "delta":
            b = delta_bytes(cfg, rounds) * kinds.count("delta")
            ach = b / (ms / 1e3) / 1e9
            row["delta"] = {"layers": kinds.count("delta"), "update_ms": round(ms, 5), "kernels_ms": kern,
                            "bytes": b, "bound": "hbm", "achieved": round(ach, 1), "unit": "GB/s",
                            "peak": HBM_PEAK_GBS, "frac": round(ach / HBM_PEAK_GBS, 4)}
        else:
            f = attention_flops(cfg, rounds) * kinds.count("attn")
            att = kern.get("attention")
            row["attention_path"] = {"layers": kinds.count("attn"), "update_ms": round(ms, 5), "kernels_ms": kern,
                                     "attention_tflops": round(f / (att / 1e3) / 1e12, 1) if att else None,
                                     "attention_frac": round(f / (att / 1e3) / 1e12 / MFMA16_PEAK_TFLOPS, 4)
                                     if att else None}
        del copies, ups, ws
    return row


def slot_runs(R):
    """Positions of a slot-placed tail: the removed records' slots in order, then a free
    range 10,000 positions past the cursor for the tokens that do not fit."""
    out = []
    for rr, T, c0 in zip(R["ranges"], R["T"], R["cursor"]):
        runs, left = [], T
        for (a0, b0) in [tuple(x) for x in rr]:
            n = min(left, int(b0) - int(a0))
            if n > 0:
                runs.append((int(a0), int(a0) + n))
                left -= n
        if left > 0:
            runs.append((c0 + 10000, c0 + 10000 + left))
        out.append(runs)
    return out


# ----------------------------------------------------------------------------- algorithmic work

def attention_flops(cfg, rounds):
    a = cfg.attn
    return sum(4.0 * a.n_q_heads * a.head_dim * (T * Lk + T * (T + 1) / 2.0)
               for R in rounds for T, Lk in zip(R["T"], R["L_keep"]))


def delta_bytes(cfg, rounds):
    d = cfg.delta
    per_tok = d.n_k_heads * d.d_k * 2 * 2 + d.n_v_heads * d.d_v * 2 + d.n_v_heads * 8 + d.n_v_heads * d.d_v * 4
    state = d.n_v_heads * d.d_v * d.d_k * 4 * 2
    return sum(T * per_tok + state for R in rounds for T in R["T"])


def attention_kv_bytes(cfg, rounds):
    """K and V of every row an attention layer reads (surviving + new), once."""
    a = cfg.attn
    return sum((Lk + T) * a.n_kv_heads * a.head_dim * 2 * 2 for R in rounds for T, Lk in zip(R["T"], R["L_keep"]))


def stack_ideal_ms(cfg, rounds, mfma_tflops, hbm_gbs):
    """The step at the roofline: per step of the path its algorithmic work at the peak that
    bounds it (attention: max of its flops over the matrix peak and its K/V bytes over HBM;
    delta rule and compaction: bytes over HBM), summed over the layers."""
    kinds = cfg.layer_kinds()
    attn = max(attention_flops(cfg, rounds) / (mfma_tflops * 1e12), attention_kv_bytes(cfg, rounds) / (hbm_gbs * 1e9))
    delta = delta_bytes(cfg, rounds) / (hbm_gbs * 1e9)
    comp = gather_bytes(cfg, rounds) / (hbm_gbs * 1e9)
    return 1e3 * (kinds.count("attn") * (attn + comp) + kinds.count("delta") * delta)


def gather_bytes(cfg, rounds):
    """Minimum: every surviving row behind the first hole is read and written once."""
    a = cfg.attn
    row = a.n_kv_heads * a.head_dim * 2
    total = 0
    for R in rounds:
        for rng_, Lk, iv in zip(R["ranges"], R["L_keep"], R["intervals"]):
            if len(rng_) == 0:
                continue
            p = int(rng_[0][0])
            first = sum(max(0, min(e, p) - s) for (s, e) in iv)   # live rows below the first removed position
            total += 2 * 2 * (Lk - first) * row                    # K and V, read + write
    return total


# ----------------------------------------------------------------------------- CPU oracle leg

def cpu_baseline(cfg, seed, budget_s):
    """The float64 oracle on this host: one full update of the workload's first context
    (all tail rows of one attention layer, all tail tokens of one delta layer), repeated
    while within the budget, scaled to the workload's layer counts."""
    import numpy as np
    import oracle
    import synth
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threadpool_limits(cores)
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [cores])
    except Exception:
        blas_threads = cores
    sc = synth.make_scenario(cfg.index, seed=seed, cfg=cfg)
    r = sc.chars[0].rounds[0]
    a, d = cfg.attn, cfg.delta
    kb, vb = synth.gen_attn_cache(seed, cfg.index, 0, r.L_old, a)
    q, k, v = synth.gen_attn_tail(seed, cfg.index, 0, r.T, a)
    S0 = synth.gen_delta_state(seed, cfg.index, 1, d).astype(np.float64)
    dq, dk, dv, beta, g = synth.gen_delta_inputs(seed, cfg.index, 1, r.T, d)
    # rows / tokens sampled so one repetition stays within the budget
    rows = np.arange(r.T)
    toks = r.T
    est = (4.0 * a.n_q_heads * a.head_dim * r.T * (r.L_keep + r.T) / 2e10) + r.T * 4e-3
    if est > budget_s:
        frac = budget_s / est
        rows = np.unique(np.linspace(0, r.T - 1, max(8, int(r.T * frac))).astype(np.int64))
        toks = max(16, int(r.T * frac))
    t_attn, t_delta, reps = [], [], 0
    t_start = time.time()
    while reps < 3 and (reps == 0 or time.time() - t_start < budget_s):
        t0 = time.time()
        oracle.attention_layer_update(np.arange(r.L_old), kb, vb, r.ranges, r.cursor, q, k, v, a.rdim, a.rope_theta,
                                      a.softmax_scale, rows=rows)
        t1 = time.time()
        oracle.delta_layer_update(S0, dq[:toks], dk[:toks], dv[:toks], beta[:toks], g[:toks], d.scale)
        t2 = time.time()
        t_attn.append((t1 - t0) * r.T / len(rows))
        t_delta.append((t2 - t1) * r.T / toks)
        reps += 1
    kinds = cfg.layer_kinds()
    n_attn = kinds.count("attn")
    n_delta = kinds.count("delta")
    per_char = n_attn * min(t_attn) + n_delta * min(t_delta)
    total_T = sum(rd.T for c in sc.chars for rd in c.rounds)
    # other contexts and later rounds scale with their tail length
    scale = total_T / r.T
    secs = per_char * scale
    n_rounds = len(sc.chars[0].rounds)
    sample = (f"round 0 of context 0 of the workload: attention layer rows {len(rows)}/{r.T}, delta tokens "
              f"{toks}/{r.T}, {reps} repetitions (best), scaled to {n_attn} attention + {n_delta} delta layers"
              + (f" and {len(sc.chars)} contexts by tail length" if len(sc.chars) > 1 else "")
              + (f" and {n_rounds} rounds by tail length" if n_rounds > 1 else ""))
    return {"value": total_T / secs, "unit": "tail tokens/s", "cores": int(blas_threads), "kind": "oracle",
            "sample": sample, "seconds_per_update": secs}


# ----------------------------------------------------------------------------- main

def short_conv_row(tu, synth, cfg, T, dev, reps):
    """Short causal convolution continued from its carried state over the tail of one
    delta layer: the q, k and v projections (channels Hk*d_k, Hk*d_k, Hv*d_v), width 4,
    SiLU. Algorithmic bytes: x and y once, the carried rows read and written, weights."""
    import numpy as np
    import torch
    d = cfg.delta
    W = 4
    chans = [d.n_k_heads * d.d_k, d.n_k_heads * d.d_k, d.n_v_heads * d.d_v]
    bufs = []
    for i, C in enumerate(chans):
        st, x, w = synth.gen_conv_inputs(0, T, C, W, layer=i)
        dv = lambda b: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
        bufs.append((dv(st), dv(x), dv(w), torch.empty((T, C), dtype=torch.bfloat16, device=dev)))
    tu.short_conv_continue_batch(bufs)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        tu.short_conv_continue_batch(bufs)   # one launch for the three tensors
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = sum(2 * T * C * 2 + 2 * (W - 1) * C * 2 + C * W * 2 for C in chans)
    ach = nbytes / (ms / 1e3) / 1e9
    return {"tokens": T, "channels": chans, "width": W, "launches": 1, "ms": round(ms, 5),
            "bytes": nbytes, "bound": "hbm", "achieved": round(ach, 1), "unit": "GB/s", "peak": HBM_PEAK_GBS,
            "frac": round(ach / HBM_PEAK_GBS, 4)}


def t_sweep_row(tu, synth, dev, attn_p, delta_p, seed, reps, warmup=2):
    """The update (one attention + one delta layer, one 64-token record removed) at 32,768
    surviving rows for tails of 1 .. 2048 tokens. Short tails are decode-like: the
    attention kernel then reads the whole K/V cache for a few queries and is bound by
    HBM (algorithmic bytes: K and V of the surviving + new rows once); long ones are
    bound by its MFMA products."""
    import torch
    rows = []
    for T in synth.T_SWEEP:
        cfg = synth.t_sweep_config(T)
        _, chars, rounds, layers, _ = build_workload(cfg, seed, dev, tu)
        copies = [make_copy(tu, chars, layers, dev) for _ in range(warmup + 2 * reps)]
        ups = [round_updates(tu, c, o, layers, rounds, attn_p, delta_p) for (c, o) in copies]
        ws = torch.empty(max(u[0].workspace_size() for u in ups), dtype=torch.uint8, device=dev)
        for u in ups[:warmup]:
            u[0].run(ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for u in ups[warmup:warmup + reps]:
            u[0].run(ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tu.profile_enable(True)
        for u in ups[warmup + reps:]:
            u[0].run(ws)
        prof = tu.profile_collect()
        tu.profile_enable(False)
        kern = {n: t / c for n, (c, t) in prof.items()}
        a = cfg.attn
        Lk = rounds[0]["L_keep"][0]
        kv_bytes = (Lk + T) * a.n_kv_heads * a.head_dim * 2 * 2
        flops = attention_flops(cfg, rounds)
        hbm = T * a.n_q_heads / a.n_kv_heads < 312   # below the ridge of 2.5 PFLOP/s over 8 TB/s
        att = kern.get("attention")
        row = {"T": T, "L_keep": Lk, "update_ms": round(ms, 5), "tail_tok_s": round(T / (ms / 1e3), 1),
               "attention_ms": round(att, 5) if att else None,
               "stage_ms": round(kern["rope_vt_pack"], 5) if "rope_vt_pack" in kern else None,
               "merge_ms": round(kern["attention_merge"], 5) if "attention_merge" in kern else None,
               "attention_bound": "hbm" if hbm else "mfma"}
        if att:
            if hbm:
                row.update({"achieved": round(kv_bytes / (att / 1e3) / 1e9, 1), "unit": "GB/s", "peak": HBM_PEAK_GBS,
                            "bytes": kv_bytes})
            else:
                row.update({"achieved": round(flops / (att / 1e3) / 1e12, 1), "unit": "TFLOP/s",
                            "peak": MFMA16_PEAK_TFLOPS, "flops": flops})
            row["frac"] = round(row["achieved"] / row["peak"], 4)
        rows.append(row)
        print(f"[bench] t sweep: {json.dumps(row)}", file=sys.stderr, flush=True)
        del copies, ups, ws, layers, rounds
    return rows


def paper_trace_row(tu, synth, dev, attn_p, delta_p, seed, reps, warmup=1):
    """Eight revisions shaped like the paper's measured trace (its Section 6.6: an
    ~11.9K-token prefix of ~390-token records in 10K-position slots; each revision
    replaces one or two whole records by 214-362 tokens at fresh slots past the cursor,
    with 11 framing tokens prefilled and removed again) through the 48-layer hybrid
    stack of the 64K workload (12 attention + 36 delta layers). Reports each revision's
    update time, the least-squares line time = fixed + per_token * m over the eight
    revisions (m = replacement-record tokens, the paper's fit variable), and the refill of
    the final context (contiguous positions, zero states) through the same kernels."""
    import numpy as np
    import torch
    cfg = synth.CONFIGS[4]
    a, d = cfg.attn, cfg.delta
    kinds = cfg.layer_kinds()
    tr = synth.make_paper_trace(seed)
    L0 = len(tr.positions)
    cap = max([L0] + [r.L_old + r.T for r in tr.revisions])
    rng = DevRng(seed * 1000 + 200, dev)
    layers, inputs = [], [[] for _ in tr.revisions]
    for kind in kinds:
        if kind == "attn":
            layers.append({"kind": "attn", "caches": [(rng.bf16((cap, a.n_kv_heads, a.head_dim)),
                                                       rng.bf16((cap, a.n_kv_heads, a.head_dim)))]})
        else:
            layers.append({"kind": "delta", "states": [rng.normal((d.n_v_heads, d.d_v, d.d_k), std=0.1)]})
        for r, rv in enumerate(tr.revisions):
            T = rv.T
            if kind == "attn":
                inputs[r].append({"q": rng.bf16((T, a.n_q_heads, a.head_dim)), "k": rng.bf16((T, a.n_kv_heads, a.head_dim)),
                                  "v": rng.bf16((T, a.n_kv_heads, a.head_dim)),
                                  "out": torch.empty((T, a.n_q_heads, a.head_dim), dtype=torch.float32, device=dev)})
            else:
                inputs[r].append({"q": rng.bf16((T, d.n_k_heads, d.d_k)), "k": rng.unit_bf16((T, d.n_k_heads, d.d_k)),
                                  "v": rng.bf16((T, d.n_v_heads, d.d_v)), "beta": rng.beta((T, d.n_v_heads)),
                                  "g": rng.gate((T, d.n_v_heads)),
                                  "out": torch.empty((T, d.n_v_heads, d.d_v), dtype=torch.float32, device=dev)})
    pos0 = torch.from_numpy(tr.positions.astype(np.int32)).to(dev)
    attach_vt_copies(tu, layers, [{"cap": cap, "intervals": tr.intervals, "cursor": tr.cursor}], dev)

    def fresh():
        ctx = tu.Context(cap, device=dev)
        ctx.pos[:L0] = pos0
        ctx.set_metadata(tr.intervals, tr.cursor, vt_rows=L0 if VT_COPIES else 0)
        own = []
        for L in layers:
            if L["kind"] == "attn":
                o = {"caches": [(k.clone(), v.clone()) for (k, v) in L["caches"]]}
                if "vts" in L:
                    o["vts"] = [vt.clone() for vt in L["vts"]]
                own.append(o)
            else:
                own.append({"states": [x.clone() for x in L["states"]]})
        return ctx, [stack_update(tu, [ctx], own, layers, inputs[r], [rv.ranges], [rv.T], attn_p, delta_p,
                                  post=[rv.post], placement=["slot"], place_runs=[rv.runs])
                     for r, rv in enumerate(tr.revisions)]

    ws = None
    times = []
    for rep in range(warmup + reps):
        ctx, ups = fresh()
        if ws is None:
            # the largest workspace any revision needs, each sized on the metadata it will see
            need = 0
            for u, rv in zip(ups, tr.revisions):
                ctx.set_metadata(rv.intervals, rv.cursor)
                need = max(need, u.workspace_size())
            ctx.set_metadata(tr.intervals, tr.cursor, vt_rows=L0 if VT_COPIES else 0)
            ws = torch.empty(need, dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(ups) + 1)]
        ev[0].record()
        for i, u in enumerate(ups):
            u.run(ws)
            ev[i + 1].record()
        torch.cuda.synchronize()
        if rep >= warmup:
            times.append([ev[i].elapsed_time(ev[i + 1]) for i in range(len(ups))])
        final_rows, final_cursor = ctx.len, ctx.next_pos
        del ctx, ups
    per = np.median(np.asarray(times), axis=0)
    m = np.asarray([rv.m for rv in tr.revisions], dtype=np.float64)
    per_tok, fixed = np.polyfit(m, per, 1)
    # refill of the final context through the same stack
    N = int(final_rows)
    rin = []
    for kind in kinds:
        if kind == "attn":
            rin.append({"q": rng.bf16((N, a.n_q_heads, a.head_dim)), "k": rng.bf16((N, a.n_kv_heads, a.head_dim)),
                        "v": rng.bf16((N, a.n_kv_heads, a.head_dim)),
                        "out": torch.empty((N, a.n_q_heads, a.head_dim), dtype=torch.float32, device=dev)})
        else:
            rin.append({"q": rng.bf16((N, d.n_k_heads, d.d_k)), "k": rng.unit_bf16((N, d.n_k_heads, d.d_k)),
                        "v": rng.bf16((N, d.n_v_heads, d.d_v)), "beta": rng.beta((N, d.n_v_heads)),
                        "g": rng.gate((N, d.n_v_heads)),
                        "out": torch.empty((N, d.n_v_heads, d.d_v), dtype=torch.float32, device=dev)})
    caches = [[(torch.empty((N, a.n_kv_heads, a.head_dim), dtype=torch.bfloat16, device=dev),
                torch.empty((N, a.n_kv_heads, a.head_dim), dtype=torch.bfloat16, device=dev))]
              if L["kind"] == "attn" else None for L in layers]
    rt = []
    for rep in range(warmup + reps):
        ctx = tu.Context(N, device=dev)
        ctx.set_metadata([], 0)
        own = [{"caches": C, "vts": [tu.new_vt_cache(N, a.n_kv_heads, a.head_dim, dev)] if VT_COPIES else None}
               if L["kind"] == "attn" else
               {"states": [torch.zeros((d.n_v_heads, d.d_v, d.d_k), dtype=torch.float32, device=dev)]}
               for L, C in zip(layers, caches)]
        u = stack_update(tu, [ctx], own, layers, rin, [np.zeros((0, 2), np.int64)], [N], attn_p, delta_p)
        rws = torch.empty(u.workspace_size(), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        u.run(rws)
        e1.record()
        torch.cuda.synchronize()
        if rep >= warmup:
            rt.append(e0.elapsed_time(e1))
        del u, rws, own, ctx
    refill_ms = float(np.median(rt))
    row = {"layers": len(kinds), "attention_layers": kinds.count("attn"), "delta_layers": kinds.count("delta"),
           "initial_rows": L0, "initial_cursor": tr.cursor, "final_rows": N, "final_cursor": int(final_cursor),
           "revisions": [{"m": rv.m, "T": rv.T, "removed_rows": int(np.sum(rv.ranges[:, 1] - rv.ranges[:, 0])),
                          "live_rows_before": rv.L_old, "ms": round(float(t), 5)}
                         for rv, t in zip(tr.revisions, per)],
           "total_ms": round(float(per.sum()), 5),
           "fit_ms": {"fixed": round(float(fixed), 5), "per_token": round(float(per_tok), 7)},
           "refill_ms": round(refill_ms, 5), "refill_over_mean_revision": round(refill_ms / float(per.mean()), 2),
           "placement": "each replacement record at a fresh 10K-position slot past the cursor (explicit positions)"}
    del caches, rin, layers, inputs, ws
    return row


def lib_probe_ws(tu, attn_p, length, n_probe):
    import ctypes
    return max(256, int(tu.lib().attention_probe_workspace_size(ctypes.byref(attn_p), length, n_probe)))


def measured_peaks(dev):
    """Rates this GPU sustains in this run, as a second reference beside the datasheet peaks:
    a plain 1 GiB device copy (bytes read + written per second) and an 8192^3 bf16 GEMM
    (torch.matmul, contiguous operands), each timed over repeated back-to-back launches."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    a.fill_(1)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    reps = 10
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 2.0 * n * reps / (e0.elapsed_time(e1) / 1e3) / 1e9
    del a, b
    m = 8192
    x = torch.randn((m, m), device=dev, dtype=torch.float32).to(torch.bfloat16)
    y = torch.randn((m, m), device=dev, dtype=torch.float32).to(torch.bfloat16)
    for _ in range(5):
        z = torch.matmul(x, y)
    torch.cuda.synchronize()
    reps = 50
    e0.record()
    for _ in range(reps):
        z = torch.matmul(x, y)
    e1.record()
    torch.cuda.synchronize()
    gemm_tflops = 2.0 * m ** 3 * reps / (e0.elapsed_time(e1) / 1e3) / 1e12
    del x, y, z
    torch.cuda.empty_cache()
    return {"copy_gbs": round(copy_gbs, 1), "copy_bytes": 2 * n, "bf16_gemm_tflops": round(gemm_tflops, 1),
            "gemm_shape": [m, m, m], "gemm_launches": reps}


def measured_traffic(kernel, cfg_index, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE and
    WRITE_SIZE passes of this workload (profiles/traffic_config<N>.json), or None when
    there is no record for it or the kernel's sources changed since the counters were
    taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_config{cfg_index}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel") != kernel or rec.get("workload") != workload:
        return None
    if sources_sha256(rec["sources"]) != rec["sources_sha256"]:
        return None
    return {"bytes_per_launch": rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"],
            "read": rec["fetch_bytes_per_launch"], "written": rec["write_bytes_per_launch"],
            "source": rec["summary"]}


def sources_sha256(srcs):
    h = hashlib.sha256()
    for src in srcs:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


# sources each kernel's traffic record depends on
KERNEL_SOURCES = {
    "attention": ["paper_2609_18935_amd/csrc/attention.hip", "paper_2609_18935_amd/csrc/common.h"],
}
KERNEL_SYMBOL = {"attention": "k_attn<256>"}


def calibrate_copy(mib):
    """A plain device copy of `mib` MiB, five times: under rocprofv3 --pmc FETCH_SIZE (then
    WRITE_SIZE) it shows what the counters report for exactly that many bytes read and
    written, the factor that scales the library kernels' counters to bytes."""
    import torch
    n = mib << 20
    a = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x 5", flush=True)


PROFILE_COMMANDS = """rocprofv3 --kernel-trace --stats -f csv -d <out>/trace -o run -- python3 <repo>/bench.py --config {c} --steps 10 --warmup 2 --only-update
rocprofv3 --pmc FETCH_SIZE -f csv -d <out>/calib_FETCH_SIZE -o run -- python3 <repo>/bench.py --calibrate-copy 256
rocprofv3 --pmc FETCH_SIZE -f csv -d <out>/pmc_FETCH_SIZE -o run -- python3 <repo>/bench.py --config {c} --steps 2 --warmup 1 --only-update
rocprofv3 --pmc WRITE_SIZE -f csv -d <out>/calib_WRITE_SIZE -o run -- python3 <repo>/bench.py --calibrate-copy 256
rocprofv3 --pmc WRITE_SIZE -f csv -d <out>/pmc_WRITE_SIZE -o run -- python3 <repo>/bench.py --config {c} --steps 2 --warmup 1 --only-update
python3 <repo>/bench.py --config {c} --summarize-profile <out>"""


def describe(cfg):
    """One line naming a workload's shapes and sizes."""
    a, d = cfg.attn, cfg.delta
    kinds = cfg.layer_kinds()
    if cfg.L_old is not None:
        pre = f"{cfg.L_old} cached rows"
    elif cfg.L_keep is not None:
        pre = f"{cfg.L_keep} surviving rows"
    else:
        pre = f"surviving rows uniform in [{cfg.L_keep_range[0]}, {cfg.L_keep_range[1]}]"
    rec = (f"{cfg.n_records[0]}-{cfg.n_records[1]}" if cfg.n_records[0] != cfg.n_records[1] else f"{cfg.n_records[0]}")
    rl = (f"{cfg.record_len[0]}-{cfg.record_len[1]}" if cfg.record_len[0] != cfg.record_len[1] else f"{cfg.record_len[0]}")
    tl = f"{cfg.tail[0]}-{cfg.tail[1]}" if cfg.tail[0] != cfg.tail[1] else f"{cfg.tail[0]}"
    return (f"{cfg.n_chars} context(s), {cfg.n_rounds} round(s); {pre}; {rec} record(s) of {rl} rows removed and "
            f"{tl} tail tokens appended per round; {len(kinds)} layers ({kinds.count('attn')} attention "
            f"{a.n_q_heads}q/{a.n_kv_heads}kv x {a.head_dim}, {kinds.count('delta')} gated delta-rule "
            f"{d.n_k_heads}k/{d.n_v_heads}v x {d.d_k}, chunk {d.chunk}).")


def _profile_tables(out_dir):
    """The kernel-duration table and the copy-calibrated HBM traffic per dispatch (MiB) of
    the rocprofv3 CSV outputs under out_dir (trace/, calib_*/, pmc_*/), as markdown lines,
    and the calibrated KiB per dispatch by kernel."""
    import csv
    import re
    import statistics

    def short(n):
        n = n.replace("tu::(anonymous namespace)::", "").replace("void ", "")
        return re.sub(r"\(.*\)$", "", n)

    def rows(sub, name):
        path = os.path.join(out_dir, sub, name)
        with open(path) as f:
            return list(csv.DictReader(f))

    stats = [r for r in rows("trace", "run_kernel_stats.csv") if "tu::" in r["Name"]]

    def pmc(kind):
        per = {}
        for r in rows(f"pmc_{kind}", "run_counter_collection.csv"):
            if "tu::" in r["Kernel_Name"]:
                per.setdefault(short(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
        return {k: statistics.median(v) for k, v in per.items()}

    def calib(kind):
        vals = [float(r["Counter_Value"]) for r in rows(f"calib_{kind}", "run_counter_collection.csv")]
        return max(vals)   # the copy dispatches (KiB)

    true_kib = 256 * 1024
    fr, wr = pmc("FETCH_SIZE"), pmc("WRITE_SIZE")
    fc, wc = calib("FETCH_SIZE"), calib("WRITE_SIZE")
    ff, wf = true_kib / fc, true_kib / wc
    out = ["## Kernel durations (rocprofv3 --kernel-trace --stats, every dispatch of the traced command)\n",
           "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        out.append(f"| {short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    out += ["\n## HBM traffic per dispatch (median over the dispatches, MiB)\n",
            f"Calibration with a plain 256 MiB device copy: FETCH_SIZE reported {fc:,.1f} KiB for 262,144 KiB read "
            f"(factor {ff:.3f}), WRITE_SIZE {wc:,.1f} KiB for 262,144 KiB written (factor {wf:.3f}). Values below "
            "are scaled by those factors.\n", "| kernel | read MiB | written MiB |", "|---|---|---|"]
    for k in sorted(fr, key=lambda k: -fr[k]):
        out.append(f"| {k} | {fr[k] * ff / 1024:.2f} | {wr.get(k, 0) * wf / 1024:.2f} |")
    read_kib = {k: v * ff for k, v in fr.items()}
    written_kib = {k: v * wf for k, v in wr.items()}
    return out, read_kib, written_kib, (ff, wf)


def summarize_profile(out_dir, cfg_index):
    """Writes profiles/update_stack_config<N>.md (kernel durations of the traced update,
    calibrated HBM bytes per dispatch) and profiles/traffic_config<N>.json (the attention
    kernel's bytes per launch, with the hash of its sources) from rocprofv3 CSV outputs."""
    import synth
    cfg = synth.CONFIGS[cfg_index]
    tables, read_kib, written_kib, (ff, wf) = _profile_tables(out_dir)
    workload = f"config {cfg.index}: {cfg.name}"
    out = [f"# Update, {workload}: kernel trace and HBM traffic\n",
           f"Workload: {describe(cfg)}\n",
           "Commands (repository root on the GPU host; rocprofv3 run from /tmp with TMPDIR=/tmp; each pass in "
           "its own process; the last line runs here, on the CPU):\n", "```",
           PROFILE_COMMANDS.format(c=cfg.index), "```\n"] + tables
    blog = os.path.join(out_dir, "trace_bench.log")
    if os.path.exists(blog):
        lines = [l for l in open(blog) if l.startswith("{")]
        if lines:
            out += ["\n## Bench line of the traced run\n", "```json", lines[-1].strip(), "```"]
    md = f"profiles/update_stack_config{cfg.index}.md"
    with open(os.path.join(ROOT, md), "w") as f:
        f.write("\n".join(out) + "\n")
    sym = KERNEL_SYMBOL["attention"]
    if sym in read_kib and sym in written_kib:
        rec = {"workload": workload, "kernel": "attention", "kernel_symbol": sym,
               "sources": KERNEL_SOURCES["attention"], "sources_sha256": sources_sha256(KERNEL_SOURCES["attention"]),
               "fetch_bytes_per_launch": int(read_kib[sym] * 1024), "write_bytes_per_launch": int(written_kib[sym] * 1024),
               "calibration": {"fetch_factor": round(ff, 4), "write_factor": round(wf, 4)}, "summary": md}
        with open(os.path.join(ROOT, "profiles", f"traffic_config{cfg.index}.json"), "w") as f:
            json.dump(rec, f, indent=1)
    print("\n".join(out[:40]))


DIAGNOSTICS_COMMANDS = """\
python3 <repo>/bench.py --config {c} --only-diagnostics --steps 5
rocprofv3 --kernel-trace --stats -f csv -d <out>/trace -o run -- python3 <repo>/bench.py --config {c} --only-diagnostics --steps 5
rocprofv3 --pmc FETCH_SIZE -f csv -d <out>/calib_FETCH_SIZE -o run -- python3 <repo>/bench.py --calibrate-copy 256
rocprofv3 --pmc FETCH_SIZE -f csv -d <out>/pmc_FETCH_SIZE -o run -- python3 <repo>/bench.py --config {c} --only-diagnostics --steps 2
rocprofv3 --pmc WRITE_SIZE -f csv -d <out>/calib_WRITE_SIZE -o run -- python3 <repo>/bench.py --calibrate-copy 256
rocprofv3 --pmc WRITE_SIZE -f csv -d <out>/pmc_WRITE_SIZE -o run -- python3 <repo>/bench.py --config {c} --only-diagnostics --steps 2
python3 <repo>/bench.py --config {c} --summarize-diagnostics <out>"""


def summarize_diagnostics(out_dir, cfg_index):
    """Writes profiles/attention_diagnostics_config<N>.md: the kernel durations and
    calibrated HBM bytes per dispatch of the attention diagnostics (bench --only-diagnostics),
    with the row of the plain run (<out>/plain.log) and each score pass's key bytes."""
    import synth
    cfg = synth.CONFIGS[cfg_index]
    a = cfg.attn
    tables, read_kib, written_kib, _ = _profile_tables(out_dir)
    workload = f"config {cfg.index}: {cfg.name}"
    plog = os.path.join(out_dir, "plain.log")
    plain = [l for l in open(plog) if l.startswith("{")] if os.path.exists(plog) else []
    live = json.loads(plain[-1])["attention_diagnostics"]["live_rows"] if plain else cfg.L_old
    key_mib = live * a.n_kv_heads * a.head_dim * 2 / 2 ** 20
    out = [f"# Attention diagnostics, {workload}: kernel trace and HBM traffic\n",
           f"Workload: {describe(cfg)} The diagnostics follow the first round: the probe of the last 8 tail rows "
           "of each of the attention layers (one call per layer), the masses of 390-position memory groups and the "
           "total variation between the first and the last attention layer's probes.\n",
           f"Each score pass (`k_probe_part`, `k_probe_keysum`) reads one layer's key cache: {key_mib:.1f} MiB "
           f"({live:,} live rows, all KV heads, bf16).\n",
           "Commands (repository root on the GPU host; rocprofv3 run from /tmp with TMPDIR=/tmp; each pass in "
           "its own process; the last line runs here, on the CPU):\n", "```",
           DIAGNOSTICS_COMMANDS.format(c=cfg.index), "```\n"] + tables
    if plain:
        out += ["\n## Row of the plain run\n", "```json", plain[-1].strip(), "```"]
    md = f"profiles/attention_diagnostics_config{cfg.index}.md"
    with open(os.path.join(ROOT, md), "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


# ----------------------------------------------------------------------------- one workload

def workload_stage_fracs(cfg, rounds, kern):
    """Algorithmic work per step of each stage against the summed durations of its kernels."""
    kinds = cfg.layer_kinds()
    work = {
        "attention": (["rope_vt_pack", "attention", "attention_merge"], "mfma",
                      attention_flops(cfg, rounds) * kinds.count("attn") / 1e12, "TFLOP/s", MFMA16_PEAK_TFLOPS),
        "delta": (["delta_prep", "delta_chain"], "hbm", delta_bytes(cfg, rounds) * kinds.count("delta") / 1e9,
                  "GB/s", HBM_PEAK_GBS),
        "compaction": (["compact"], "hbm", gather_bytes(cfg, rounds) * kinds.count("attn") / 1e9, "GB/s",
                       HBM_PEAK_GBS),
    }
    stages = {}
    for name, (ks, bound, units, unit, peak) in work.items():
        ms = sum(kern[k]["ms_per_step"] for k in ks if k in kern)
        if ms > 0 and units > 0:
            ach = units / (ms / 1e3)
            stages[name] = {"kernels": ks, "ms_per_step": round(ms, 5), "bound": bound, "achieved": round(ach, 3),
                            "peak": peak, "unit": unit, "frac": round(ach / peak, 4)}
    return stages


def measure_update(tu, cfg, seed, dev, attn_p, delta_p, W, K, refill_steps, keep=False):
    """Times K updates of the workload (each on its own pristine copy, after W warm-ups),
    then the same steps with per-kernel HIP events, then (refill_steps > 0) the full
    refill of the live context after every round through the same kernels."""
    import numpy as np
    import torch
    sc, chars, rounds, layers, rng = build_workload(cfg, seed, dev, tu)
    a, d = cfg.attn, cfg.delta
    n_rounds = len(rounds)
    sumT = sum(sum(R["T"]) for R in rounds)
    print(f"[bench] config {cfg.index} ({cfg.name}): {len(chars)} context(s), {len(layers)} layers, "
          f"{n_rounds} round(s), sum T = {sumT}", file=sys.stderr, flush=True)

    def workspace_for(ctxs, ups):
        """Largest workspace any round of a step needs (each round sized on its own metadata)."""
        n = 0
        vt0 = [ctx.vt_rows for ctx in ctxs]
        for R, u in zip(rounds, ups):
            for c, ctx in enumerate(ctxs):
                ctx.set_metadata(R["intervals"][c], R["cursor"][c])
            n = max(n, u.workspace_size())
        for c, ctx in enumerate(ctxs):
            ctx.set_metadata(chars[c]["intervals"], chars[c]["cursor"], vt_rows=vt0[c])
        return n

    # ---- update: one pristine copy per step; a step is every round of the workload
    copies = [make_copy(tu, chars, layers, dev) for _ in range(W + K)]
    ups = [round_updates(tu, ctxs, own, layers, rounds, attn_p, delta_p) for (ctxs, own) in copies]
    ws = torch.empty(workspace_for(copies[0][0], ups[0]), dtype=torch.uint8, device=dev)
    for i in range(W):
        run_step(ups[i], ws)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    h0 = time.perf_counter()
    ev0.record()
    for i in range(W, W + K):
        run_step(ups[i], ws)
    ev1.record()
    torch.cuda.synchronize()
    h1 = time.perf_counter()
    upd_ms = ev0.elapsed_time(ev1) / K
    print(f"[bench] config {cfg.index} update: {upd_ms:.4f} ms/step (host {1e3 * (h1 - h0) / K:.4f})",
          file=sys.stderr, flush=True)
    del copies, ups
    round_ms = None
    if n_rounds > 1:
        # per-round durations, from events between the rounds of the same steps
        copies = [make_copy(tu, chars, layers, dev) for _ in range(K)]
        ups = [round_updates(tu, ctxs, own, layers, rounds, attn_p, delta_p) for (ctxs, own) in copies]
        torch.cuda.synchronize()
        marks = [[torch.cuda.Event(enable_timing=True) for _ in rounds] for _ in range(K)]
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
        for i in range(K):
            starts[i].record()
            run_step(ups[i], ws, marks[i])
        torch.cuda.synchronize()
        round_ms = [sorted(((marks[i][r - 1] if r else starts[i]).elapsed_time(marks[i][r]) for i in range(K)))[K // 2]
                    for r in range(n_rounds)]
        del copies, ups

    # ---- profiled pass over the same steps (fresh copies), per-kernel HIP events
    copies2 = [make_copy(tu, chars, layers, dev) for _ in range(K)]
    ups2 = [round_updates(tu, ctxs, own, layers, rounds, attn_p, delta_p) for (ctxs, own) in copies2]
    torch.cuda.synchronize()
    tu.profile_enable(True)
    for u in ups2:
        run_step(u, ws)
    prof = tu.profile_collect()
    tu.profile_enable(False)
    del copies2, ups2
    kern = {n: {"launches_per_step": c / K, "avg_ms": t / c, "ms_per_step": t / K} for n, (c, t) in prof.items()}
    print(f"[bench] config {cfg.index} kernels: {json.dumps(kern)}", file=sys.stderr, flush=True)

    # ---- full refill, through the same kernels, of the live context after every round
    # (zero recurrent state, contiguous positions from 0, fresh caches); the speedup is
    # the summed refill time over the summed update time
    refill = None
    if refill_steps > 0:
        R_ = refill_steps
        refill_rounds = []
        for ri, R in enumerate(rounds):
            N = [Lk + T for Lk, T in zip(R["L_keep"], R["T"])]
            sumN = sum(N)
            rin = []
            for L in layers:
                if L["kind"] == "attn":
                    rin.append({"q": rng.bf16((sumN, a.n_q_heads, a.head_dim)),
                                "k": rng.bf16((sumN, a.n_kv_heads, a.head_dim)),
                                "v": rng.bf16((sumN, a.n_kv_heads, a.head_dim)),
                                "out": torch.empty((sumN, a.n_q_heads, a.head_dim), dtype=torch.float32, device=dev)})
                else:
                    rin.append({"q": rng.bf16((sumN, d.n_k_heads, d.d_k)),
                                "k": rng.unit_bf16((sumN, d.n_k_heads, d.d_k)),
                                "v": rng.bf16((sumN, d.n_v_heads, d.d_v)), "beta": rng.beta((sumN, d.n_v_heads)),
                                "g": rng.gate((sumN, d.n_v_heads)),
                                "out": torch.empty((sumN, d.n_v_heads, d.d_v), dtype=torch.float32, device=dev)})
            # refill writes every cache row and starts from zero states: caches are shared
            # by the repetitions, states are zeroed per repetition
            caches = [[(torch.empty((n, a.n_kv_heads, a.head_dim), dtype=torch.bfloat16, device=dev),
                        torch.empty((n, a.n_kv_heads, a.head_dim), dtype=torch.bfloat16, device=dev)) for n in N]
                      if L["kind"] == "attn" else None for L in layers]
            # fresh V^T copies too (the refill packs every row into them)
            vts = [[tu.new_vt_cache(n, a.n_kv_heads, a.head_dim, dev) for n in N]
                   if L["kind"] == "attn" and VT_COPIES else None for L in layers]
            rups = []
            for i in range(R_ + 1):
                ctxs = []
                for n in N:
                    ctx = tu.Context(n, device=dev)
                    ctx.set_metadata([], 0)
                    ctxs.append(ctx)
                own_i = [{"caches": C, "vts": V} if L["kind"] == "attn" else
                         {"states": [torch.zeros((d.n_v_heads, d.d_v, d.d_k), dtype=torch.float32, device=dev)
                                     for _ in N]} for L, C, V in zip(layers, caches, vts)]
                rups.append(stack_update(tu, ctxs, own_i, layers, rin, [np.zeros((0, 2), np.int64)] * len(N), N,
                                         attn_p, delta_p))
            rws = torch.empty(max(u.workspace_size() for u in rups), dtype=torch.uint8, device=dev)
            rups[0].run(rws)
            torch.cuda.synchronize()
            ev0.record()
            for u in rups[1:]:
                u.run(rws)
            ev1.record()
            torch.cuda.synchronize()
            refill_rounds.append({"tokens": sumN, "ms": ev0.elapsed_time(ev1) / R_})
            del rups, rin, caches, rws
        refill_ms = sum(x["ms"] for x in refill_rounds)
        refill = {"ms": refill_ms, "tokens": sum(x["tokens"] for x in refill_rounds), "speedup": refill_ms / upd_ms}
        if n_rounds > 1:
            refill["rounds"] = [{"tail": sum(R["T"]), "live_after": x["tokens"], "update_ms": round(um, 5),
                                 "refill_ms": round(x["ms"], 5), "speedup": round(x["ms"] / um, 3)}
                                for R, x, um in zip(rounds, refill_rounds, round_ms)]
        print(f"[bench] config {cfg.index} refill: {refill_ms:.4f} ms ({refill['tokens']} tokens over {n_rounds} "
              f"round(s)), speedup {refill_ms / upd_ms:.2f}x", file=sys.stderr, flush=True)
    res = {"cfg": cfg, "upd_ms": upd_ms, "round_ms": round_ms, "kern": kern, "refill": refill, "sumT": sumT,
           "stages": workload_stage_fracs(cfg, rounds, kern), "chars": chars, "rounds": rounds}
    if keep:
        res.update({"layers": layers, "rng": rng, "ws": ws})
    else:
        del layers, ws
        torch.cuda.empty_cache()
    return res


def config_row(m):
    """Summary of one measured workload for extra_rows."""
    cfg, rounds = m["cfg"], m["rounds"]
    kinds = cfg.layer_kinds()
    row = {"workload": f"config {cfg.index}: {cfg.name}", "contexts": len(m["chars"]), "layers": len(kinds),
           "rounds": len(rounds), "tail_tokens": m["sumT"], "update_ms": round(m["upd_ms"], 5),
           "tail_tok_s": round(m["sumT"] / (m["upd_ms"] / 1e3), 1), "stages": m["stages"],
           "stack_roofline_frac": round(stack_ideal_ms(cfg, rounds, MFMA16_PEAK_TFLOPS, HBM_PEAK_GBS) / m["upd_ms"], 4),
           "kernels": {n: {k: (round(v, 6) if isinstance(v, float) else v) for k, v in kv.items()}
                       for n, kv in m["kern"].items()}}
    if m["refill"]:
        row.update({"refill_ms": round(m["refill"]["ms"], 5), "speedup_vs_refill": round(m["refill"]["speedup"], 3)})
        if "rounds" in m["refill"]:
            row["refill_rounds"] = m["refill"]["rounds"]
    return row


def run_step(ups, ws, per_round=None):
    for i, u in enumerate(ups):
        u.run(ws)
        if per_round is not None:
            per_round[i].record()


def main():
    args = parse()
    if args.summarize_profile:
        summarize_profile(args.summarize_profile, args.config)
        return
    if args.summarize_diagnostics:
        summarize_diagnostics(args.summarize_diagnostics, args.config)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the update of one context does not "
                                   "span devices here (--gpus 1)"}))
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    global VT_COPIES
    VT_COPIES = not args.no_vt_copy
    import numpy as np
    import torch
    import synth
    import paper_2609_18935_amd as tu

    dev = "cuda:0"
    torch.cuda.set_device(0)
    tu.lib()
    cfg = synth.CONFIGS[args.config]
    a, d = cfg.attn, cfg.delta
    attn_p = tu.attn_params(a.n_q_heads, a.n_kv_heads, a.head_dim, a.rdim, a.rope_theta, a.softmax_scale,
                            kv_splits=args.kv_splits)
    delta_p = tu.delta_params(d.n_k_heads, d.n_v_heads, d.d_k, d.d_v, d.chunk, d.scale)
    W, K = args.warmup, args.steps
    if args.only_diagnostics:
        sc, chars, rounds, layers, _ = build_workload(cfg, args.seed, dev, tu)
        if not cfg.layer_kinds().count("attn") or len(chars) != 1:
            print(json.dumps({"error": "the diagnostics need one context with attention layers"}))
            sys.exit(2)
        row = diagnostics_row(tu, cfg, chars, rounds, layers, attn_p, delta_p, dev, K)
        print(json.dumps({"config": f"config {cfg.index}: {cfg.name}", "attention_diagnostics": row}), flush=True)
        return
    refill_steps = 0 if (args.no_refill or args.only_update) else args.refill_steps
    m = measure_update(tu, cfg, args.seed, dev, attn_p, delta_p, W, K, refill_steps, keep=not args.only_update)
    upd_ms, round_ms, kern, refill, sumT = m["upd_ms"], m["round_ms"], m["kern"], m["refill"], m["sumT"]
    chars, rounds = m["chars"], m["rounds"]
    n_rounds = len(rounds)
    stages = m["stages"]
    kinds = cfg.layer_kinds()
    # the attention kernel carries the workload's dominant work (it is MFMA-bound and on the
    # caller's stream); side-stream durations include waits for CUs it holds, so they are not
    # used to pick the dominant kernel
    dom = "attention" if "attention" in kern else max(kern, key=lambda n: kern[n]["ms_per_step"])
    if dom == "attention":
        units = attention_flops(cfg, rounds) * kinds.count("attn") / 1e12
        launches = kern[dom]["launches_per_step"]
        ach = units / (kern[dom]["ms_per_step"] / 1e3)
        roofline = {"bound": "mfma", "achieved": round(ach, 3), "peak": MFMA16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(ach / MFMA16_PEAK_TFLOPS, 4), "traffic": None, "kernel": dom,
                    "per_launch": round(units / launches, 6), "per_launch_unit": "TFLOP",
                    "avg_launch_ms": round(kern[dom]["avg_ms"], 5), "launches_per_step": launches}
    else:
        roofline = {"bound": None, "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None,
                    "kernel": dom}
    # HBM bytes per launch of the dominant kernel, from the committed counter passes
    traffic = measured_traffic(dom, cfg.index, f"config {cfg.index}: {cfg.name}")
    if traffic is not None:
        roofline["traffic"] = traffic["bytes_per_launch"]
        roofline["traffic_unit"] = "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
        roofline["traffic_detail"] = traffic

    extra = {}
    if not args.only_update:
        extra.update(headline_extras(tu, args, cfg, m, attn_p, delta_p, dev))
    del m
    torch.cuda.empty_cache()

    # ---- the other workloads: update time, refill speedup (per round for the 8-round
    # 32K workload, the >= 10x target at 32K contexts) and stage fractions
    if not args.only_update and args.extra_configs:
        rows = {}
        for ci in [int(x) for x in args.extra_configs.split(",") if x.strip() != ""]:
            if ci == cfg.index:
                continue
            c2 = synth.CONFIGS[ci]
            a2, d2 = c2.attn, c2.delta
            ap2 = tu.attn_params(a2.n_q_heads, a2.n_kv_heads, a2.head_dim, a2.rdim, a2.rope_theta, a2.softmax_scale,
                                 kv_splits=args.kv_splits)
            dp2 = tu.delta_params(d2.n_k_heads, d2.n_v_heads, d2.d_k, d2.d_v, d2.chunk, d2.scale)
            m2 = measure_update(tu, c2, args.seed, dev, ap2, dp2, min(W, 3), min(K, 10),
                                0 if args.no_refill else min(args.refill_steps, 3))
            rows[str(ci)] = config_row(m2)
            print(f"[bench] config {ci}: {json.dumps({k: v for k, v in rows[str(ci)].items() if k != 'kernels'})}",
                  file=sys.stderr, flush=True)
            del m2
            torch.cuda.empty_cache()
        extra["configs"] = rows

    # ---- revisions shaped like the paper's measured trace, through the 48-layer stack
    if not args.only_update and not args.no_paper_trace:
        a1, d1 = synth.CONFIGS[1].attn, synth.CONFIGS[1].delta
        ap1 = tu.attn_params(a1.n_q_heads, a1.n_kv_heads, a1.head_dim, a1.rdim, a1.rope_theta, a1.softmax_scale,
                             kv_splits=args.kv_splits)
        dp1 = tu.delta_params(d1.n_k_heads, d1.n_v_heads, d1.d_k, d1.d_v, d1.chunk, d1.scale)
        extra["paper_trace"] = paper_trace_row(tu, synth, dev, ap1, dp1, args.seed, min(K, 5))
        print(f"[bench] paper-shaped trace: {json.dumps(extra['paper_trace'])}", file=sys.stderr, flush=True)
        # ---- tail-length sweep at 32K surviving rows, with the single-refresh workload's shapes
        if not args.no_t_sweep:
            extra["t_sweep"] = t_sweep_row(tu, synth, dev, ap1, dp1, args.seed, min(K, 10))

    # ---- measured peaks of this part in this run: device copy bandwidth and a bf16 GEMM
    peaks = None if (args.no_peaks or args.only_update) else measured_peaks(dev)
    if peaks is not None:
        meas = peaks["bf16_gemm_tflops"] if roofline.get("bound") == "mfma" else peaks["copy_gbs"]
        if roofline.get("achieved") is not None and meas:
            roofline["measured_peak"] = meas
            roofline["frac_of_measured"] = round(roofline["achieved"] / meas, 4)
        for row in extra.values():
            if isinstance(row, dict) and "achieved" in row:
                row["frac_of_measured_copy"] = round(row["achieved"] / peaks["copy_gbs"], 4)
        print(f"[bench] measured peaks: {json.dumps(peaks)}", file=sys.stderr, flush=True)

    # the whole step against its roofline: the summed ideal time of every step of the path
    # (datasheet peaks; and the rates this part reached in this run, when measured)
    ideal = stack_ideal_ms(cfg, rounds, MFMA16_PEAK_TFLOPS, HBM_PEAK_GBS)
    stack_roofline = {"ideal_ms": round(ideal, 5), "measured_ms": round(upd_ms, 5), "frac": round(ideal / upd_ms, 4),
                      "peaks": {"mfma_tflops": MFMA16_PEAK_TFLOPS, "hbm_gbs": HBM_PEAK_GBS}}
    if peaks is not None:
        ideal_m = stack_ideal_ms(cfg, rounds, peaks["bf16_gemm_tflops"], peaks["copy_gbs"])
        stack_roofline.update({"ideal_ms_measured_peaks": round(ideal_m, 5),
                               "frac_of_measured_peaks": round(ideal_m / upd_ms, 4)})
    print(f"[bench] stack roofline: {json.dumps(stack_roofline)}", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline and not args.only_update:
        print("[bench] cpu oracle leg ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, args.seed, args.cpu_budget_s)

    line = {
        "metric": METRIC,
        "value": round(sumT / (upd_ms / 1e3), 1),
        "unit": "tail tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(upd_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"config {cfg.index}: {cfg.name}", "contexts": len(chars), "layers": len(kinds),
                   "attention_layers": kinds.count("attn"), "delta_layers": kinds.count("delta"),
                   "rounds": n_rounds, "tail_tokens": sumT, "surviving_rows": rounds[0]["L_keep"][:4],
                   "removed_rows": sum(o - k for R in rounds for o, k in zip(R["L_old"], R["L_keep"])),
                   "attn": f"{a.n_q_heads}q/{a.n_kv_heads}kv x {a.head_dim}",
                   "delta": f"{d.n_k_heads}k/{d.n_v_heads}v x {d.d_k}, chunk {d.chunk}"},
        "layout": {"vt_copies": VT_COPIES},
        "roofline": roofline,
        "stack_roofline": stack_roofline,
        "measured_peaks": peaks,
        "speedup_vs_refill": round(refill["speedup"], 3) if refill else None,
        "refill_ms": round(refill["ms"], 5) if refill else None,
        "refill_rounds": refill.get("rounds") if refill else None,
        "stages": stages,
        "extra_rows": extra,
        "kernels": {n: {k: (round(v, 6) if isinstance(v, float) else v) for k, v in kv.items()}
                    for n, kv in kern.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def diagnostics_row(tu, cfg, chars, rounds, layers, attn_p, delta_p, dev, K):
    """Attention diagnostics (Section 5.3) after the workload's first round: the float32
    reference-softmax probe of the last eight tail rows of every attention layer (averaged
    over layers), masses of 390-token memory groups with the effective group count, and
    the total variation between the probes of the first and the last attention layer.
    GPU time of the library's launches over K repetitions."""
    import torch
    a = cfg.attn
    (ctxs, own) = make_copy(tu, chars, layers, dev)
    up = round_updates(tu, ctxs, own, layers, rounds[:1], attn_p, delta_p)
    wsd = torch.empty(up[0].workspace_size(), dtype=torch.uint8, device=dev)
    run_step(up, wsd)
    torch.cuda.synchronize()
    ctx = ctxs[0]
    n_probe = min(8, ctx.len)
    att = [(L, O) for L, O in zip(layers, own) if L["kind"] == "attn"]
    qs = [rounds[0]["inputs"][i]["q"][-n_probe:].contiguous() for i, L in enumerate(layers) if L["kind"] == "attn"]
    probs = torch.zeros(ctx.len, dtype=torch.float32, device=dev)
    pws = torch.empty(lib_probe_ws(tu, attn_p, ctx.len, n_probe), dtype=torch.uint8, device=dev)
    first = torch.zeros_like(probs)
    last = torch.zeros_like(probs)

    def probe_all():
        probs.zero_()
        for (L, O), q in zip(att, qs):
            tu.attention_probe(ctx, O["caches"][0][0], attn_p, q, probs, weight=1.0 / len(att), workspace=pws)
    probe_all()
    tu.attention_probe(ctx, att[0][1]["caches"][0][0], attn_p, qs[0], first, workspace=pws)
    tu.attention_probe(ctx, att[-1][1]["caches"][0][0], attn_p, qs[-1], last, workspace=pws)
    groups = [(g, min(g + 390, ctx.next_pos)) for g in range(0, ctx.next_pos, 390)]
    gws = torch.empty(1 << 20, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    tu.profile_enable(True)      # GPU time of the library's launches (HIP events on the stream)
    for _ in range(K):
        probe_all()
        mass, win, summary = tu.attention_group_mass(ctx, probs, groups, window=8, workspace=gws)
        tv = tu.attention_tv_distance(first, last, workspace=gws)
    dp = tu.profile_collect()
    tu.profile_enable(False)
    probe_ms = dp["probe"][1] / K
    group_ms = dp["group_mass"][1] / K
    tv_ms = dp["tv_distance"][1] / K
    kbytes = ctx.len * a.n_kv_heads * a.head_dim * 2 * len(att)
    s = summary.cpu().tolist()
    row = {
        "probe_rows": n_probe, "layers": len(att), "live_rows": ctx.len, "probe_ms": round(probe_ms, 5),
        "probe_key_bytes": kbytes, "bound": "hbm",
        "achieved": round(kbytes / (probe_ms / 1e3) / 1e9, 1), "unit": "GB/s", "peak": HBM_PEAK_GBS,
        "groups": len(groups), "group_mass_ms": round(group_ms, 5), "tv_ms": round(tv_ms, 5),
        "memory_mass": round(s[0], 6), "effective_group_count": round(s[1], 3), "window_share": round(s[2], 5),
        "tv_first_last_attention_layer": round(float(tv[0]), 6) if len(att) > 1 else None,
        "timing": "GPU time of the library's launches (HIP events around each launch)"}
    del ctxs, own, up, wsd, pws, gws
    return row


def headline_extras(tu, args, cfg, m, attn_p, delta_p, dev):
    """Rows measured on the headline workload's shapes: delimiter removal after prefill,
    the slot-preserving and tail-and-relocate placements, the attention diagnostics and the
    short-convolution continuation."""
    import numpy as np
    import torch
    import synth
    W, K = args.warmup, args.steps
    a = cfg.attn
    chars, rounds, layers = m["chars"], m["rounds"], m["layers"]
    round_ms, upd_ms = m["round_ms"], m["upd_ms"]
    kinds = cfg.layer_kinds()
    sumT = m["sumT"]
    extra = {}
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    # ---- the same update with an 11-token opening and a 3-token closing maintenance
    # delimiter in every tail, removed from the caches once the tail is prefilled
    extra = {}
    if kinds.count("attn") and all(T >= 14 for R in rounds for T in R["T"]):
        def post(R):
            return [np.array([[c0, c0 + 11], [c0 + T - 3, c0 + T]]) for c0, T in zip(R["cursor"], R["T"])]
        # later rounds' removal ranges were drawn without delimiter holes; only the first
        # round of each context is run with delimiters
        rd = rounds[:1]
        copies3 = [make_copy(tu, chars, layers, dev) for _ in range(W + K)]
        ups3 = [round_updates(tu, ctxs, own, layers, rd, attn_p, delta_p, post=post) for (ctxs, own) in copies3]
        plain = [round_updates(tu, ctxs, own, layers, rd, attn_p, delta_p) for (ctxs, own) in copies3]
        ws3 = torch.empty(max(ups3[0][0].workspace_size(), plain[0][0].workspace_size()), dtype=torch.uint8,
                          device=dev)
        del plain
        for i in range(W):
            run_step(ups3[i], ws3)
        torch.cuda.synchronize()
        ev0.record()
        for i in range(W, W + K):
            run_step(ups3[i], ws3)
        ev1.record()
        torch.cuda.synchronize()
        post_ms = ev0.elapsed_time(ev1) / K
        first_ms = round_ms[0] if round_ms else upd_ms
        row_b = a.n_kv_heads * a.head_dim * 2
        moved = sum(T - 11 - 3 for T in rd[0]["T"])   # tail rows behind the first delimiter that survive
        extra["delimiter_removal"] = {
            "removed_rows_per_context": 14, "rounds": 1, "update_ms_with": round(post_ms, 5),
            "update_ms_without": round(first_ms, 5), "extra_ms": round(post_ms - first_ms, 5),
            "bytes": 2 * 2 * moved * row_b * kinds.count("attn"), "bound": "hbm"}
        print(f"[bench] delimiter removal: {json.dumps(extra['delimiter_removal'])}", file=sys.stderr, flush=True)
        del copies3, ups3, ws3

    # ---- the delta layers alone and the attention path alone
    extra["paths_alone"] = paths_alone_row(tu, cfg, m, attn_p, delta_p, dev, 1, min(K, 5))
    print(f"[bench] paths alone: {json.dumps(extra['paths_alone'])}", file=sys.stderr, flush=True)

    # ---- the placement arms the paper compares (Section 5.2): slot-preserving (rotated at
    # the removed records' slots) and tail-and-relocate (computed at the true tail, stored
    # keys then rotated to the slots), on the first round
    if kinds.count("attn"):
        rd = rounds[:1]
        first_ms = round_ms[0] if round_ms else upd_ms
        place_row = {"update_ms_true_tail": round(first_ms, 5)}
        for arm in ("slot", "relocate"):
            copies4 = [make_copy(tu, chars, layers, dev) for _ in range(W + 2 * K)]
            ups4 = [round_updates(tu, ctxs, own, layers, rd, attn_p, delta_p, arm=arm, place=slot_runs)
                    for (ctxs, own) in copies4]
            ws4 = torch.empty(ups4[0][0].workspace_size(), dtype=torch.uint8, device=dev)
            for i in range(W):
                run_step(ups4[i], ws4)
            torch.cuda.synchronize()
            ev0.record()
            for i in range(W, W + K):
                run_step(ups4[i], ws4)
            ev1.record()
            torch.cuda.synchronize()
            place_row[f"update_ms_{arm}"] = round(ev0.elapsed_time(ev1) / K, 5)
            if arm == "relocate":
                tu.profile_enable(True)
                for i in range(W + K, W + 2 * K):
                    run_step(ups4[i], ws4)
                rp = tu.profile_collect()
                tu.profile_enable(False)
                if "relocate" in rp:
                    c_, t_ = rp["relocate"]
                    rows = sum(rd[0]["T"]) * kinds.count("attn")
                    nbytes = rows * (2 * a.n_kv_heads * a.head_dim * 2 + 8)   # key rows read + written, labels
                    kms = t_ / c_
                    place_row["relocate_kernel"] = {
                        "launches_per_step": c_ / K, "avg_ms": round(kms, 5), "rows": rows, "bytes": nbytes,
                        "bound": "hbm", "achieved": round(nbytes / (t_ / K / 1e3) / 1e9, 1), "unit": "GB/s",
                        "peak": HBM_PEAK_GBS}
            del copies4, ups4, ws4
        extra["placement"] = place_row
        print(f"[bench] placements: {json.dumps(place_row)}", file=sys.stderr, flush=True)

    # ---- attention diagnostics (Section 5.3)
    if kinds.count("attn") and len(chars) == 1:
        extra["attention_diagnostics"] = diagnostics_row(tu, cfg, chars, rounds, layers, attn_p, delta_p, dev, K)
        print(f"[bench] attention diagnostics: {json.dumps(extra['attention_diagnostics'])}", file=sys.stderr,
              flush=True)

    # ---- the short-convolution continuation of one delta layer's q, k, v (width 4, SiLU)
    if kinds.count("delta"):
        extra["short_conv"] = short_conv_row(tu, synth, cfg, sumT, dev, K)
        print(f"[bench] short conv: {json.dumps(extra['short_conv'])}", file=sys.stderr, flush=True)
    return extra


if __name__ == "__main__":
    main()
