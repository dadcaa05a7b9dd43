/*
 * tailupdate.h - C ABI of the true-tail hybrid-state update for MI355X (gfx950).
 *
 * A character context is the state (A_t, R_t, p_t) of the paper's Section 4.1:
 * the live attention KV cache of every attention layer, the recurrent state of
 * every gated delta-rule layer, and the next position id (the cursor). An
 * update removes the direct KV of superseded records (Eq. 2) and runs the
 * replacement tokens at the true tail: rotary positions p_t, p_t + 1, ...,
 * attention over the surviving plus new KV, and the recurrence continuing from
 * the carried state (Eq. 3). Section 4.2 fixes the bookkeeping: deletion ranges
 * are verified against the live spans first, removed positions become holes
 * (no placeholder rows), keys are never rotated back, and the cursor keeps
 * growing independently of the live length. The other placements the paper
 * compares (Section 5.2, Section 6.3) are available as variants of the stack
 * update (slot-preserving, tail-and-relocate) and as relocate_keys.
 *
 * Conventions for every call below
 *  - Device buffers are caller-owned; the library never allocates or frees
 *    device memory. Scratch memory is a caller-supplied workspace of at least
 *    the size returned by the matching *_workspace_size function (256-byte
 *    aligned), reused freely by the library within a call.
 *  - bf16 tensors are passed as `void*` to 16-bit bfloat16 storage.
 *  - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued
 *    asynchronously; calls on one context must be ordered by the caller's
 *    stream. Nothing here synchronises the device.
 *  - Every check happens on the host before anything is enqueued: an error
 *    return leaves all device buffers and all host metadata unchanged.
 *  - Status codes: TU_OK (0) or a negative TU_ERR_*; tu_last_error() returns a
 *    thread-local message for the last failure of the calling thread.
 *  - Checks that only the device can make (see tu_workspace_faults) report into the
 *    first word of the call's workspace.
 *  - Input range. Some products take operands rounded to f16 (10 stored mantissa
 *    bits, largest finite value 65504), because bf16 operands there would exceed the
 *    accuracy bound: attention values (v), and in the delta rule the state S, the
 *    pseudo-values U = T (beta v) - W S^T and their decayed copies, q, k and v
 *    themselves, and the WY factors. Inputs whose magnitudes reach 2^16 in these
 *    places have no f16 counterpart: the results are then not meaningful and the call sets
 *    TU_FAULT_RANGE in its status word. The delta rule expects L2-normalised keys
 *    (||k_t|| <= 1), beta in [0, 1] and g in [0, 1] (g = 0 is computed as 2^-100).
 */
#ifndef TAILUPDATE_H
#define TAILUPDATE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TU_ABI_VERSION 5

#define TU_OK 0
#define TU_ERR_ARG (-1)       /* null pointer, unsupported or inconsistent shape */
#define TU_ERR_RANGE (-2)     /* deletion range not sorted/disjoint/non-empty/live/below cursor */
#define TU_ERR_CAPACITY (-3)  /* surviving + tail rows exceed the cache capacity, or interval list full */
#define TU_ERR_WORKSPACE (-4) /* workspace missing or smaller than required */
#define TU_ERR_HIP (-5)       /* a HIP launch failed */

#define TU_MAX_RANGES 128     /* deletion ranges per context per call (and row spans they map to) */
#define TU_MAX_PLACE_RUNS 32  /* position runs of a slot-preserving or relocated tail */

#define TU_LAYER_ATTN 0
#define TU_LAYER_DELTA 1

/* Half-open interval [begin, end) of position ids. */
typedef struct tu_interval {
  int64_t begin;
  int64_t end;
} tu_interval;

/*
 * One character context (Section 4.1 state; D3/D4 bookkeeping of Section 4.2).
 * Host-side metadata plus the device position array. Cache rows [0, len) hold
 * the live tokens in the order they were computed (work order); d_pos labels each
 * row with its position. `live` lists the positions as runs in row order: run i
 * covers positions [begin, end) held by consecutive rows, runs are pairwise
 * disjoint, two consecutive runs are never position-contiguous (they would be one
 * run), and the lengths sum to `len`. With true-tail updates only, rows are in
 * increasing position order and the runs are sorted; slot-preserving and relocated
 * rows keep their work-order row but carry earlier positions.
 */
typedef struct tu_seq {
  int64_t len;        /* live rows */
  int64_t capacity;   /* rows allocated in d_pos and in each K/V buffer of this context */
  int64_t next_pos;   /* cursor p_t; every live position is below it */
  tu_interval* live;  /* host array [live_cap] */
  int32_t n_live;     /* intervals in use */
  int32_t live_cap;   /* intervals allocated */
  int32_t* d_pos;     /* device int32 [capacity]: position id of each cache row */
  /* Rows [0, vt_rows) of every attention layer's V^T copy (see tu_vt_cache_bytes) hold
   * the current values of those cache rows. 0 for a new context; the library lowers it
   * when rows move and raises it to len once every layer's copy is refreshed. */
  int64_t vt_rows;
} tu_seq;

/*
 * Attention-layer shape. Query head h reads KV head h / (n_q_heads / n_kv_heads).
 * head_dim must be 64, 128 or 256; rotary_dim even, 0 <= rotary_dim <= head_dim
 * (rotate-half pairs (j, j + rotary_dim/2), angle pos * rope_theta^(-2j/rotary_dim)).
 * kv_splits = 0 lets the library choose how many workgroups share one key range
 * (from the waves of workgroups a launch runs in; up to 128 for short tails over long
 * contexts); a value in [1, 64] forces that many splits (results are the same up to
 * rounding). Other values are rejected with TU_ERR_ARG.
 */
typedef struct tu_attn_params {
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t rotary_dim;
  double rope_theta;
  float softmax_scale;
  int32_t kv_splits;
} tu_attn_params;

/*
 * Gated delta-rule layer shape (Gated DeltaNet, cited in Section 4.1).
 * Value head h reads key/query head h / (n_v_heads / n_k_heads).
 * d_k = d_v in {64, 128}; chunk in {16, 32, 64}. `scale` multiplies S q.
 */
typedef struct tu_delta_params {
  int32_t n_k_heads;
  int32_t n_v_heads;
  int32_t d_k;
  int32_t d_v;
  int32_t chunk;
  float scale;
} tu_delta_params;

/* ABI version (TU_ABI_VERSION) and the calling thread's last error message. */
int tu_abi_version(void);
const char* tu_last_error(void);

/*
 * Device-side checks of a call. Section 4.2 keeps the live spans on the host while
 * the device holds the position labels: while scanning, the compaction kernels check
 * that every row the deletion ranges keep (by its d_pos label) lies outside the
 * removed row spans the host derived from its live runs, and every removed row
 * inside one; every bounded wait of the in-place move must end in time; and operands
 * rounded to f16 must be finite (see the input range above). A failed check does not
 * stop the call (moves follow the host's spans and stay in bounds): it sets a bit in
 * the status the call keeps in the first 256 bytes of its workspace (compact_kv,
 * tail_prefill_attention, delta_rule_continue, refresh_vt_cache and
 * update_layer_stack). Each call is numbered, the bits carry its number and its
 * kernels record it, so the status never needs clearing and never shows bits of an
 * earlier call (a call with nothing to enqueue, T = 0, leaves it as it was):
 *   TU_FAULT_POSITIONS  d_pos disagrees with the host metadata (`live`, `len`), so
 *                       the update did not remove exactly the rows whose labels lie
 *                       in the ranges;
 *   TU_FAULT_WAIT       a wait of the in-place move expired; moved rows may be wrong;
 *   TU_FAULT_RANGE      a value rounded to f16 overflowed; the results are not
 *                       meaningful.
 * tu_workspace_faults enqueues a read of that status on `stream` (the stream the
 * call ran on), synchronises `stream` and stores the last call's bits in *faults
 * (host pointer). Each call owns its workspace while it runs, so calls on other
 * streams with other workspaces never touch it. Returns TU_OK, TU_ERR_ARG (a null
 * pointer) or TU_ERR_HIP.
 */
#define TU_FAULT_POSITIONS 1
#define TU_FAULT_WAIT 2
#define TU_FAULT_RANGE 4
int tu_workspace_faults(const void* workspace, int32_t* faults, void* stream);

/*
 * Range verification (Section 4.2; host only, no device access).
 * ranges: host int64 [n_ranges][2] half-open position ranges. Accepts iff the
 * ranges are non-empty, sorted, pairwise disjoint, below seq->next_pos and each
 * lies entirely inside the live positions of `seq`. Writes the number of
 * removed rows to *n_removed (may be NULL). Returns TU_OK or TU_ERR_RANGE /
 * TU_ERR_ARG.
 */
int tu_validate_ranges(const tu_seq* seq, const int64_t* ranges, int32_t n_ranges,
                       int64_t* n_removed);

/*
 * KV invalidation, Eq. 2 (Section 4.1) with the Section 4.2 bookkeeping.
 * Removes the rows whose positions fall in `ranges` from every attention layer
 * of one context, keeping the surviving rows in order and bit-identical.
 *  k_layers, v_layers: host arrays [n_layers] of device bf16 [capacity][n_kv_heads][head_dim].
 *  src_index: optional device int32 [>= seq->len]; on success entry j (< new len)
 *             holds the old row index of the j-th surviving row. May be NULL.
 * On success seq->len and seq->live are updated (seq->vt_rows drops to the first
 * removed row); seq->next_pos is unchanged.
 * The device kernels compute the keep mask from d_pos, turn it into offsets by
 * wavefront prefix sums, and move only the rows behind the first hole, in place.
 */
size_t compact_kv_workspace_size(int64_t len, int32_t n_layers, int32_t n_kv_heads, int32_t head_dim);
int compact_kv(tu_seq* seq, void* const* k_layers, void* const* v_layers, int32_t n_layers,
               int32_t n_kv_heads, int32_t head_dim, const int64_t* ranges, int32_t n_ranges,
               int32_t* src_index, void* workspace, size_t workspace_bytes, void* stream);

/*
 * compact_kv for callers that cannot allocate (code under graph capture, serving loops
 * that forbid allocation): the same removal, with the call's scratch (the index list
 * when src_index is NULL, the move's counters) in a fixed array the library holds on
 * every GPU it runs on, TU_NOALLOC_SCRATCH_BYTES (8 MiB) per GPU, kept until the
 * process ends. No allocation of any kind. A call whose scratch would exceed the array
 * fails with TU_ERR_WORKSPACE before anything is enqueued (with 1 KB cache rows,
 * contexts up to about 1.3M rows fit). Calls on one GPU share the array: calls that
 * overlap in time on that GPU (other streams or threads) race and must not be made.
 *  status: optional device buffer of 256 bytes (16-byte aligned) that receives the
 *          call's device-check status (read it with tu_workspace_faults(status, ...));
 *          NULL keeps the status in the scratch, where it cannot be read.
 * Every other argument, and the result, as for compact_kv.
 */
#define TU_NOALLOC_SCRATCH_BYTES (8u << 20)
int compact_kv_noalloc(tu_seq* seq, void* const* k_layers, void* const* v_layers, int32_t n_layers,
                       int32_t n_kv_heads, int32_t head_dim, const int64_t* ranges, int32_t n_ranges,
                       int32_t* src_index, void* status, void* stream);

/*
 * Persistent V^T copy of one attention layer's value cache (optional, caller-owned):
 * the values in the f16 transposed tile layout the attention kernel reads (64 keys
 * per tile; the layout is private to the library). With a copy, a call refreshes only
 * the tiles from row seq->vt_rows on (the rows a removal moved, and the tail), instead
 * of packing every row of the cache into the workspace on every call. Bytes of a copy
 * for `capacity` rows (0 for invalid shapes); 16-byte aligned device memory.
 */
size_t tu_vt_cache_bytes(int64_t capacity, int32_t n_kv_heads, int32_t head_dim);

/*
 * Brings the V^T copies of up to 32 attention layers of one context up to date: rows
 * [seq->vt_rows, seq->len) of each value cache are packed (with the rest of their
 * 64-row tiles), then seq->vt_rows = seq->len. For a copy attached to a context that
 * already holds rows (vt_rows 0 packs every row). v_layers, vt_layers: host arrays
 * [n_layers] of device pointers (bf16 [capacity][n_kv_heads][head_dim] caches, copies
 * of tu_vt_cache_bytes(seq->capacity, ...)). The workspace holds only the status word
 * (256 bytes; TU_FAULT_RANGE for values without an f16 counterpart).
 */
int refresh_vt_cache(tu_seq* seq, void* const* v_layers, void* const* vt_layers, int32_t n_layers, int32_t n_kv_heads,
                     int32_t head_dim, void* workspace, size_t workspace_bytes, void* stream);

/*
 * True-tail attention of one layer, Eq. 3 (Section 4.1): rotary embedding of the
 * T tail tokens at positions seq->next_pos + i (angles in float64, results
 * rounded to bf16 round-to-nearest-even), append of the rotated keys and the
 * values at cache rows [seq->len, seq->len + T) (and their positions in d_pos),
 * then causal grouped-query softmax attention: tail row i attends to cache rows
 * 0 .. seq->len + i.
 *  q: device bf16 [T][n_q_heads][head_dim]; k, v: device bf16 [T][n_kv_heads][head_dim]
 *     (k before rotation).
 *  out: device fp32 [T][n_q_heads][head_dim].
 *  q_hat: optional device bf16 [T][n_q_heads][head_dim] receiving the rotated queries.
 *  vt_cache: optional V^T copy of this layer (tu_vt_cache_bytes(seq->capacity, ...));
 *     tiles from row seq->vt_rows on are refreshed. NULL: every tile is packed into the
 *     workspace.
 * Does not change `seq` (several layers share one context): call commit_tail once
 * after the last layer, or use update_layer_stack.
 */
size_t tail_prefill_attention_workspace_size(const tu_attn_params* p, int64_t T, int64_t len);
int tail_prefill_attention(const tu_seq* seq, void* k_cache, void* v_cache, void* vt_cache, const tu_attn_params* p,
                           const void* q, const void* k, const void* v, int64_t T, float* out,
                           void* q_hat, void* workspace, size_t workspace_bytes, void* stream);

/* Advance a context by T appended tokens: len += T, live gains [next_pos, next_pos+T),
 * next_pos += T (Section 4.2: the cursor grows by every appended token); vt_rows
 * becomes len (every layer's V^T copy, if any, was refreshed by
 * tail_prefill_attention). Host only. */
int commit_tail(tu_seq* seq, int64_t T);

/*
 * Recurrence continuation, Eq. 3 for a gated delta-rule layer: from the carried
 * state, for each tail token t
 *   S <- g_t * S (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,   o_t = scale * S q_t,
 * evaluated in chunks of p->chunk tokens (chunk-parallel WY preparation, then a
 * sequential chain over chunks with the fp32 state held on chip).
 *  state: device fp32 [n_v_heads][d_v][d_k], updated in place.
 *  q, k:  device bf16 [T][n_k_heads][d_k];  v: device bf16 [T][n_v_heads][d_v].
 *  beta, g: device fp32 [T][n_v_heads];  out: device fp32 [T][n_v_heads][d_v].
 */
size_t delta_rule_continue_workspace_size(const tu_delta_params* p, int64_t T);
int delta_rule_continue(float* state, const void* q, const void* k, const void* v, const float* beta,
                        const float* g, int64_t T, const tu_delta_params* p, float* out,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * Convolution-state continuation (Section 4.1 and Fig. 2: the recurrent layers'
 * convolution state continues over the replacement tokens without rollback),
 * read as the short depthwise causal convolution of Gated DeltaNet layers. For
 * each tail token t and channel c of one projected tensor
 *   y_t[c] = act( sum_{j<width} w[c][j] * xt[t + j][c] ),
 * where xt is the width-1 carried rows followed by the T new rows; act is SiLU
 * (x * sigmoid(x), TU_CONV_SILU) or the identity (TU_CONV_IDENTITY). Products
 * are summed in fp32 in tap order and rounded to bf16 (nearest even).
 *  state:  device bf16 [width-1][channels], the last width-1 input rows of the
 *          context; replaced in place by the last width-1 rows of xt (may be NULL
 *          when width == 1).
 *  x:      device bf16 [T][channels] new rows (before the convolution).
 *  weight: device bf16 [channels][width], tap width-1 multiplies the newest row.
 *  out:    device bf16 [T][channels]; must not overlap x or state.
 * channels: a positive multiple of 8; width 1 .. 8. T == 0 leaves state unchanged.
 * Needs no workspace. Errors: TU_ERR_ARG (sizes, activation, null or misaligned
 * pointers), TU_ERR_HIP (launch failure).
 */
#define TU_CONV_IDENTITY 0
#define TU_CONV_SILU 1
int short_conv_continue(void* state, const void* x, const void* weight, int64_t T, int32_t channels, int32_t width,
                        int32_t activation, void* out, void* stream);

/* Several independent tensors (e.g. the q, k and v projections of a layer, or the
 * layers and contexts of a stack) in as few launches as possible: up to 16 tensors
 * share one launch. Every field has the meaning it has in short_conv_continue;
 * width and activation are common. All tensors are checked before any launch. */
typedef struct tu_conv_tensor {
  void* state;          /* device bf16 [width-1][channels], in place */
  const void* x;        /* device bf16 [T][channels] */
  const void* weight;   /* device bf16 [channels][width] */
  void* out;            /* device bf16 [T][channels] */
  int64_t T;
  int32_t channels;
  int32_t reserved;     /* 0 */
} tu_conv_tensor;
int short_conv_continue_batch(const tu_conv_tensor* tensors, int32_t n, int32_t width, int32_t activation,
                              void* stream);

/*
 * Placement of a context's replacement tokens (Section 5.2; compared in Section 6.3):
 *  TU_PLACE_TAIL      the method: rotated and kept at the next positions
 *                     next_pos, next_pos + 1, ...; the cursor advances by T.
 *  TU_PLACE_SLOT      slot-preserving maintenance: computed at the causal work tail
 *                     (after every surviving row) but rotated at the positions of
 *                     `place_runs`, which the rows then keep; the cursor becomes
 *                     max(next_pos, last placed position + 1).
 *  TU_PLACE_RELOCATE  tail-and-relocate: computed exactly as TU_PLACE_TAIL, then the
 *                     stored keys are rotated from their tail positions to those of
 *                     `place_runs` and the rows relabelled (values and recurrent state
 *                     untouched); the cursor advances by T (or past the last placed
 *                     position if that is further).
 * place_runs: host int64 [n_place_runs][2] half-open position ranges, in tail order:
 * the T tail tokens take their positions one run after the other (the lengths sum to
 * T); the runs are disjoint, free of live positions after this call's removals, and
 * below 2^31 - 1. At most TU_MAX_PLACE_RUNS runs.
 */
#define TU_PLACE_TAIL 0
#define TU_PLACE_SLOT 1
#define TU_PLACE_RELOCATE 2

/* One context's part of a stack update. */
typedef struct tu_seq_update {
  tu_seq* seq;
  const int64_t* ranges;  /* host int64 [n_ranges][2], may be NULL when n_ranges == 0 */
  int32_t n_ranges;
  int64_t T;              /* tail tokens */
  int32_t* src_index;     /* optional device int32 [>= seq->len] (see compact_kv) */
  /* Rows removed once the tail is prefilled (Section 4.1: temporary maintenance
   * delimiters whose direct KV are subsequently removed; Section 4.2): host int64
   * [n_post_ranges][2] half-open position ranges made of this call's tail positions
   * (their final positions: [next_pos, next_pos + T) for TU_PLACE_TAIL, the placed
   * positions otherwise), sorted, disjoint, non-empty. May be NULL when
   * n_post_ranges == 0. */
  const int64_t* post_ranges;
  int32_t n_post_ranges;
  int32_t placement;            /* TU_PLACE_TAIL (0), TU_PLACE_SLOT or TU_PLACE_RELOCATE */
  const int64_t* place_runs;    /* host [n_place_runs][2]; NULL for TU_PLACE_TAIL */
  int32_t n_place_runs;
} tu_seq_update;

/*
 * One layer of the stack. Tail inputs of all contexts are packed in context
 * order: context s owns rows [sum of earlier T, + T_s).
 *  attention: k_cache[s], v_cache[s] device bf16 caches, vt_cache[s] an optional
 *             V^T copy; q, k, v, out as in tail_prefill_attention; beta, g, state
 *             unused.
 *  delta:     state[s] device fp32 [Hv][d_v][d_k]; q, k, v, beta, g, out as in
 *             delta_rule_continue; k_cache, v_cache unused.
 */
typedef struct tu_layer_io {
  int32_t kind;                /* TU_LAYER_ATTN or TU_LAYER_DELTA */
  void* const* k_cache;        /* host array [n_seq] of device pointers */
  void* const* v_cache;
  void* const* vt_cache;       /* attention: NULL, or host array [n_seq] of V^T copies (entries may be NULL) */
  float* const* state;         /* host array [n_seq] of device pointers */
  const void* q;
  const void* k;
  const void* v;
  const float* beta;
  const float* g;
  float* out;
} tu_layer_io;

typedef struct tu_update {
  int32_t n_seq;
  tu_seq_update* seqs;         /* host array [n_seq] */
  int32_t n_layers;
  const tu_layer_io* layers;   /* host array [n_layers], in model order */
  tu_attn_params attn;
  tu_delta_params delta;
} tu_update;

/*
 * Whole update of a hybrid layer stack for n_seq contexts (Eq. 1-3): verify every
 * context's ranges, placement and capacity; compact every attention layer's cache
 * once per context (one index list per context, reused by all attention layers);
 * then, in layer order, tail attention for attention layers and recurrence
 * continuation for delta layers, batched over the contexts; then relocate the keys
 * of TU_PLACE_RELOCATE contexts; then remove each context's post-prefill rows
 * (post_ranges) from every attention layer; finally commit each context's metadata
 * (len = survivors + T - post-removed rows, live runs, cursor as the placement
 * says: the positions of post-removed rows become holes, and the recurrent state
 * keeps their influence). A full refill is the same call on empty contexts (len 0)
 * with zero states.
 * Every context's vt_rows ends at its new len (V^T copies refreshed), or at the first
 * row the post-prefill removal moved.
 * Delta layers read nothing the attention path writes, so they run concurrently
 * with it on a side stream of the current device, forked after the work already
 * queued on `stream` and joined back into `stream` before the call returns (also
 * when a launch fails): all results are ordered on `stream`. The side stream and the
 * two events of the fork and join are the library's only state besides the
 * thread-local error message: created on the first such call of a thread on a
 * device (default priority, non-blocking) and kept for the thread's life.
 * tu_validate_update performs only the host checks (no device access).
 */
size_t update_layer_stack_workspace_size(const tu_update* u);
int tu_validate_update(const tu_update* u);
int update_layer_stack(const tu_update* u, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Key relocation (Section 5.2, tail-and-relocate: stored keys rotated to other
 * positions; values, row order and recurrent state unchanged). For every move
 * (src_begin, src_end, dst_begin) the rows holding positions [src_begin, src_end)
 * get their keys rotated by delta = dst_begin - src_begin, pair (j, j + r/2) by the
 * angle delta * theta^(-2j/r) (float64 angle and rotation of the stored bf16 value,
 * rounded to bf16 nearest even), and are relabelled with positions + delta.
 *  k_layers: host array [n_layers] of device bf16 [capacity][n_kv_heads][head_dim]
 *            key caches (the attention layers of the context; n_layers may be 0 to
 *            relabel positions only). p: head shape, rotary_dim and rope_theta.
 *  moves:    host int64 [n_moves][3]; sources sorted, disjoint and live;
 *            destinations disjoint and not held by rows that stay; below 2^31 - 1.
 * On success seq->live is relabelled and seq->next_pos becomes
 * max(next_pos, last destination + 1). Needs no workspace. At most TU_MAX_RANGES
 * moves (and row spans they map to). Errors: TU_ERR_ARG, TU_ERR_RANGE, TU_ERR_HIP.
 */
int relocate_keys(tu_seq* seq, void* const* k_layers, int32_t n_layers, const tu_attn_params* p,
                  const int64_t* moves, int32_t n_moves, void* stream);

/*
 * Attention diagnostics (Section 5.3, Appendix C). The probe queries are the last
 * n_probe rows of a context; probe query i sees rows 0 .. len - n_probe + i (the
 * causal rule of the update). Their raw queries are rotated at the rows' positions
 * (float64 angles, bf16 nearest even, as the cached keys were); scores
 * softmax_scale * q.k are products of the bf16 values summed in fp32; the reference
 * softmax over the visible rows is fp32. Holes hold no rows, so they are in no
 * denominator.
 *
 * attention_probe: probs[j] += weight * (mean over the n_probe queries and all query
 * heads of the softmax probability of row j), for j < seq->len (rows no query sees
 * get 0). Averaging layers: call once per attention layer with weight 1 / layers.
 *  k_cache: device bf16 [capacity][n_kv_heads][head_dim] of the layer;
 *  q:       device bf16 [n_probe][n_q_heads][head_dim] raw queries of the probe rows;
 *  probs:   device fp32 [>= seq->len], read and written.
 *  1 <= n_probe <= len, n_probe * n_q_heads / n_kv_heads <= 128. The workspace
 *  holds the rotated queries and per-row and per-key partial sums (about
 *  (n_probe * n_q_heads / 4 + n_kv_heads) x len floats); no score row is stored.
 *
 * attention_group_mass: memory groups given as host int64 [n_groups][2] position
 * ranges (sorted, disjoint; one per record). mass[g] = sum of probs over the rows whose
 * position lies in group g; window_mass[g] (optional) the same over the group's first
 * `window` positions (the paper uses 8); summary (optional, device fp32 [3]) = {memory
 * mass M = sum_g mass[g], effective group count exp(-sum_g a_g log a_g) with
 * a_g = mass[g] / M, boundary-window share sum_g window_mass[g] / M}. Summed in
 * float64 in a fixed order (the same bits on every run), reported as fp32.
 *
 * attention_tv_distance: tv[0] = 0.5 * sum_j |p[j] - q[map(j)]| over j < n, where
 * map = q_row_of_p (device int32 [n], the row of the same token in the other
 * construction) or the identity when NULL. Float64 partial sums in a fixed order.
 */
size_t attention_probe_workspace_size(const tu_attn_params* p, int64_t len, int32_t n_probe);
int attention_probe(const tu_seq* seq, const void* k_cache, const tu_attn_params* p, const void* q, int32_t n_probe,
                    float weight, float* probs, void* workspace, size_t workspace_bytes, void* stream);
size_t attention_group_mass_workspace_size(int64_t len, int32_t n_groups);
int attention_group_mass(const tu_seq* seq, const float* probs, const int64_t* groups, int32_t n_groups,
                         int32_t window, float* mass, float* window_mass, float* summary, void* workspace,
                         size_t workspace_bytes, void* stream);
size_t attention_tv_workspace_size(int64_t n);
int attention_tv_distance(const float* p, const float* q, const int32_t* q_row_of_p, int64_t n, float* tv,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * Kernel timing (diagnostics, not part of the update). While enabled for the
 * calling thread, every kernel the library launches is bracketed by two HIP
 * events recorded on the launch's stream. tu_profile_collect waits for those
 * events, then reports per kernel name (NUL-terminated, `name_stride` bytes per
 * entry in `names`) the launch count and the summed duration in milliseconds,
 * for at most `max_entries` kernels; it returns the number of entries written
 * (or a negative status) and clears the records. Names (one per launch or pair
 * of launches): compact (keep-scan, then gather), rope_vt_pack (RoPE + append of
 * the tail with the V^T packing of the key tiles), attention, attention_merge,
 * delta_prep, delta_chain, short_conv, relocate, probe, group_mass, tv_distance.
 */
int tu_profile_enable(int on);
int tu_profile_collect(char* names, int32_t name_stride, int32_t* counts, double* total_ms, int32_t max_entries);

#ifdef __cplusplus
}
#endif

#endif /* TAILUPDATE_H */
