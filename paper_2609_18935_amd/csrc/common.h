// Shared device types and helpers of the tail-update library (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tu {

typedef uint16_t bf16_t;  // bfloat16 storage
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;
typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr int kMaxSeqPerLaunch = 32;
constexpr int kMaxSeqPerDelta = 48;   // (layer, context) items of one delta-rule launch
constexpr int kMaxRangesPerLaunch = 128;
constexpr int kMaxBufPerLaunch = 64;
constexpr int kMaxSeqPerCompact = 16;
// Every kernel takes its launch record by value; each record (all arguments of one
// kernel together) stays within this many bytes.
constexpr size_t kMaxKernargBytes = 4096;
constexpr int kScanRows = 1024;  // rows per keep-scan workgroup (a multiple of 256, at most 16K)
constexpr int kFlagStride = 32;   // compaction stripe counters sit one per 128-byte line
constexpr int kGatherStripeBytes = 256 * 16 * 16;  // threads x vectors x 16 B
constexpr int kAttnRows = 256;  // packed query rows per attention workgroup
constexpr int kAttnKeys = 64;   // keys per attention K/V tile
constexpr int kVtRow = kAttnKeys + 8;  // f16 per row of a packed V^T tile (64 keys + pad)

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// float -> bf16, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// double -> bf16, round to nearest even from the exact value. The double is first
// rounded to float with round-to-odd (truncate, then force the last bit to 1 when
// inexact); float carries 16 more significand bits than bf16, so the second
// rounding to bf16 is then correctly rounded (no double-rounding error).
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double x) {
  float f = (float)x;                       // round to nearest
  uint32_t u = __float_as_uint(f);
  double back = (double)f;
  if (back != x) {
    // step toward zero if the nearest float overshot |x|
    if (fabs(back) > fabs(x)) u -= 1u;
    u |= 1u;                                // sticky bit: round-to-odd
  }
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// XCD-aware remap: blocks are dispatched round-robin over the 8 XCDs (block b runs
// on XCD b % 8). Returns the work item for block b so that consecutive work items
// land on the same XCD and share its L2.
__device__ __forceinline__ int xcd_remap(int b, int n_blocks) {
  const int per = (n_blocks + 7) >> 3;
  const int xcd = b & 7;
  const int slot = b >> 3;
  return xcd * per + slot;
}

// Key order inside a 16-key group of a packed V^T tile: bits 2 and 3 swapped, so that
// the 8 keys one lane feeds to a P.V product are one contiguous 16-byte chunk.
// Workgroup barrier over LDS only: this wave's LDS accesses have completed when it
// arrives, while its global stores may still be in flight. For kernels whose
// workgroups never read back, within the kernel, what they stored to global memory
// (__syncthreads would also wait for those stores).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int key_slot(int k) {
  return (k & ~0xC) | ((k & 4) << 1) | ((k & 8) >> 1);
}

// ------------------------------------------------------------------ call status

// Device-check bits of one call (the kFault* values). The first 256 bytes of a call's
// workspace hold a 64-bit status word (call number in the high half, bits in the low
// half) and, 64 bytes further, the 32-bit number of the call that last ran there. Every
// call has its own number; kernels tag the bits they set with it, and every workgroup 0
// of the call's launches stores it as the last call's number. A reader takes the bits
// when the two numbers agree (and none otherwise), so no launch is needed to clear the
// word and stale bits of earlier calls are never reported.
struct CallStatus {
  unsigned long long* word;
  uint32_t* last;
  uint32_t call;
  uint32_t pad;
};

__device__ __forceinline__ void status_raise(const CallStatus& st, uint32_t bits) {
  unsigned long long old = __hip_atomic_load(st.word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    const uint32_t mine = (uint32_t)(old >> 32) == st.call ? (uint32_t)old : 0u;
    const unsigned long long want = ((unsigned long long)st.call << 32) | (mine | bits);
    if (want == old) return;
    const unsigned long long seen = atomicCAS(st.word, old, want);
    if (seen == old) return;
    old = seen;
  }
}

__device__ __forceinline__ void status_mark(const CallStatus& st) {
  if (blockIdx.x == 0 && threadIdx.x == 0) *st.last = st.call;
}

// ------------------------------------------------------------------ launch records

struct ScanSeq {
  const int32_t* pos;  // [L_old] positions of the cache rows (read only)
  int32_t* src_index;  // [L_old] out
  int32_t L_old;
  int32_t range_begin; // index into CompactArgs::ranges
  int32_t n_ranges;
  int32_t span_begin;  // index into CompactArgs::spans
  int32_t n_spans;
  int32_t block_begin; // first scan workgroup of this context
};

struct GatherSeq {
  int32_t* pos;         // d_pos of the context when this entry also moves positions, else null
  int32_t row_begin;    // first destination row handled (aligned, <= first moved row)
  int32_t n_keep;       // destination rows end
  int32_t n_stripes;
  int32_t item_begin;   // first item of this context
  int32_t buf_begin;    // index of its first buffer in CompactArgs::bufs
  int32_t n_buf;        // items per stripe: one per K/V buffer (the first also moves positions)
  int32_t flag_begin;   // its stripe read-counters
  int32_t window;       // stripes before s whose sources may reach stripe s's rows
  int32_t span_begin;   // index into CompactArgs::spans
  int32_t n_spans;
};

// One cooperative compaction launch: keep-scan for n_scan contexts and the row move
// for n_seq (context, buffer-group) entries.
struct CompactArgs {
  ScanSeq scan[kMaxSeqPerCompact];
  GatherSeq seq[kMaxSeqPerCompact];
  void* bufs[kMaxBufPerLaunch];
  int32_t ranges[kMaxRangesPerLaunch][2];  // position ranges [a, b) of the scan contexts
  int32_t spans[kMaxRangesPerLaunch][2];   // (kept rows before the span, span length) per removed span
  int32_t n_scan;          // scan contexts
  int32_t n_scan_blocks;   // scan workgroups (kScanRows rows each)
  int32_t n_seq;
  int32_t total_items;
  int32_t rows_per_stripe;
  int32_t row_bytes;
  int32_t n_flag_words;   // stripe counters x kFlagStride
  int32_t n_counter_words; // kFlagStride + n_flag_words: cleared by the scan launch
  int32_t n_workers;       // gather workgroups
  int32_t* claim;   // next unclaimed gather item (its own 128-byte line), then the flags
  int32_t* flags;   // [n_flag_words] stripe read counters, kFlagStride apart
  CallStatus status;
};

struct RopeSeq {
  const bf16_t* q;
  const bf16_t* k;
  const bf16_t* v;
  bf16_t* q_hat;
  bf16_t* k_cache;
  bf16_t* v_cache;
  int32_t* pos;
  int64_t cursor;
  int32_t L_keep;
  int32_t T;
  int32_t tok_begin;
  int32_t run_begin;   // slot placement: first entry in RopeArgs::runs (n_runs == 0: cursor + i)
  int32_t n_runs;
  int32_t pad;
};

constexpr int kMaxPlaceRunsPerLaunch = 32;   // TU_MAX_PLACE_RUNS

struct RopeArgs {
  RopeSeq seq[kMaxSeqPerLaunch];
  int32_t runs[kMaxPlaceRunsPerLaunch][2];   // (first position, first tail token) of each placement run
  int32_t n_seq;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t rotary_dim;
  int32_t pad;
  double theta;
};

// V^T packing of one context's key tiles [tile_begin, tile_end) (the rows of its V
// cache and, past L_keep, of the tail's values; RopeArgs::seq[i] of the same index).
struct PackSeq {
  _Float16* vt;          // [Hkv][head_tiles][D * kVtRow]
  int32_t tile_begin;
  int32_t tile_end;
  int32_t head_tiles;    // tiles per KV head in vt (its capacity)
  int32_t pack_begin;    // first packing workgroup of this context
};

struct PackArgs {
  PackSeq seq[kMaxSeqPerLaunch];
  int32_t n_seq;
  int32_t pack_items;    // packing workgroups
  CallStatus status;     // kFaultRange when a value exceeds f16
};

struct AttnSeq {
  const bf16_t* q_hat;   // [T][Hq][D]
  const bf16_t* k_cache; // [cap][Hkv][D]
  const _Float16* vt;    // [Hkv][head_tiles][D * kVtRow] packed f16 V^T tiles
  float* out;            // [T][Hq][D]
  _Float16* part_o;      // [splits][T*Hq][D] normalised split outputs (unused when splits == 1)
  float* part_ml;        // [splits][T*Hq][2] (reference max in log2 units, sum)
  int32_t L_keep;
  int32_t T;
  int32_t n_tiles;       // ceil(T*G / kAttnRows)
  int32_t n_splits;
  int32_t item_begin;    // first attention workgroup of this context
  int32_t head_tiles;    // tiles per KV head in vt
};

struct AttnArgs {
  AttnSeq seq[kMaxSeqPerLaunch];
  int32_t n_seq;
  int32_t total_items;   // attention workgroups
  int32_t n_q_heads;
  int32_t n_kv_heads;
  float scale_log2;      // softmax_scale * log2(e)
  int32_t pad;
};

constexpr int kXcds = 8;              // dies of the chip; workgroup b is dispatched to die b % 8
constexpr int kCus = 256;             // compute units of the chip
constexpr int kMaxAttnGroups = 256;   // entries of an attention launch's die table

// Placement of the attention workgroups of a launch on the dies. The items of a group
// (one context, kv head and key split: its query tiles) are consecutive; die x runs
// the groups [die_begin[x], die_begin[x + 1]) in that order, its workgroup slot s taking
// item grp_item0[g] + s - (slots of the die's earlier groups). Item numbers and slot
// counts are 16-bit; launches beyond that use the equal-share order.
struct AttnOrder {
  int32_t n_groups;                   // 0: equal item counts per die in item order (xcd_remap)
  int32_t blocks;                     // grid size
  int32_t die_begin[kXcds + 1];
  int32_t pad;
  uint16_t grp_item0[kMaxAttnGroups];
  uint16_t grp_end[kMaxAttnGroups];   // slots of the die up to and including group g
};

struct MergeArgs {
  AttnSeq seq[kMaxSeqPerLaunch];
  int32_t n_seq;
  int32_t n_q_heads;
  int32_t split_lanes;   // lanes per 8 output dims of a row (1, 2, 4 or 8), each a share of the splits
  int32_t row_begin[kMaxSeqPerLaunch + 1];  // prefix of T*Hq over contexts
};

struct DeltaSeq {
  const bf16_t* q;       // [T][Hk][dk]
  const bf16_t* k;
  const bf16_t* v;       // [T][Hv][dv]
  const float* beta;     // [T][Hv]
  const float* g;
  float* state;          // [Hv][dv][dk]
  float* out;            // [T][Hv][dv]
  int32_t T;
  int32_t n_chunks;
  int32_t chunk_begin;   // first global chunk index (workspace slot)
  int32_t pad;
};

struct DeltaArgs {
  DeltaSeq seq[kMaxSeqPerDelta];
  int32_t n_seq;
  int32_t n_k_heads;
  int32_t n_v_heads;
  int32_t total_chunks;
  float scale;
  int32_t n_slices;      // d_v slices per value head in the chain kernel
  CallStatus status;     // kFaultRange when an f16 operand overflows
  _Float16* ws_w;        // [chunks][Hv][C][dk]  W = T diag(beta 2^lg) K, d in operand order
  _Float16* ws_tv;       // [chunks][Hv][C][C]   T diag(beta)
  _Float16* ws_p;        // [chunks][Hv][C][max(C, 32)]  scale lower(G .* Q K^T), operand order
  float* ws_dec;         // [chunks][Hv][2][C]  decay factors 2^(lg_last - lg_s) and 2^lg_s
  _Float16* ws_q;        // [chunks][Hk][C][dk]  q in f16, d in operand order
  _Float16* ws_kt;       // [chunks][Hk][dk][max(C, 32)]  k^T in f16, s in operand order
};

// Key relocation: one workgroup per moved row; every key buffer of the launch gets the
// row's rotary pairs turned by delta positions, and d_pos (when given) the new label.
constexpr int kMaxRelocSpans = 64;
struct RelocArgs {
  bf16_t* bufs[kMaxBufPerLaunch];              // key caches [cap][Hkv][D]
  int32_t* pos;                                // d_pos, or null
  int32_t row[kMaxRelocSpans];                 // first row of each span
  int32_t delta[kMaxRelocSpans];               // position shift of each span
  int32_t block_begin[kMaxRelocSpans + 1];     // prefix of the span lengths
  int32_t n_spans;
  int32_t n_bufs;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t rotary_dim;
  int32_t pad;
  double theta;
};

// Attention diagnostics: probe of the last n_probe rows of one layer of one context.
constexpr int kProbeKeys = 64;       // keys per item of the probe score passes
constexpr int kProbeMaxRows = 128;   // n_probe x (query heads per KV head)
struct ProbeArgs {
  const bf16_t* q;       // [n_probe][Hq][D] raw queries of the probe rows
  bf16_t* q_hat;         // [n_probe][Hq][D] rotated (workspace)
  const bf16_t* k_cache; // [cap][Hkv][D]
  const int32_t* pos;    // d_pos
  float* stats;          // [Hq * n_probe][2] (max, 1 / sum) (workspace)
  float* part;           // [Hq * n_probe][n_parts][2] (max, sum of exp) per 32-key block (workspace)
  float* key_sum;        // [Hkv][ld] normalised scores summed over a KV head's rows (workspace)
  int32_t n_parts;       // 32-key blocks of a score row: ld / 32
  float* probs;          // [len] accumulated: probs += weight * mean distribution
  int32_t len;
  int32_t n_probe;
  int32_t ld;            // len rounded up to a multiple of kProbeKeys
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t rotary_dim;
  float scale;
  float weight;
  int32_t pad;
  double theta;
};

constexpr int kMaxGroupsPerLaunch = 256;
constexpr int kGroupMinRows = 1024;      // rows of one group-mass workgroup, at least
constexpr int kGroupMaxBlocks = 256;     // group-mass workgroups of a launch, at most
struct GroupArgs {
  int32_t range[kMaxGroupsPerLaunch][2];   // this launch's groups: sorted, disjoint position ranges
  const int32_t* pos;    // d_pos
  const float* probs;    // [len]
  double* partial;       // [n_blocks][2][n_total] per-workgroup mass, window mass (workspace)
  float* mass;           // [n_total]
  float* window_mass;    // [n_total] or null
  float* summary;        // [3] or null
  int32_t len;
  int32_t n;             // groups in this launch
  int32_t g_begin;       // index of its first group
  int32_t n_total;
  int32_t window;
  int32_t n_blocks;      // workgroups: min(kGroupMaxBlocks, ceil(len / kGroupMinRows)), at least 1
  int32_t block_rows;    // rows of one workgroup, a multiple of 256; n_blocks * block_rows >= len
};

constexpr int kTvRowsPerBlock = 4096;
struct TvArgs {
  const float* p;
  const float* q;
  const int32_t* map;    // row of q for each row of p, or null (identity)
  double* partial;       // [n_blocks] (workspace)
  float* tv;             // [1]
  int64_t n;
  int32_t n_blocks;
  int32_t pad;
};

// One tensor of a short-convolution launch: x [T][C] bf16, weights [C][W] bf16, state
// [W-1][C] bf16 (in place), out [T][C] bf16.
struct ConvJob {
  bf16_t* state;
  const bf16_t* x;
  const bf16_t* w;
  bf16_t* out;
  int32_t T;
  int32_t C;            // a multiple of 8
  int32_t act;          // 1: SiLU, 0: identity
  int32_t block_begin;  // first workgroup of this job
  int32_t n_cblocks;    // workgroups across the channels
  int32_t pad;
};

constexpr int kMaxConvJobs = 16;
struct ConvArgs {
  ConvJob job[kMaxConvJobs];
  int32_t n_jobs;
};

// ------------------------------------------------------------------ launchers
// (defined in the kernel translation units; return a hipError_t)
int compact_max_blocks();   // resident workgroups of the gather kernel over the device
// device-check bits of a call's status word (the values of TU_FAULT_*)
constexpr int32_t kFaultPositions = 1;
constexpr int32_t kFaultWait = 2;
constexpr int32_t kFaultRange = 4;
// one workgroup that only records a call's number (for calls that launch nothing else)
hipError_t launch_status_mark(const CallStatus& st, hipStream_t s);
constexpr int kMaxGatherWorkers = 2048;
hipError_t launch_compact(const CompactArgs& a, hipStream_t s);
// RoPE + append of the tail tokens and the V^T packing of every key tile, one launch
hipError_t launch_stage(const RopeArgs& r, int rope_tokens, const PackArgs& p, int head_dim, hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, const AttnOrder& o, int head_dim, hipStream_t s);
hipError_t launch_relocate(const RelocArgs& a, hipStream_t s);
hipError_t launch_probe(const ProbeArgs& a, hipStream_t s);
hipError_t launch_group_mass(const GroupArgs& a, hipStream_t s);
hipError_t launch_group_final(const GroupArgs& a, hipStream_t s);
hipError_t launch_tv(const TvArgs& a, hipStream_t s);
int conv_blocks(ConvJob& j, int block_begin);   // sets block_begin / n_cblocks, returns the job's workgroups
hipError_t launch_short_conv(const ConvArgs& a, int blocks, int width, hipStream_t s);
hipError_t launch_attention_merge(const MergeArgs& a, int total_rows, int head_dim, hipStream_t s);
hipError_t launch_delta_prep(const DeltaArgs& a, int d, int chunk, hipStream_t s);
hipError_t launch_delta_chain(const DeltaArgs& a, int d, int chunk, hipStream_t s);

}  // namespace tu
