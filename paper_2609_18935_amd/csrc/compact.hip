// KV invalidation (paper Section 4.1, Eq. 2): keep mask, prefix-sum offsets and the
// order-preserving in-place move of the surviving rows, in two launches on the
// caller's stream. The first scans the old positions (before anything moves them) and
// clears the move's counters; the second moves the rows.
//
// Scan workgroups (k_compact_scan, kScanRows rows each): rounds of
// 256 consecutive rows, one row per lane, so every load is coalesced. A lane's keep
// flag is "position in no deletion range"; the wavefront ballot + mbcnt gives each
// kept row its rank inside the wave, one wave scans the 64 per-(round, wave) counts,
// and the rows kept before the workgroup's first row (from the verified spans) give
// the destination. They write src_index; a row whose keep flag disagrees with the
// host's live spans sets kFaultPositions in the call's status word.
//
// Gather workgroups (k_compact_gather): move whole rows of every attention layer's K and V
// buffers, and the position array, in place, only from the first removed row on. The
// source of destination row j is j plus the lengths of the removed row spans that
// start at or before it (spans are verified on the host), so moving rows does not
// wait for the scan. Sources never precede destinations, so rows only move toward the
// front. Work is a sequence of (stripe, buffer) items that workgroups claim in
// increasing order from an atomic counter. An item loads its source rows into
// registers, bumps its stripe's read counter, waits until every earlier stripe whose
// sources can reach its destination rows has been read by all buffers, then stores.
// Every wait targets smaller items, which running workgroups have already claimed, and
// the workgroup holding the smallest unfinished item never waits, so the scheme
// progresses without any guarantee about which workgroups are resident: an ordinary
// launch on the caller's stream. One lane polls, with back-off, counters that sit on
// separate cache lines. Each wait is also bounded: on expiry the item proceeds, the
// call's status word gets kFaultWait, and every wave exits.
#include <atomic>

#include "common.h"

namespace tu {

namespace {

constexpr int kThreads = 256;
constexpr int kScanRounds = kScanRows / kThreads;
constexpr int kScanWaves = kThreads / 64;
constexpr int kGatherVec = kGatherStripeBytes / (kThreads * 16);   // 16-byte vectors per thread
constexpr int kPosVec = (kGatherStripeBytes / 16 + kThreads - 1) / kThreads;  // positions per thread
constexpr long kSpinLimit = 1l << 20;                               // bounded wait per counter

__device__ __forceinline__ int lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// The launch's removed spans as old-row intervals [first, end), in LDS: span q of a
// context starts at (kept rows before it) + (rows of the context's earlier spans).
__device__ __forceinline__ void stage_spans(const CompactArgs& a, int32_t (*sp)[2]) {
  for (int i = threadIdx.x; i < kMaxRangesPerLaunch; i += kThreads) {
    sp[i][0] = a.spans[i][0];
    sp[i][1] = a.spans[i][1];
  }
}

// Number of removed rows before old row i.
__device__ __forceinline__ int removed_before(const int32_t (*sp)[2], int span_begin, int n_spans, int i) {
  int full = 0, removed = 0;
  for (int q = 0; q < n_spans; ++q) {
    const int row = sp[span_begin + q][0] + full;   // old row of the span start
    if (row >= i) break;
    removed = full + min(sp[span_begin + q][1], i - row);
    full += sp[span_begin + q][1];
  }
  return removed;
}

// Old row that destination row j of a context receives: j plus the lengths of the
// removed spans whose start, counted in kept rows, is at or before j.
__device__ __forceinline__ int source_row(const int32_t (*sp)[2], const GatherSeq& S, int j) {
  int src = j;
  for (int q = 0; q < S.n_spans; ++q) {
    if (sp[S.span_begin + q][0] > j) break;
    src += sp[S.span_begin + q][1];
  }
  return src;
}

// One scan workgroup: kScanRows consecutive old rows of one context.
__device__ void keep_scan(const CompactArgs& a, const ScanSeq& s, int chunk) {
  __shared__ int32_t rng[kMaxRangesPerLaunch][2];
  __shared__ int32_t sp[kMaxRangesPerLaunch][2];
  __shared__ int32_t cnt[kScanRounds * kScanWaves];
  __shared__ int32_t off[kScanRounds * kScanWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < s.n_ranges; i += kThreads) {
    rng[i][0] = a.ranges[s.range_begin + i][0];
    rng[i][1] = a.ranges[s.range_begin + i][1];
  }
  stage_spans(a, sp);
  const int base = chunk * kScanRows;
  int32_t p[kScanRounds];
  uint64_t m[kScanRounds];
#pragma unroll
  for (int r = 0; r < kScanRounds; ++r) {
    const int idx = base + r * kThreads + tid;
    p[r] = idx < s.L_old ? s.pos[idx] : 0;
  }
  __syncthreads();
  bool bad = false;
#pragma unroll
  for (int r = 0; r < kScanRounds; ++r) {
    const int idx = base + r * kThreads + tid;
    bool keep = idx < s.L_old;
    for (int q = 0; q < s.n_ranges; ++q) keep = keep && !(p[r] >= rng[q][0] && p[r] < rng[q][1]);
    // the device positions must agree with the host's live spans: the row is kept
    // exactly when it lies in no removed row span
    bool in_span = false;
    for (int q = 0, full = 0; q < s.n_spans; ++q) {
      const int first = sp[s.span_begin + q][0] + full;
      const int len = sp[s.span_begin + q][1];
      in_span = in_span || (idx >= first && idx < first + len);
      full += len;
    }
    bad |= idx < s.L_old && keep == in_span;
    m[r] = __ballot(keep);
    if (lane == 0) cnt[r * kScanWaves + wave] = __popcll(m[r]);
  }
  __syncthreads();
  if (wave == 0) {
    // per-(round, wave) counts in row order; lane owns one
    const int c = lane < kScanRounds * kScanWaves ? cnt[lane] : 0;
    int incl = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(incl, d, 64);
      if (lane >= d) incl += y;
    }
    if (lane < kScanRounds * kScanWaves) off[lane] = incl - c;
  }
  __syncthreads();
  // rows kept before this chunk, from the verified spans
  const int kept_before = base - removed_before(sp, s.span_begin, s.n_spans, base);
#pragma unroll
  for (int r = 0; r < kScanRounds; ++r) {
    const int idx = base + r * kThreads + tid;
    if ((m[r] >> lane) & 1ull) s.src_index[kept_before + off[r * kScanWaves + wave] + lane_rank(m[r])] = idx;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0 && bad) status_raise(a.status, kFaultPositions);
}

__device__ bool gather_items(const CompactArgs& a) {
  __shared__ int32_t s_src[kGatherStripeBytes / 16];
  __shared__ int32_t sp[kMaxRangesPerLaunch][2];
  __shared__ int32_t s_item;
  bool expired = false;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.rows_per_stripe;
  const int RB = a.row_bytes;
  const int vpr = RB >> 4;  // 16-byte vectors per row
  // with no more items than workgroups every workgroup's single claim gets an item, so
  // none claims again (a claim is a device-scope round trip, longer when many
  // workgroups claim at once)
  const bool one_each = a.n_workers >= a.total_items;
  for (bool first = true;; first = false) {
    if (tid == 0) s_item = __hip_atomic_fetch_add(a.claim, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (first) stage_spans(a, sp);   // overlaps the first claim's round trip
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(s_item);
    if (item >= a.total_items) break;
    int si = 0;
    while (si + 1 < a.n_seq && a.seq[si + 1].item_begin <= item) ++si;
    const GatherSeq& S = a.seq[si];
    const int local = item - S.item_begin;
    const int stripe = local / S.n_buf;
    const int b = local - stripe * S.n_buf;
    const bool with_pos = S.pos != nullptr && b == 0;   // the first buffer's item also moves positions
    char* buf = (char*)a.bufs[S.buf_begin + b];
    const int row0 = S.row_begin + stripe * R;
    const int rows = min(R, S.n_keep - row0);
    // source row of each destination row of the stripe
    for (int t = tid; t < rows; t += kThreads) s_src[t] = source_row(sp, S, row0 + t);
    __syncthreads();
    const int n_vec = rows * vpr;
    u32x4 data[kGatherVec];
#pragma unroll
    for (int i = 0; i < kGatherVec; ++i) {
      const int e = tid + i * kThreads;
      if (e < n_vec) {
        const int r = e / vpr;
        data[i] = *(const u32x4*)(buf + (long)s_src[r] * RB + (long)(e - r * vpr) * 16);
      }
    }
    int32_t pv[kPosVec];
    if (with_pos) {
#pragma unroll
      for (int i = 0; i < kPosVec; ++i) {
        const int t = tid + i * kThreads;
        if (t < rows) pv[i] = S.pos[s_src[t]];
      }
    }
    // every source value of this item is in registers before its counter moves
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (wave == 0) {
      if (lane == 0)
        __hip_atomic_fetch_add(a.flags + kFlagStride * (S.flag_begin + stripe), 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
      // the wave polls up to 64 earlier stripes at once, nearest first; a lane skips a
      // stripe whose source rows (an increasing function of its destination rows, so
      // within [source of its first row, source of its last row]) miss this stripe's rows
      const int lo = max(0, stripe - S.window);
      for (int w0 = stripe - 1; w0 >= lo; w0 -= 64) {
        const int w = w0 - lane;
        bool done = w < lo;
        if (!done) {
          const int first = S.row_begin + w * R;
          const int last = min(first + R, S.n_keep) - 1;
          done = source_row(sp, S, last) < row0 || source_row(sp, S, first) >= row0 + rows;
        }
        long spins = 0;
        for (;;) {
          if (!done)
            done = __hip_atomic_load(a.flags + kFlagStride * (S.flag_begin + w), __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) >= S.n_buf;
          if (__all(done)) break;
          __builtin_amdgcn_s_sleep(2);
          if (++spins > kSpinLimit) {
            expired = true;
            break;
          }
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kGatherVec; ++i) {
      const int e = tid + i * kThreads;
      if (e < n_vec) {
        const int r = e / vpr;
        *(u32x4*)(buf + (long)(row0 + r) * RB + (long)(e - r * vpr) * 16) = data[i];
      }
    }
    if (with_pos) {
#pragma unroll
      for (int i = 0; i < kPosVec; ++i) {
        const int t = tid + i * kThreads;
        if (t < rows) S.pos[row0 + t] = pv[i];
      }
    }
    if (one_each) break;
    __syncthreads();   // s_src and s_item are rewritten by the next item
  }
  return expired;
}

__global__ __launch_bounds__(64) void k_status_mark(CallStatus st) { status_mark(st); }

// Workgroups 0 .. n_scan_blocks - 1 scan; the last one clears the claim counter and
// the stripe counters of the move that follows on the same stream.
__global__ __launch_bounds__(kThreads) void k_compact_scan(CompactArgs a) {
  status_mark(a.status);
  const int sb = blockIdx.x;
  if (sb == a.n_scan_blocks) {
    for (int i = threadIdx.x; i < a.n_counter_words; i += kThreads) a.claim[i] = 0;
    return;
  }
  int si = 0;
  while (si + 1 < a.n_scan && a.scan[si + 1].block_begin <= sb) ++si;
  keep_scan(a, a.scan[si], sb - a.scan[si].block_begin);
}

__global__ __launch_bounds__(kThreads) void k_compact_gather(CompactArgs a) {
  status_mark(a.status);
  const bool expired = gather_items(a);
  if (threadIdx.x == 0 && expired) status_raise(a.status, kFaultWait);
}

}  // namespace

int compact_max_blocks() {
  static std::atomic<int> cached{-1};   // queried once; calls from several threads may race to fill it
  int v = cached.load(std::memory_order_relaxed);
  if (v < 0) {
    int dev = 0, per_cu = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_compact_gather, kThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    v = per_cu * cus;
    cached.store(v, std::memory_order_relaxed);
  }
  return v;
}

hipError_t launch_status_mark(const CallStatus& st, hipStream_t s) {
  hipLaunchKernelGGL(k_status_mark, dim3(1), dim3(64), 0, s, st);
  return hipGetLastError();
}

static_assert(sizeof(CompactArgs) <= kMaxKernargBytes, "compaction launch record");

hipError_t launch_compact(const CompactArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_compact_scan, dim3(a.n_scan_blocks + 1), dim3(kThreads), 0, s, a);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (a.n_workers <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_compact_gather, dim3(a.n_workers), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace tu
