// KV invalidation (paper Section 4.1, Eq. 2): keep mask, prefix-sum offsets and the
// order-preserving in-place move of the surviving rows, in one cooperative launch.
//
// Scan workgroups (the last n_scan_blocks of the grid, 4096 rows each): 16 rounds of
// 256 consecutive rows, one row per lane, so every load is coalesced. A lane's keep
// flag is "position in no deletion range"; the wavefront ballot + mbcnt gives each
// kept row its rank inside the wave, one wave scans the 64 per-(round, wave) counts,
// and the rows kept before the workgroup's first row (from the verified spans) give
// the destination. They write src_index and flag an error if a destination differs
// from the one the host's live spans imply.
//
// Gather workgroups (all others): move whole rows of every attention layer's K and V
// buffers, and the position array, in place, only from the first removed row on. The
// source of destination row j is j plus the lengths of the removed row spans that
// start at or before it (spans are verified on the host), so moving rows does not
// wait for the scan. Sources never precede destinations, so rows only move toward the
// front. Work is a sequence of (stripe, buffer) items; workgroup b handles items b,
// b + G, b + 2G, ... in order. An item loads its source rows into registers, bumps its
// stripe's read counter, waits until every earlier stripe whose sources can reach its
// destination rows has been read by all buffers, then stores. The launch is
// cooperative, so every workgroup is resident; every wait targets a smaller item
// index, and the workgroup holding the smallest unread item never waits, so the scheme
// always progresses. One lane polls, with back-off, counters that sit on separate
// cache lines. Each wait is also bounded: on expiry an error word is set and the item
// proceeds, so every wave exits.
#include "common.h"

namespace tu {

namespace {

constexpr int kThreads = 256;
constexpr int kScanRounds = 16;
constexpr int kScanWaves = kThreads / 64;
constexpr int kGatherVec = kGatherStripeBytes / (kThreads * 16);   // 16-byte vectors per thread
constexpr long kSpinLimit = 1l << 20;                               // bounded wait per counter

__device__ __forceinline__ int lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Number of removed rows before old row i, from the verified spans.
__device__ __forceinline__ int removed_before(const CompactArgs& a, int span_begin, int n_spans, int i) {
  int full = 0, removed = 0;
  for (int q = 0; q < n_spans; ++q) {
    const int row = a.spans[span_begin + q][0] + full;   // old row of the span start
    if (row >= i) break;
    removed = full + min(a.spans[span_begin + q][1], i - row);
    full += a.spans[span_begin + q][1];
  }
  return removed;
}

// One scan workgroup: kScanRows consecutive old rows of one context.
__device__ void keep_scan(const CompactArgs& a, const ScanSeq& s, int chunk) {
  __shared__ int32_t rng[kMaxRangesPerLaunch][2];
  __shared__ int32_t cnt[kScanRounds * kScanWaves];
  __shared__ int32_t off[kScanRounds * kScanWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < s.n_ranges; i += kThreads) {
    rng[i][0] = a.ranges[s.range_begin + i][0];
    rng[i][1] = a.ranges[s.range_begin + i][1];
  }
  const int base = chunk * kScanRows;
  int32_t p[kScanRounds];
  uint64_t m[kScanRounds];
#pragma unroll
  for (int r = 0; r < kScanRounds; ++r) {
    const int idx = base + r * kThreads + tid;
    p[r] = idx < s.L_old ? s.pos[idx] : 0;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kScanRounds; ++r) {
    const int idx = base + r * kThreads + tid;
    bool keep = idx < s.L_old;
    for (int q = 0; q < s.n_ranges; ++q) keep = keep && !(p[r] >= rng[q][0] && p[r] < rng[q][1]);
    m[r] = __ballot(keep);
    if (lane == 0) cnt[r * kScanWaves + wave] = __popcll(m[r]);
  }
  __syncthreads();
  if (wave == 0) {
    // 64 counts in (round, wave) order = row order; lane owns one
    const int c = cnt[lane];
    int incl = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(incl, d, 64);
      if (lane >= d) incl += y;
    }
    off[lane] = incl - c;
  }
  __syncthreads();
  // rows kept before this chunk, from the verified spans
  const int kept_before = base - removed_before(a, s.span_begin, s.n_spans, base);
  bool bad = false;
#pragma unroll
  for (int r = 0; r < kScanRounds; ++r) {
    const int idx = base + r * kThreads + tid;
    if ((m[r] >> lane) & 1ull) {
      const int dst = kept_before + off[r * kScanWaves + wave] + lane_rank(m[r]);
      s.src_index[dst] = idx;
      // the device positions must agree with the host's live spans
      bad |= dst != idx - removed_before(a, s.span_begin, s.n_spans, idx);
    }
  }
  if (bad) __hip_atomic_store(a.err, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ void gather_items(const CompactArgs& a, int worker, int n_workers) {
  __shared__ int32_t s_src[kGatherStripeBytes / 16];
  const int tid = threadIdx.x;
  const int R = a.rows_per_stripe;
  const int RB = a.row_bytes;
  const int vpr = RB >> 4;  // 16-byte vectors per row
  for (int item = worker; item < a.total_items; item += n_workers) {
    int si = 0;
    while (si + 1 < a.n_seq && a.seq[si + 1].item_begin <= item) ++si;
    const GatherSeq& S = a.seq[si];
    const int local = item - S.item_begin;
    const int stripe = local / S.n_buf;
    const int b = local - stripe * S.n_buf;
    const bool is_pos = S.pos != nullptr && b == S.n_buf - 1;
    char* buf = is_pos ? nullptr : (char*)a.bufs[S.buf_begin + b];
    const int row0 = S.row_begin + stripe * R;
    const int rows = min(R, S.n_keep - row0);
    // source row of each destination row of the stripe
    for (int t = tid; t < rows; t += kThreads) {
      const int j = row0 + t;
      int src = j;
      for (int q = 0; q < S.n_spans; ++q) {
        if (a.spans[S.span_begin + q][0] > j) break;
        src += a.spans[S.span_begin + q][1];
      }
      s_src[t] = src;
    }
    __syncthreads();
    const int n_vec = is_pos ? 0 : rows * vpr;
    u32x4 data[kGatherVec];
#pragma unroll
    for (int i = 0; i < kGatherVec; ++i) {
      const int e = tid + i * kThreads;
      if (e < n_vec) {
        const int r = e / vpr;
        data[i] = *(const u32x4*)(buf + (long)s_src[r] * RB + (long)(e - r * vpr) * 16);
      }
    }
    int32_t pv[(kGatherStripeBytes / 16 + kThreads - 1) / kThreads];
    if (is_pos) {
#pragma unroll
      for (int i = 0; i < (kGatherStripeBytes / 16 + kThreads - 1) / kThreads; ++i) {
        const int t = tid + i * kThreads;
        if (t < rows) pv[i] = S.pos[s_src[t]];
      }
    }
    // every source vector of this item is in registers before its counter moves
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
      __hip_atomic_fetch_add(a.flags + kFlagStride * (S.flag_begin + stripe), 1, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      // one lane walks the window from the nearest stripe down: stripes finish their reads
      // roughly in order, so once the nearest ones are done the rest usually are too
      for (int w = stripe - 1; w >= max(0, stripe - S.window); --w) {
        long spins = 0;
        while (__hip_atomic_load(a.flags + kFlagStride * (S.flag_begin + w), __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT) < S.n_buf) {
          __builtin_amdgcn_s_sleep(4);
          if (++spins > kSpinLimit) {
            __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
    if (is_pos) {
#pragma unroll
      for (int i = 0; i < (kGatherStripeBytes / 16 + kThreads - 1) / kThreads; ++i) {
        const int t = tid + i * kThreads;
        if (t < rows) S.pos[row0 + t] = pv[i];
      }
    }
    __syncthreads();   // s_src is rewritten by the next item
  }
}

__global__ __launch_bounds__(kThreads) void k_compact(CompactArgs a) {
  const int n_workers = gridDim.x - a.n_scan_blocks;
  if ((int)blockIdx.x >= n_workers) {
    const int sb = blockIdx.x - n_workers;
    int si = 0;
    while (si + 1 < a.n_scan && a.scan[si + 1].block_begin <= sb) ++si;
    keep_scan(a, a.scan[si], sb - a.scan[si].block_begin);
    return;
  }
  gather_items(a, blockIdx.x, n_workers);
}

__global__ void k_zero(int32_t* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

}  // namespace

int compact_max_blocks() {
  static int cached = -1;
  if (cached < 0) {
    int dev = 0, per_cu = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_compact, kThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cached = per_cu * cus;
  }
  return cached;
}

hipError_t launch_compact(const CompactArgs& a, int n_workers, hipStream_t s) {
  const int blocks = n_workers + a.n_scan_blocks;
  if (blocks <= 0) return hipSuccess;
  const int nz = a.n_flag_words + 1;   // error word + stripe counters
  hipLaunchKernelGGL(k_zero, dim3((nz + 255) / 256), dim3(256), 0, s, a.err, nz);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  void* args[] = {(void*)&a};
  return hipLaunchCooperativeKernel((const void*)k_compact, dim3(blocks), dim3(kThreads), args, 0, s);
}

}  // namespace tu
