// KV invalidation (paper Section 4.1, Eq. 2): keep mask, prefix-sum offsets and the
// order-preserving in-place gather of the surviving K/V rows.
//
// k_keep_scan: one workgroup of 1024 threads per context. Each pass covers 16K
// cache rows as 16 rounds of 1024 consecutive rows (one row per lane), so every
// load is coalesced. A lane's keep flag is "position in no deletion range"; the
// wavefront ballot + mbcnt gives each kept row its rank inside the wave, the
// 256 per-(round, wave) counts are scanned by one wave, and the sum gives the
// destination. The kernel writes src_index and compacts d_pos in place (a pass
// only writes rows it has already read).
//
// k_gather: moves whole rows of every attention layer's K and V buffers, in
// place, only from the first removed row on. src_index[j] >= j, so a row is only
// ever copied toward the front. Work is a stream of (stripe, buffer) items
// handed out in increasing order by an atomic ticket; an item loads its
// stripe's source rows into registers, bumps that stripe's read counter, waits
// until every earlier stripe whose sources can overlap its destination rows has
// been read by all buffers, then stores. Waits only target items that took
// their ticket earlier, so they are resident and never wait on later items: the
// scheme cannot deadlock. Each wait is additionally bounded; on expiry the
// kernel records an error word and continues, so every wave always exits.
#include "common.h"

namespace tu {

namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanRounds = 16;
constexpr int kScanWaves = kScanThreads / 64;

__device__ __forceinline__ int lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__global__ __launch_bounds__(kScanThreads) void k_keep_scan(ScanArgs a) {
  // clear the gather's tickets and stripe counters (ordered before the gather by the stream)
  for (int i = blockIdx.x * kScanThreads + threadIdx.x; i < a.zero_count; i += gridDim.x * kScanThreads)
    a.zero_ptr[i] = 0;
  if ((int)blockIdx.x >= a.n_seq) return;
  const ScanSeq s = a.seq[blockIdx.x];

  __shared__ int32_t rng[kMaxRangesPerLaunch][2];
  __shared__ int32_t cnt[kScanRounds * kScanWaves];
  __shared__ int32_t off[kScanRounds * kScanWaves];
  __shared__ int32_t total;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  for (int i = tid; i < s.n_ranges; i += kScanThreads) {
    rng[i][0] = a.ranges[s.range_begin + i][0];
    rng[i][1] = a.ranges[s.range_begin + i][1];
  }
  __syncthreads();

  int running = 0;
  for (int base = 0; base < s.L_old; base += kScanRounds * kScanThreads) {
    int32_t p[kScanRounds];
    uint64_t m[kScanRounds];
#pragma unroll
    for (int r = 0; r < kScanRounds; ++r) {
      const int idx = base + r * kScanThreads + tid;
      p[r] = idx < s.L_old ? s.pos[idx] : 0;
    }
#pragma unroll
    for (int r = 0; r < kScanRounds; ++r) {
      const int idx = base + r * kScanThreads + tid;
      bool keep = idx < s.L_old;
      for (int q = 0; q < s.n_ranges; ++q)
        keep = keep && !(p[r] >= rng[q][0] && p[r] < rng[q][1]);
      m[r] = __ballot(keep);
      if (lane == 0) cnt[r * kScanWaves + wave] = __popcll(m[r]);
    }
    __syncthreads();
    if (wave == 0) {
      // 256 counts in (round, wave) order = row order; lane owns 4 consecutive entries
      const int c0 = cnt[4 * lane], c1 = cnt[4 * lane + 1], c2 = cnt[4 * lane + 2], c3 = cnt[4 * lane + 3];
      int incl = c0 + c1 + c2 + c3;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(incl, d, 64);
        if (lane >= d) incl += y;
      }
      const int excl = incl - (c0 + c1 + c2 + c3);
      off[4 * lane] = excl;
      off[4 * lane + 1] = excl + c0;
      off[4 * lane + 2] = excl + c0 + c1;
      off[4 * lane + 3] = excl + c0 + c1 + c2;
      if (lane == 63) total = incl;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kScanRounds; ++r) {
      const int idx = base + r * kScanThreads + tid;
      if ((m[r] >> lane) & 1ull) {
        const int dst = running + off[r * kScanWaves + wave] + lane_rank(m[r]);
        s.src_index[dst] = idx;
        s.pos[dst] = p[r];
      }
    }
    running += total;
    __syncthreads();
  }
}

constexpr int kGatherThreads = 256;
constexpr int kGatherVec = 8;          // 16-byte vectors per thread per stripe
constexpr long kSpinLimit = 1l << 22;  // bounded wait per stripe counter

__global__ __launch_bounds__(kGatherThreads) void k_gather(GatherArgs a) {
  __shared__ int32_t s_item;
  if (threadIdx.x == 0) s_item = atomicAdd(a.ticket, 1);
  __syncthreads();
  const int item = s_item;
  if (item >= a.total_items) return;
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].item_begin <= item) ++si;
  const GatherSeq S = a.seq[si];
  const int local = item - S.item_begin;
  const int stripe = local / S.n_buf;
  const int b = local - stripe * S.n_buf;
  char* buf = (char*)a.bufs[S.buf_begin + b];
  const int R = a.rows_per_stripe;
  const int RB = a.row_bytes;
  const int vpr = RB >> 4;  // 16-byte vectors per row
  const int row0 = S.row_begin + stripe * R;
  const int rows = min(R, S.n_keep - row0);
  const int n_vec = rows * vpr;

  u32x4 data[kGatherVec];
  long dst_off[kGatherVec];
#pragma unroll
  for (int i = 0; i < kGatherVec; ++i) {
    const int e = threadIdx.x + i * kGatherThreads;
    dst_off[i] = -1;
    if (e < n_vec) {
      const int r = e / vpr;
      const int c = e - r * vpr;
      const long src = S.src_index[row0 + r];
      data[i] = *(const u32x4*)(buf + src * RB + (long)c * 16);
      dst_off[i] = (long)(row0 + r) * RB + (long)c * 16;
    }
  }
  // every source vector of this stripe is in registers before the counter moves
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(a.flags + S.flag_begin + stripe, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (threadIdx.x < 64) {
    const int lo = max(0, stripe - S.window);
    for (int w = lo + (int)threadIdx.x; w < stripe; w += 64) {
      long spins = 0;
      while (__hip_atomic_load(a.flags + S.flag_begin + w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
             S.n_buf) {
        __builtin_amdgcn_s_sleep(2);
        if (++spins > kSpinLimit) {
          __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kGatherVec; ++i)
    if (dst_off[i] >= 0) *(u32x4*)(buf + dst_off[i]) = data[i];
}

}  // namespace

hipError_t launch_keep_scan(const ScanArgs& a, hipStream_t s) {
  int blocks = a.n_seq > 0 ? a.n_seq : 1;
  hipLaunchKernelGGL(k_keep_scan, dim3(blocks), dim3(kScanThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& a, int n_blocks, hipStream_t s) {
  if (n_blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather, dim3(n_blocks), dim3(kGatherThreads), 0, s, a);
  return hipGetLastError();
}

static_assert(kGatherStripeBytes == kGatherThreads * kGatherVec * 16, "stripe size");

}  // namespace tu
