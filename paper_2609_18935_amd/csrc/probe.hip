// Attention diagnostics (paper Section 5.3, Appendix C): the float32 reference
// softmax of the last n query tokens of a context over the rows they see, averaged
// over tokens and heads into one token distribution, the memory-group masses of that
// distribution with the effective group count and boundary-window share, and the
// total variation distance between two distributions of the same tokens.
//
// Probe query i of n is the token in cache row len - n + i; it sees rows
// 0 .. len - n + i. The raw queries are rotated at the rows' positions (float64
// angles, bf16 nearest even, as the cached keys were). Scores S = scale * q.k are
// products of bf16 values summed in fp32 on v_mfma_f32_32x32x16_bf16. The key cache is
// read twice and no score is stored: a first pass keeps each 32-key block's max and sum
// of exponentials per row, a small kernel combines them into each row's max and sum,
// and a second pass recomputes the scores, normalises them and sums them over the rows
// of each key. Every sum is taken in a fixed order (deterministic). HBM-bound.
#include <atomic>

#include "common.h"

namespace tu {

namespace {

typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;

constexpr int kThreads = 256;

__device__ __forceinline__ float block_reduce_max(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float r = sh[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) r = fmaxf(r, sh[i]);
  __syncthreads();
  return r;
}

__device__ __forceinline__ double block_reduce_sum(double v, double* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double r = 0.0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) r += sh[i];
  __syncthreads();
  return r;
}

// One workgroup per (probe token, query head): each thread rotates its own dimension
// (and computes that dimension's angle), so a workgroup waits on one load.
__global__ __launch_bounds__(kThreads) void k_probe_rope(ProbeArgs a) {
  const int i = blockIdx.x, h = blockIdx.y;
  const int D = a.head_dim, Hq = a.n_q_heads, r = a.rotary_dim, half = r >> 1;
  const bf16_t* x = a.q + ((long)i * Hq + h) * D;
  bf16_t* o = a.q_hat + ((long)i * Hq + h) * D;
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    if (d >= r) {
      o[d] = x[d];
      continue;
    }
    const int j = d < half ? d : d - half;
    const double av = (double)bf16_to_f32(x[j]), bv = (double)bf16_to_f32(x[j + half]);
    const int64_t p = a.pos[a.len - a.n_probe + i];
    const double w = pow(a.theta, -2.0 * (double)j / (double)r);
    double sn, cs;
    sincos((double)p * w, &sn, &cs);
    o[d] = (bf16_t)f64_to_bf16_rne(d < half ? av * cs - bv * sn : bv * cs + av * sn);
  }
}

// Both score passes stream (KV head, 64-key tile) items: a launch holds as many
// workgroups as fit on the chip at once (a multiple of the KV head count), and workgroup
// b takes items b, b + grid, ... , all of KV head b % Hkv, prefetching the next item's
// key tile into registers while it computes on the current one in LDS. Rows are (token
// i, head g of the group) as r = i * G + g, at most kProbeMaxRows, in R32 row tiles of
// 32; the keys of a tile are two half tiles of 32. Wave w keeps the query fragments of
// row tile w % R32 for the whole launch and takes the half tiles w / R32,
// w / R32 + 4 / R32, ... (R32 <= 4, so every (row tile, half tile) pair has one wave).
template <int D>
struct KeyTile {
  static constexpr int RC = D / 8 + 1;      // 16-byte chunks per LDS row (one of padding)
  static constexpr int PER = kProbeKeys * (D / 8) / kThreads;
  static_assert(PER * kThreads == kProbeKeys * (D / 8), "whole chunks per thread");
  u32x4 v[PER];
  // rows past len repeat row len - 1 (their scores are masked), so no load is conditional
  __device__ __forceinline__ void fetch(const ProbeArgs& a, int j0, int hkv) {
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int c = threadIdx.x + t * kThreads;
      const int j = min(j0 + c / (D / 8), a.len - 1);
      v[t] = *(const u32x4*)(a.k_cache + ((long)j * a.n_kv_heads + hkv) * D + (c % (D / 8)) * 8);
    }
  }
  __device__ __forceinline__ void put(bf16_t* s_k) const {
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int c = threadIdx.x + t * kThreads;
      *(u32x4*)(s_k + ((c / (D / 8)) * RC + c % (D / 8)) * 8) = v[t];
    }
  }
};

// One MFMA operand of row tile rt: this lane's query row rt * 32 + col, dims
// 16 s + 8 hl .. + 7 for s < D / 16 (rows past R repeat row 0; their results are
// masked).
template <int D>
__device__ __forceinline__ void load_q(const ProbeArgs& a, bf16x8* qf, int rt, int hkv, int R, int G) {
  const int lane = threadIdx.x & 63, hl = lane >> 5, col = lane & 31;
  const int rq = rt * 32 + col < R ? rt * 32 + col : 0;
  const bf16_t* qrow = a.q_hat + ((long)(rq / G) * a.n_q_heads + hkv * G + rq % G) * D + 8 * hl;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) qf[s] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qrow + 16 * s));
}

// The (row tile, half tiles) share of one wave.
struct WaveShare {
  int rt, first, step;
  bool active;
  __device__ __forceinline__ WaveShare(int R32) {
    const int wave = threadIdx.x >> 6;
    rt = wave % R32;
    first = wave / R32;
    step = (kThreads / 64) / R32;
    active = first < step;
  }
  __device__ __forceinline__ bool takes(int kt) const { return active && kt >= first && (kt - first) % step == 0; }
};

// Pass 1: each 32-key block's max and sum of exponentials of every row's masked scores,
// stored as part[(h * n + i) * n_parts + block] = {max, sum}. Keys are the A operand, so
// a lane holds 16 keys of one row and the pair of lanes l, l ^ 32 the whole block.
template <int D>
__global__ __launch_bounds__(kThreads) void k_probe_part(ProbeArgs a) {
  constexpr int RC = KeyTile<D>::RC;
  __shared__ __attribute__((aligned(16))) bf16_t s_k[kProbeKeys * RC * 8];
  const int Hkv = a.n_kv_heads, G = a.n_q_heads / Hkv, n = a.n_probe;
  const int R = n * G;
  const int R32 = (R + 31) / 32;
  const int n_items = (a.len + kProbeKeys - 1) / kProbeKeys * Hkv;
  const int hkv = blockIdx.x % Hkv;
  const int lane = threadIdx.x & 63, hl = lane >> 5, col = lane & 31;
  const WaveShare ws(R32);
  KeyTile<D> kt_regs;
  kt_regs.fetch(a, (int)blockIdx.x / Hkv * kProbeKeys, hkv);
  bf16x8 qf[D / 16];
  if (ws.active) load_q<D>(a, qf, ws.rt, hkv, R, G);
  // this lane's row and the last key its probe token sees
  const int r = ws.rt * 32 + col;
  const int i = r / G, g = r - i * G;
  const int limit = r < R ? a.len - n + i : -1;
  float* prow = a.part + ((long)(hkv * G + g) * n + i) * a.n_parts * 2;
  for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int j0 = it / Hkv * kProbeKeys;
    __syncthreads();
    kt_regs.put(s_k);
    __syncthreads();
    if (it + (int)gridDim.x < n_items) kt_regs.fetch(a, (it + (int)gridDim.x) / Hkv * kProbeKeys, hkv);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      if (!ws.takes(kt)) continue;
      f32x16 acc;
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e] = 0.f;
      const bf16_t* ka = s_k + ((kt * 32 + col) * RC + hl) * 8;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        const bf16x8 kv = __builtin_bit_cast(bf16x8, *(const u32x4*)(ka + 16 * s));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv, qf[s], acc, 0, 0, 0);
      }
      // lane holds keys j0 + kt*32 + 4 hl + o, o = 8 (e/4) + e%4, of query row r
      const int o_max = limit - (j0 + kt * 32 + 4 * hl);
      float v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = 8 * (e >> 2) + (e & 3) <= o_max ? acc[e] * a.scale : -__builtin_inff();
      float m = -__builtin_inff();
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, v[e]);
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      const float ms = m == -__builtin_inff() ? 0.f : m;
      float l = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) l += expf(v[e] - ms);
      l += __shfl_xor(l, 32, 64);
      if (r < R && hl == 0) *(f32x2*)(prow + (2 * (j0 / kProbeKeys) + kt) * 2) = f32x2{m, l};
    }
  }
}

// One workgroup per score row: its max and the inverse of its sum of exponentials, from
// the pass-1 pairs, in a fixed order. A thread takes pairs tid, tid + 256, ... in batches
// of kStatsBatch loads issued together; a row of up to kThreads * kStatsBatch pairs
// (65,536 keys) is read once and kept in registers.
constexpr int kStatsBatch = 8;
__global__ __launch_bounds__(kThreads) void k_probe_stats(ProbeArgs a) {
  __shared__ float shf[kThreads / 64];
  __shared__ double shd[kThreads / 64];
  const f32x2* pr = reinterpret_cast<const f32x2*>(a.part) + (long)blockIdx.x * a.n_parts;
  const int np = a.n_parts;
  constexpr int B = kThreads * kStatsBatch;
  f32x2 x[kStatsBatch];
  auto batch = [&](int t0) {
#pragma unroll
    for (int b = 0; b < kStatsBatch; ++b) {
      const int t = t0 + b * kThreads + (int)threadIdx.x;
      x[b] = t < np ? pr[t] : f32x2{-__builtin_inff(), 0.f};
    }
  };
  float m = -__builtin_inff();
  for (int t0 = 0; t0 < np; t0 += B) {
    batch(t0);
#pragma unroll
    for (int b = 0; b < kStatsBatch; ++b) m = fmaxf(m, x[b][0]);
  }
  m = block_reduce_max(m, shf);
  double l = 0.0;
  for (int t0 = (np - 1) / B * B; t0 >= 0; t0 -= B) {   // the last batch is still loaded
    if (t0 + B < np) batch(t0);
#pragma unroll
    for (int b = 0; b < kStatsBatch; ++b)
      if (x[b][0] != -__builtin_inff()) l += (double)(x[b][1] * expf(x[b][0] - m));
  }
  const double L = block_reduce_sum(l, shd);
  if (threadIdx.x == 0) {
    a.stats[2 * blockIdx.x] = m;
    a.stats[2 * blockIdx.x + 1] = (float)(1.0 / L);
  }
}

// Pass 2: the scores again, now with the queries as the A operand, so a lane holds one
// key and 16 rows; each visible score becomes exp(s - max) / sum with its row's
// statistics and is added over the rows in a fixed order (a lane's rows, the two lane
// halves, then the waves in wave order), giving key_sum[hkv * ld + key]. Streams items
// as pass 1 does.
template <int D>
__global__ __launch_bounds__(kThreads) void k_probe_keysum(ProbeArgs a) {
  constexpr int RC = KeyTile<D>::RC;
  __shared__ __attribute__((aligned(16))) bf16_t s_k[kProbeKeys * RC * 8];
  __shared__ float s_st[2 * kProbeMaxRows];
  __shared__ float s_sum[kThreads / 64][2][32];
  const int Hkv = a.n_kv_heads, G = a.n_q_heads / Hkv, n = a.n_probe;
  const int R = n * G;
  const int R32 = (R + 31) / 32;
  const int n_items = (a.len + kProbeKeys - 1) / kProbeKeys * Hkv;
  const int hkv = blockIdx.x % Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hl = lane >> 5, col = lane & 31;
  const WaveShare ws(R32);
  KeyTile<D> kt_regs;
  kt_regs.fetch(a, (int)blockIdx.x / Hkv * kProbeKeys, hkv);
  bf16x8 qf[D / 16];
  if (ws.active) load_q<D>(a, qf, ws.rt, hkv, R, G);
  for (int r = threadIdx.x; r < R; r += kThreads) {
    const int i = r / G, g = r - i * G;
    const f32x2 st = *(const f32x2*)(a.stats + 2 * ((long)(hkv * G + g) * n + i));
    s_st[2 * r] = st[0];
    s_st[2 * r + 1] = st[1];
  }
  for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int j0 = it / Hkv * kProbeKeys;
    __syncthreads();
    kt_regs.put(s_k);
    __syncthreads();
    if (it + (int)gridDim.x < n_items) kt_regs.fetch(a, (it + (int)gridDim.x) / Hkv * kProbeKeys, hkv);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      float t = 0.f;
      if (ws.takes(kt)) {
        f32x16 acc;
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = 0.f;
        const bf16_t* ka = s_k + ((kt * 32 + col) * RC + hl) * 8;
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
          const bf16x8 kv = __builtin_bit_cast(bf16x8, *(const u32x4*)(ka + 16 * s));
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[s], kv, acc, 0, 0, 0);
        }
        // lane holds rows r0 + o, o = 8 (e/4) + e%4, of key j0 + kt*32 + col; row r (token
        // r / G) sees the key when r / G >= key - (len - n), that is r >= r_min; rows past
        // R (statistics never written) and unseen rows are selected away
        const int r0 = ws.rt * 32 + 4 * hl;
        const int lo = max(0, j0 + kt * 32 + col - (a.len - n)) * G - r0, hi = R - r0;
        const float* st = s_st + 2 * r0;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int o = 8 * (e >> 2) + (e & 3);
          const f32x2 mv = *(const f32x2*)(st + 2 * o);
          const float pe = expf(acc[e] * a.scale - mv[0]) * mv[1];
          t += o >= lo && o < hi ? pe : 0.f;
        }
      }
      t += __shfl_xor(t, 32, 64);
      if (hl == 0) s_sum[wave][kt][col] = t;
    }
    __syncthreads();
    if (threadIdx.x < kProbeKeys) {
      const int k2 = threadIdx.x >> 5, c = threadIdx.x & 31;
      float u = s_sum[0][k2][c];
      for (int w = 1; w < kThreads / 64; ++w) u += s_sum[w][k2][c];
      a.key_sum[(long)hkv * a.ld + j0 + threadIdx.x] = u;
    }
  }
}

// probs[j] += weight * (sum over the KV heads, in order, of key_sum) / rows.
__global__ __launch_bounds__(kThreads) void k_probe_mean(ProbeArgs a) {
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= a.len) return;
  float t = 0.f;
  for (int h = 0; h < a.n_kv_heads; ++h) t += a.key_sum[(long)h * a.ld + j];
  a.probs[j] += a.weight * (t / (float)(a.n_q_heads * a.n_probe));
}

// Group masses, in a fixed summation order (the same bits on every run): workgroup b
// takes rows [b * block_rows, ...) in rounds of 256, its position and probability loads
// issued together, kGroupBatch rounds at a time; a row adds its probability to the group
// holding its position (binary search over this launch's sorted group ranges, staged in
// LDS) and to the group's boundary window. Within a wave the rows of one group are summed
// by a butterfly; each wave accumulates its rounds in order into its own LDS copy of the
// launch's groups; the four copies are added in wave order and written as the
// workgroup's partial sums of every group of the launch (zeros included), so no
// accumulator needs clearing. k_group_final adds the partials in workgroup order.
constexpr int kGroupBatch = 4;
__global__ __launch_bounds__(kThreads) void k_group_mass(GroupArgs a) {
  __shared__ double acc[kThreads / 64][2][kMaxGroupsPerLaunch];
  __shared__ int32_t rng[kMaxGroupsPerLaunch][2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < (kThreads / 64) * 2 * kMaxGroupsPerLaunch; i += kThreads) (&acc[0][0][0])[i] = 0.0;
  for (int i = tid; i < a.n; i += kThreads) {
    rng[i][0] = a.range[i][0];
    rng[i][1] = a.range[i][1];
  }
  __syncthreads();
  const int base = blockIdx.x * a.block_rows;
  for (int r0 = 0; r0 < a.block_rows; r0 += kThreads * kGroupBatch) {
    int pb[kGroupBatch];
    float vb[kGroupBatch];
#pragma unroll
    for (int u = 0; u < kGroupBatch; ++u) {
      const int j = min(base + r0 + u * kThreads + tid, a.len - 1);   // rows past len: masked below
      pb[u] = a.pos[j];
      vb[u] = a.probs[j];
    }
#pragma unroll
    for (int u = 0; u < kGroupBatch; ++u) {
      const int j = base + r0 + u * kThreads + tid;
      int g = -1;
      double v = 0.0, w = 0.0;
      if (r0 + u * kThreads < a.block_rows && j < a.len) {
        const int p = pb[u];
        int lo = 0, hi = a.n - 1;
        while (lo <= hi) {
          const int mid = (lo + hi) >> 1;
          if (rng[mid][1] <= p) lo = mid + 1;
          else if (rng[mid][0] > p) hi = mid - 1;
          else { g = mid; break; }
        }
        if (g >= 0) {
          v = (double)vb[u];
          w = p < rng[g][0] + a.window ? v : 0.0;
        }
      }
      uint64_t left = __ballot(g >= 0);
      while (left) {
        const int leader = __builtin_ctzll(left);
        const int g0 = __shfl(g, leader, 64);
        const bool mine = g == g0;
        double s = mine ? v : 0.0, sw = mine ? w : 0.0;
        for (int o = 32; o > 0; o >>= 1) {
          s += __shfl_xor(s, o, 64);
          sw += __shfl_xor(sw, o, 64);
        }
        if (lane == leader) {
          acc[wave][0][g0] += s;
          acc[wave][1][g0] += sw;
        }
        left &= ~__ballot(mine);
      }
    }
  }
  __syncthreads();
  for (int g = tid; g < a.n; g += kThreads) {
    double m = 0.0, mw = 0.0;
#pragma unroll
    for (int x = 0; x < kThreads / 64; ++x) {
      m += acc[x][0][g];
      mw += acc[x][1][g];
    }
    double* out = a.partial + (size_t)blockIdx.x * 2 * a.n_total;
    out[a.g_begin + g] = m;
    out[a.n_total + a.g_begin + g] = mw;
  }
}

// One workgroup: memory mass M, effective group count exp(-sum a log a) over a = mass / M,
// boundary-window share; the per-group masses as fp32. Sums in a fixed order.
__global__ __launch_bounds__(kThreads) void k_group_final(GroupArgs a) {
  __shared__ double shd[kThreads / 64];
  const int n = a.n_total;
  // group g's mass and window mass together: the workgroups' partials in workgroup order,
  // eight workgroups' pairs at a time (independent loads)
  auto group_sums = [&](int g, double& m, double& w) {
    const double* pg = a.partial + g;
    m = 0.0;
    w = 0.0;
    for (int b0 = 0; b0 < a.n_blocks; b0 += 8) {
      double x[8], y[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool in = b0 + u < a.n_blocks;
        x[u] = in ? pg[(size_t)(b0 + u) * 2 * n] : 0.0;
        y[u] = in ? pg[(size_t)(b0 + u) * 2 * n + n] : 0.0;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        m += x[u];
        w += y[u];
      }
    }
  };
  // a thread's first kKeep groups keep their masses in registers for the entropy sum
  constexpr int kKeep = 4;
  double keep[kKeep];
  double m = 0.0, w = 0.0;
#pragma unroll
  for (int i = 0; i < kKeep; ++i) {
    const int g = threadIdx.x + i * kThreads;
    keep[i] = 0.0;
    if (g < n) {
      double mg, wg;
      group_sums(g, mg, wg);
      keep[i] = mg;
      m += mg;
      w += wg;
      a.mass[g] = (float)mg;
      if (a.window_mass) a.window_mass[g] = (float)wg;
    }
  }
  for (int g = threadIdx.x + kKeep * kThreads; g < n; g += kThreads) {
    double mg, wg;
    group_sums(g, mg, wg);
    m += mg;
    w += wg;
    a.mass[g] = (float)mg;
    if (a.window_mass) a.window_mass[g] = (float)wg;
  }
  const double M = block_reduce_sum(m, shd);
  const double W = block_reduce_sum(w, shd);
  double h = 0.0;
  auto add_entropy = [&](double mg) {
    const double x = M > 0.0 ? mg / M : 0.0;
    if (x > 0.0) h -= x * log(x);
  };
#pragma unroll
  for (int i = 0; i < kKeep; ++i)
    if (threadIdx.x + i * kThreads < n) add_entropy(keep[i]);
  for (int g = threadIdx.x + kKeep * kThreads; g < n; g += kThreads) {
    double mg, wg;
    group_sums(g, mg, wg);
    add_entropy(mg);
  }
  const double H = block_reduce_sum(h, shd);
  if (threadIdx.x == 0 && a.summary) {
    a.summary[0] = (float)M;
    a.summary[1] = M > 0.0 ? (float)exp(H) : 0.f;
    a.summary[2] = M > 0.0 ? (float)(W / M) : 0.f;
  }
}

// Total variation: per-workgroup partial sums of |p_j - q_map(j)| (float64, fixed
// order), then one workgroup adds the partials in order.
__global__ __launch_bounds__(kThreads) void k_tv_partial(TvArgs a) {
  __shared__ double shd[kThreads / 64];
  constexpr int PER = kTvRowsPerBlock / kThreads, B = 8;   // rows of a thread, loaded B at a time
  static_assert(PER % B == 0, "whole batches");
  double s = 0.0;
  const long base = (long)blockIdx.x * kTvRowsPerBlock;
  for (int b0 = 0; b0 < PER; b0 += B) {
    float pv[B], qv[B];
    long kv[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const long j = base + (long)(b0 + u) * kThreads + threadIdx.x;
      const long jj = j < a.n ? j : 0;   // rows past n read row 0 and are not added
      pv[u] = a.p[jj];
      kv[u] = a.map ? (long)a.map[jj] : jj;
    }
#pragma unroll
    for (int u = 0; u < B; ++u) qv[u] = a.q[kv[u]];
#pragma unroll
    for (int u = 0; u < B; ++u)
      if (base + (long)(b0 + u) * kThreads + threadIdx.x < a.n) s += fabs((double)pv[u] - (double)qv[u]);
  }
  s = block_reduce_sum(s, shd);
  if (threadIdx.x == 0) a.partial[blockIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void k_tv_final(TvArgs a) {
  __shared__ double shd[kThreads / 64];
  double s = 0.0;
  for (int b = threadIdx.x; b < a.n_blocks; b += kThreads) s += a.partial[b];
  s = block_reduce_sum(s, shd);
  if (threadIdx.x == 0) a.tv[0] = (float)(0.5 * s);
}

// A streaming pass: as many workgroups as fit on the chip at once (the kernel's own
// occupancy, queried once per kernel; two per CU if the query fails), at most the item
// count, rounded down to a multiple of the KV head count (item counts are multiples of
// it). Any such grid is correct: a workgroup walks the items b, b + grid, ...
template <void (*kernel)(ProbeArgs)>
hipError_t launch_stream_pass(int n_items, const ProbeArgs& a, hipStream_t s) {
  static std::atomic<int> cached{-1};
  int slots = cached.load(std::memory_order_relaxed);
  if (slots < 0) {
    int dev = 0, per_cu = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && per_cu > 0 && cus > 0) {
      slots = per_cu * cus;
      cached.store(slots, std::memory_order_relaxed);
    } else {
      slots = 2 * kCus;
    }
  }
  const int grid = std::max(a.n_kv_heads, std::min(n_items, slots) / a.n_kv_heads * a.n_kv_heads);
  hipLaunchKernelGGL(kernel, dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_probe(const ProbeArgs& a, hipStream_t s) {
  if (a.n_probe <= 0 || a.len <= 0) return hipSuccess;
  if (a.rotary_dim > a.head_dim || a.n_probe * (a.n_q_heads / a.n_kv_heads) > kProbeMaxRows)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_probe_rope, dim3(a.n_probe, a.n_q_heads), dim3(kThreads), 0, s, a);
  const int rows = a.n_q_heads * a.n_probe;
  const int n_items = (a.len + kProbeKeys - 1) / kProbeKeys * a.n_kv_heads;
  if (a.head_dim == 256) {
    if (hipError_t e = launch_stream_pass<k_probe_part<256>>(n_items, a, s); e != hipSuccess) return e;
    hipLaunchKernelGGL(k_probe_stats, dim3(rows), dim3(kThreads), 0, s, a);
    if (hipError_t e = launch_stream_pass<k_probe_keysum<256>>(n_items, a, s); e != hipSuccess) return e;
  } else if (a.head_dim == 128) {
    if (hipError_t e = launch_stream_pass<k_probe_part<128>>(n_items, a, s); e != hipSuccess) return e;
    hipLaunchKernelGGL(k_probe_stats, dim3(rows), dim3(kThreads), 0, s, a);
    if (hipError_t e = launch_stream_pass<k_probe_keysum<128>>(n_items, a, s); e != hipSuccess) return e;
  } else if (a.head_dim == 64) {
    if (hipError_t e = launch_stream_pass<k_probe_part<64>>(n_items, a, s); e != hipSuccess) return e;
    hipLaunchKernelGGL(k_probe_stats, dim3(rows), dim3(kThreads), 0, s, a);
    if (hipError_t e = launch_stream_pass<k_probe_keysum<64>>(n_items, a, s); e != hipSuccess) return e;
  } else {
    return hipErrorInvalidValue;
  }
  hipLaunchKernelGGL(k_probe_mean, dim3((a.len + kThreads - 1) / kThreads), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

static_assert(sizeof(GroupArgs) <= kMaxKernargBytes, "group-mass launch record");
static_assert(sizeof(ProbeArgs) <= kMaxKernargBytes && sizeof(TvArgs) <= kMaxKernargBytes, "probe launch records");

hipError_t launch_group_mass(const GroupArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_group_mass, dim3(a.n_blocks), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_group_final(const GroupArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_group_final, dim3(1), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_tv(const TvArgs& a, hipStream_t s) {
  if (a.n_blocks > 0) hipLaunchKernelGGL(k_tv_partial, dim3(a.n_blocks), dim3(kThreads), 0, s, a);
  hipLaunchKernelGGL(k_tv_final, dim3(1), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace tu
