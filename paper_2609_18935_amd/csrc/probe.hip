// Attention diagnostics (paper Section 5.3, Appendix C): the float32 reference
// softmax of the last n query tokens of a context over the rows they see, averaged
// over tokens and heads into one token distribution, the memory-group masses of that
// distribution with the effective group count and boundary-window share, and the
// total variation distance between two distributions of the same tokens.
//
// Probe query i of n is the token in cache row len - n + i; it sees rows
// 0 .. len - n + i. The raw queries are rotated at the rows' positions (float64
// angles, bf16 nearest even, as the cached keys were). Scores S = scale * q.k are
// products of bf16 values summed in fp32 on v_mfma_f32_32x32x16_bf16 (one workgroup
// per (KV head, 64-key tile), the G query heads of the KV head times the n tokens as
// rows, both operands staged in LDS), written masked to the workspace; a second
// kernel forms each row's max and sum of exponentials, a third averages the
// normalised exponentials per key in a fixed order (deterministic). All of it is
// HBM-bound: the key cache is read once.
#include "common.h"

namespace tu {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxHalfP = 128;

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

// One workgroup per probe token: rotate its query heads at the row's position.
__global__ __launch_bounds__(kThreads) void k_probe_rope(ProbeArgs a) {
  __shared__ double s_cos[kMaxHalfP];
  __shared__ double s_sin[kMaxHalfP];
  const int i = blockIdx.x;
  const int D = a.head_dim, Hq = a.n_q_heads, r = a.rotary_dim, half = r >> 1;
  const int64_t p = a.pos[a.len - a.n_probe + i];
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    const double w = pow(a.theta, -2.0 * (double)j / (double)r);
    double sn, cs;
    sincos((double)p * w, &sn, &cs);
    s_cos[j] = cs;
    s_sin[j] = sn;
  }
  __syncthreads();
  const bf16_t* q = a.q + (long)i * Hq * D;
  bf16_t* o = a.q_hat + (long)i * Hq * D;
  for (int e = threadIdx.x; e < Hq * D; e += blockDim.x) {
    const int h = e / D, d = e - h * D;
    const bf16_t* x = q + (long)h * D;
    if (d < half) {
      const double av = (double)bf16_to_f32(x[d]), bv = (double)bf16_to_f32(x[d + half]);
      o[e] = (bf16_t)f64_to_bf16_rne(av * s_cos[d] - bv * s_sin[d]);
    } else if (d < r) {
      const int j = d - half;
      const double av = (double)bf16_to_f32(x[j]), bv = (double)bf16_to_f32(x[d]);
      o[e] = (bf16_t)f64_to_bf16_rne(bv * s_cos[j] + av * s_sin[j]);
    } else {
      o[e] = x[d];
    }
  }
}

// Scores of one (KV head, 64-key tile): rows are (token i, head g of the group) as
// r = i * G + g, at most kProbeMaxRows; stored as S[(h * n + i) * ld + key].
template <int D>
__global__ __launch_bounds__(kThreads) void k_probe_scores(ProbeArgs a) {
  constexpr int RC = D / 8 + 1;             // 16-byte chunks per LDS row (one of padding)
  constexpr int NS = D / 16;
  __shared__ __attribute__((aligned(16))) bf16_t s_q[kProbeMaxRows * RC * 8];
  __shared__ __attribute__((aligned(16))) bf16_t s_k[kProbeKeys * RC * 8];
  const int hkv = blockIdx.y;
  const int j0 = blockIdx.x * kProbeKeys;
  const int Hq = a.n_q_heads, Hkv = a.n_kv_heads, G = Hq / Hkv, n = a.n_probe;
  const int R = n * G;
  const int R32 = (R + 31) / 32;
  const int tid = threadIdx.x;
  for (int c = tid; c < R32 * 32 * (D / 8); c += kThreads) {
    const int r = c / (D / 8), ch = c - r * (D / 8);
    u32x4 v = {0, 0, 0, 0};
    if (r < R) {
      const int i = r / G, g = r - i * G;
      v = *(const u32x4*)(a.q_hat + ((long)i * Hq + hkv * G + g) * D + ch * 8);
    }
    *(u32x4*)(s_q + (r * RC + ch) * 8) = v;
  }
  for (int c = tid; c < kProbeKeys * (D / 8); c += kThreads) {
    const int r = c / (D / 8), ch = c - r * (D / 8);
    const int j = j0 + r;
    u32x4 v = {0, 0, 0, 0};
    if (j < a.len) v = *(const u32x4*)(a.k_cache + ((long)j * Hkv + hkv) * D + ch * 8);
    *(u32x4*)(s_k + (r * RC + ch) * 8) = v;
  }
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6, hl = lane >> 5, col = lane & 31;
  for (int w = wave; w < 2 * R32; w += kThreads / 64) {
    const int kt = w & 1, rt = w >> 1;
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;
    const bf16_t* ka = s_k + ((kt * 32 + col) * RC + hl) * 8;
    const bf16_t* qb = s_q + ((rt * 32 + col) * RC + hl) * 8;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, *(const u32x4*)(ka + 16 * s));
      const bf16x8 bv = __builtin_bit_cast(bf16x8, *(const u32x4*)(qb + 16 * s));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
    }
    // lane holds keys kt*32 + 8 (e/4) + 4 hl + e%4 of query row rt*32 + col
    const int r = rt * 32 + col;
    if (r < R) {
      const int i = r / G, g = r - i * G;
      const int h = hkv * G + g;
      const int limit = a.len - n + i;        // last row this probe token sees
      float* srow = a.scores + ((long)h * n + i) * a.ld;
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int key0 = j0 + kt * 32 + 8 * e4 + 4 * hl;
        f32x4 v;
#pragma unroll
        for (int c = 0; c < 4; ++c) v[c] = key0 + c <= limit ? acc[4 * e4 + c] * a.scale : -__builtin_inff();
        *(f32x4*)(srow + key0) = v;
      }
    }
  }
}

// One workgroup per score row: its max and the inverse of its sum of exponentials.
__global__ __launch_bounds__(kThreads) void k_probe_stats(ProbeArgs a) {
  __shared__ float shf[kThreads / 64];
  __shared__ double shd[kThreads / 64];
  const float* s = a.scores + (long)blockIdx.x * a.ld;
  float m = -__builtin_inff();
  for (int j = threadIdx.x; j < a.len; j += kThreads) m = fmaxf(m, s[j]);
  m = block_reduce_max(m, shf);
  float l = 0.f;
  for (int j = threadIdx.x; j < a.len; j += kThreads) l += expf(s[j] - m);
  const double L = block_reduce_sum((double)l, shd);
  if (threadIdx.x == 0) {
    a.stats[2 * blockIdx.x] = m;
    a.stats[2 * blockIdx.x + 1] = (float)(1.0 / L);
  }
}

// 64 keys per workgroup, the score rows split over its 4 waves: each lane adds the
// normalised probabilities of its key over every fourth row, the waves' partial sums
// are combined in a fixed order (deterministic), scaled by `weight` and added to probs.
__global__ __launch_bounds__(kThreads) void k_probe_mean(ProbeArgs a) {
  extern __shared__ float s_st[];
  __shared__ float s_part[kThreads / 64][64];
  const int rows = a.n_q_heads * a.n_probe;
  for (int e = threadIdx.x; e < 2 * rows; e += kThreads) s_st[e] = a.stats[e];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + lane;
  float acc = 0.f;
  if (j < a.len) {
#pragma unroll 4
    for (int r = wave; r < rows; r += kThreads / 64)
      acc += expf(a.scores[(long)r * a.ld + j] - s_st[2 * r]) * s_st[2 * r + 1];
  }
  s_part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && j < a.len) {
    float t = s_part[0][lane];
    for (int w = 1; w < kThreads / 64; ++w) t += s_part[w][lane];
    a.probs[j] += a.weight * (t / (float)rows);
  }
}

// Group masses, in a fixed summation order (the same bits on every run): workgroup b
// takes rows [b * kGroupRowsPerBlock, ...) in rounds of 256; a row adds its probability
// to the group holding its position (binary search over this launch's sorted group
// ranges) and to the group's boundary window. Within a wave the rows of one group are
// summed by a butterfly; each wave accumulates its rounds in order into its own LDS
// copy of the launch's groups; the four copies are added in wave order and written as
// the workgroup's partial sums of every group of the launch (zeros included), so no
// accumulator needs clearing. k_group_final adds the partials in workgroup order.
__global__ __launch_bounds__(kThreads) void k_group_mass(GroupArgs a) {
  __shared__ double acc[kThreads / 64][2][kMaxGroupsPerLaunch];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < (kThreads / 64) * 2 * kMaxGroupsPerLaunch; i += kThreads) (&acc[0][0][0])[i] = 0.0;
  __syncthreads();
  const int base = blockIdx.x * kGroupRowsPerBlock;
  for (int r = 0; r < kGroupRowsPerBlock; r += kThreads) {
    const int j = base + r + tid;
    int g = -1;
    double v = 0.0, w = 0.0;
    if (j < a.len) {
      const int p = a.pos[j];
      int lo = 0, hi = a.n - 1;
      while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        if (a.range[mid][1] <= p) lo = mid + 1;
        else if (a.range[mid][0] > p) hi = mid - 1;
        else { g = mid; break; }
      }
      if (g >= 0) {
        v = (double)a.probs[j];
        w = p < a.range[g][0] + a.window ? v : 0.0;
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
  // group g's mass and window mass: the workgroups' partials in workgroup order
  auto group_sum = [&](int g, int which) {
    double t = 0.0;
    for (int b = 0; b < a.n_blocks; ++b) t += a.partial[(size_t)b * 2 * n + (size_t)which * n + g];
    return t;
  };
  double m = 0.0, w = 0.0;
  for (int g = threadIdx.x; g < n; g += kThreads) {
    const double mg = group_sum(g, 0), wg = group_sum(g, 1);
    m += mg;
    w += wg;
    a.mass[g] = (float)mg;
    if (a.window_mass) a.window_mass[g] = (float)wg;
  }
  const double M = block_reduce_sum(m, shd);
  const double W = block_reduce_sum(w, shd);
  double h = 0.0;
  for (int g = threadIdx.x; g < n; g += kThreads) {
    const double x = M > 0.0 ? group_sum(g, 0) / M : 0.0;
    if (x > 0.0) h -= x * log(x);
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
  double s = 0.0;
  const long base = (long)blockIdx.x * kTvRowsPerBlock;
  for (int e = threadIdx.x; e < kTvRowsPerBlock; e += kThreads) {
    const long j = base + e;
    if (j < a.n) {
      const long k = a.map ? (long)a.map[j] : j;
      s += fabs((double)a.p[j] - (double)a.q[k]);
    }
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

}  // namespace

hipError_t launch_probe(const ProbeArgs& a, hipStream_t s) {
  if (a.n_probe <= 0 || a.len <= 0) return hipSuccess;
  if (a.rotary_dim > 2 * kMaxHalfP || a.n_probe * (a.n_q_heads / a.n_kv_heads) > kProbeMaxRows)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_probe_rope, dim3(a.n_probe), dim3(kThreads), 0, s, a);
  const dim3 grid((a.len + kProbeKeys - 1) / kProbeKeys, a.n_kv_heads);
  if (a.head_dim == 256)
    hipLaunchKernelGGL(k_probe_scores<256>, grid, dim3(kThreads), 0, s, a);
  else if (a.head_dim == 128)
    hipLaunchKernelGGL(k_probe_scores<128>, grid, dim3(kThreads), 0, s, a);
  else if (a.head_dim == 64)
    hipLaunchKernelGGL(k_probe_scores<64>, grid, dim3(kThreads), 0, s, a);
  else
    return hipErrorInvalidValue;
  const int rows = a.n_q_heads * a.n_probe;
  hipLaunchKernelGGL(k_probe_stats, dim3(rows), dim3(kThreads), 0, s, a);
  hipLaunchKernelGGL(k_probe_mean, dim3((a.len + 63) / 64), dim3(kThreads), sizeof(float) * 2 * rows, s, a);
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
