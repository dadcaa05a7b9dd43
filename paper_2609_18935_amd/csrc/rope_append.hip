// True-tail placement (paper Section 4.1, Eq. 3; Section 4.2): the replacement
// tokens are rotated at their actual new tail positions cursor + i, and their
// keys and values are appended after the surviving rows. Keys are never rotated
// back and no placeholder rows are written.
//
// One workgroup per tail token (all contexts of a launch packed). Thread j owns
// rotary pair j: the angle (cursor + i) * theta^(-2j/r) and its sine and cosine
// are formed in float64 once and applied to every query and key head; the rotated
// values are rounded straight from float64 to bf16 (round to nearest even).
// Head dimensions beyond the rotary dimension are copied unchanged.
#include "common.h"

namespace tu {

namespace {

constexpr int kRopeThreads = 128;

__device__ __forceinline__ void rotate_heads(const bf16_t* __restrict__ x, bf16_t* __restrict__ y, int n_heads,
                                             int D, int j, int half, double cs, double sn) {
  for (int h = 0; h < n_heads; ++h) {
    const double a = (double)bf16_to_f32(x[h * D + j]);
    const double b = (double)bf16_to_f32(x[h * D + j + half]);
    y[h * D + j] = (bf16_t)f64_to_bf16_rne(a * cs - b * sn);
    y[h * D + j + half] = (bf16_t)f64_to_bf16_rne(b * cs + a * sn);
  }
}

__global__ __launch_bounds__(kRopeThreads) void k_rope_append(RopeArgs a) {
  const int tok = blockIdx.x;
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].tok_begin <= tok) ++si;
  const RopeSeq S = a.seq[si];
  const int i = tok - S.tok_begin;
  const int D = a.head_dim;
  const int Hq = a.n_q_heads;
  const int Hkv = a.n_kv_heads;
  const int r = a.rotary_dim;
  const int half = r >> 1;
  const int64_t p = S.cursor + i;
  const long row = (long)S.L_keep + i;

  const bf16_t* q = S.q + (long)i * Hq * D;
  const bf16_t* k = S.k + (long)i * Hkv * D;
  bf16_t* qo = S.q_hat + (long)i * Hq * D;
  bf16_t* ko = S.k_cache + row * Hkv * D;

  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    const double w = pow(a.theta, -2.0 * (double)j / (double)r);
    const double ang = (double)p * w;
    double sn, cs;
    sincos(ang, &sn, &cs);
    rotate_heads(q, qo, Hq, D, j, half, cs, sn);
    rotate_heads(k, ko, Hkv, D, j, half, cs, sn);
  }
  // components beyond the rotary dimension pass through
  const int rest = D - r;
  for (int e = threadIdx.x; e < rest * Hq; e += blockDim.x) {
    const int h = e / rest, d = r + e % rest;
    qo[h * D + d] = q[h * D + d];
  }
  for (int e = threadIdx.x; e < rest * Hkv; e += blockDim.x) {
    const int h = e / rest, d = r + e % rest;
    ko[h * D + d] = k[h * D + d];
  }
  // values are appended as they are
  const int nvec = (Hkv * D) >> 3;
  const u32x4* vs = (const u32x4*)(S.v + (long)i * Hkv * D);
  u32x4* vd = (u32x4*)(S.v_cache + row * Hkv * D);
  for (int e = threadIdx.x; e < nvec; e += blockDim.x) vd[e] = vs[e];
  if (threadIdx.x == 0) S.pos[row] = (int32_t)p;
}

}  // namespace

hipError_t launch_rope_append(const RopeArgs& a, int total_tokens, hipStream_t s) {
  if (total_tokens <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_rope_append, dim3(total_tokens), dim3(kRopeThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace tu
