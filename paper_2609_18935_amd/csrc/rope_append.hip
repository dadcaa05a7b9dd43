// True-tail placement (paper Section 4.1, Eq. 3; Section 4.2): the replacement
// tokens are rotated at their actual new tail positions cursor + i, and their
// keys and values are appended after the surviving rows. Keys are never rotated
// back and no placeholder rows are written.
//
// One workgroup per tail token (all contexts of a launch packed). The angles
// (cursor + i) * theta^(-2j/r) and their sines and cosines are formed in float64,
// once per rotary pair j, into LDS. Then each thread rotates 8 consecutive pairs of
// one query or key head: two 16-byte loads (components j .. j+7 and j+r/2 ..
// j+r/2+7), the rotation in float64, rounding straight from float64 to bf16 (round
// to nearest even), two 16-byte stores. A rotary dimension not divisible by 16 takes
// a scalar path; head dimensions beyond the rotary dimension are copied unchanged.
#include "common.h"

namespace tu {

namespace {

constexpr int kRopeThreads = 256;
constexpr int kMaxHalf = 128;   // rotary pairs per head (head_dim <= 256)

__device__ __forceinline__ uint32_t pack_bf16(double lo, double hi) {
  return f64_to_bf16_rne(lo) | (f64_to_bf16_rne(hi) << 16);
}

__global__ __launch_bounds__(kRopeThreads) void k_rope_append(RopeArgs a) {
  __shared__ double s_cos[kMaxHalf];
  __shared__ double s_sin[kMaxHalf];
  const int tok = blockIdx.x;
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].tok_begin <= tok) ++si;
  const RopeSeq& S = a.seq[si];
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
    double sn, cs;
    sincos((double)p * w, &sn, &cs);
    s_cos[j] = cs;
    s_sin[j] = sn;
  }
  __syncthreads();

  // rotate: groups of 8 pairs, heads 0 .. Hq-1 are queries, then Hkv keys (16-byte
  // accesses need r / 2 to be a multiple of 8; otherwise every pair goes the scalar way)
  const int n_grp = (half & 7) ? 0 : half >> 3;
  const int H = Hq + Hkv;
  for (int w = threadIdx.x; w < H * n_grp; w += blockDim.x) {
    const int h = w / n_grp;
    const int j0 = (w - h * n_grp) * 8;
    const bf16_t* x = h < Hq ? q + (long)h * D : k + (long)(h - Hq) * D;
    bf16_t* y = h < Hq ? qo + (long)h * D : ko + (long)(h - Hq) * D;
    const u32x4 va = *(const u32x4*)(x + j0);
    const u32x4 vb = *(const u32x4*)(x + half + j0);
    u32x4 oa, ob;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double ra[2], rb[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int j = j0 + 2 * e + t;
        const double av = (double)bf16_to_f32(t ? (va[e] >> 16) : (va[e] & 0xFFFFu));
        const double bv = (double)bf16_to_f32(t ? (vb[e] >> 16) : (vb[e] & 0xFFFFu));
        ra[t] = av * s_cos[j] - bv * s_sin[j];
        rb[t] = bv * s_cos[j] + av * s_sin[j];
      }
      oa[e] = pack_bf16(ra[0], ra[1]);
      ob[e] = pack_bf16(rb[0], rb[1]);
    }
    *(u32x4*)(y + j0) = oa;
    *(u32x4*)(y + half + j0) = ob;
  }
  // pairs past the last full group
  const int tail = half - n_grp * 8;
  for (int w = threadIdx.x; w < H * tail; w += blockDim.x) {
    const int h = w / tail;
    const int j = n_grp * 8 + (w - h * tail);
    const bf16_t* x = h < Hq ? q + (long)h * D : k + (long)(h - Hq) * D;
    bf16_t* y = h < Hq ? qo + (long)h * D : ko + (long)(h - Hq) * D;
    const double av = (double)bf16_to_f32(x[j]);
    const double bv = (double)bf16_to_f32(x[j + half]);
    y[j] = (bf16_t)f64_to_bf16_rne(av * s_cos[j] - bv * s_sin[j]);
    y[j + half] = (bf16_t)f64_to_bf16_rne(bv * s_cos[j] + av * s_sin[j]);
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
  if (a.rotary_dim > 2 * kMaxHalf) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_rope_append, dim3(total_tokens), dim3(kRopeThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace tu
