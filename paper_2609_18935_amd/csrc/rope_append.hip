// True-tail placement (paper Section 4.1, Eq. 3; Section 4.2): the replacement
// tokens are rotated at their actual new tail positions cursor + i, and their
// keys and values are appended after the surviving rows. Keys are never rotated
// back and no placeholder rows are written. For the slot-preserving arm the paper
// compares (Section 5.2) the rotation uses positions from a short table of runs
// instead, the rows still being appended after the surviving ones.
//
// The same launch also packs the 64-key V tiles of the attention into the f16 V^T
// layout the attention kernel stages (k_stage: the first workgroups rotate tokens, the
// rest pack tiles): every tile, or, with a V^T copy kept beside the cache, only the
// tiles from the first row that changed since the copy was last refreshed. The pack
// reads the tail's values from the input rather than from the rows this launch
// appends, so the two parts never wait on each other.
//
// RoPE: one workgroup per tail token (all contexts of a launch packed). The angles
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

__device__ void rope_token(const RopeArgs& a, int tok) {
  __shared__ double s_cos[kMaxHalf];
  __shared__ double s_sin[kMaxHalf];
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].tok_begin <= tok) ++si;
  const RopeSeq& S = a.seq[si];
  const int i = tok - S.tok_begin;
  const int D = a.head_dim;
  const int Hq = a.n_q_heads;
  const int Hkv = a.n_kv_heads;
  const int r = a.rotary_dim;
  const int half = r >> 1;
  int64_t p = S.cursor + i;
  if (S.n_runs > 0) {   // slot placement: the run holding tail token i
    int q = S.run_begin;
    while (q + 1 < S.run_begin + S.n_runs && a.runs[q + 1][1] <= i) ++q;
    p = (int64_t)a.runs[q][0] + (i - a.runs[q][1]);
  }
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


// V^T pack: one workgroup per (context, kv head, 64-key tile) of the tiles to refresh:
// V rows -> f16 V^T tile in the attention kernel's LDS layout: D rows (dims) of kVtRow
// halves, each 64 keys in key_slot order within 16-key groups followed by 8 halves of
// padding (zeros; the attention kernel never reads them). Keys past the cache's data are
// zero. Thread (c, m) builds chunk c (8 keys) of the 8 rows 8m .. 8m + 7: it loads those
// 8 keys' dims 8m .. 8m + 7 (16 bytes each), transposes the 8 x 8 block in registers and
// writes 8 chunks; the threads of chunk 7 also write the rows' pads, so every cache line
// of the tile is written whole (lines written in part cost a read from HBM first). c is
// the fastest-moving index: a wave's load reads 128 contiguous bytes of each of 8 rows,
// and its store writes the 8 chunks of each of 8 V^T rows contiguously. bf16 values of magnitude 2^16 or more (or not finite) have no f16
// counterpart: the tile then holds infinities and the call's status gets kFaultRange.
template <int D>
__device__ void vt_pack_tile(const RopeArgs& r, const PackArgs& pa, int item) {
  constexpr int M = D / 8;                 // 8-dim blocks per row
  constexpr int CPR = kVtRow / 8;          // chunks per V^T row
  int si = 0;
  while (si + 1 < pa.n_seq && pa.seq[si + 1].pack_begin <= item) ++si;
  const PackSeq& P = pa.seq[si];
  const RopeSeq& S = r.seq[si];
  const int local = item - P.pack_begin;
  const int n_tiles = P.tile_end - P.tile_begin;
  const int kt = P.tile_begin + local % n_tiles;
  const int hkv = local / n_tiles;
  const int L_keep = S.L_keep;
  const int n_valid = L_keep + S.T;
  const int key0 = kt * kAttnKeys;
  const long rs = (long)r.n_kv_heads * D;
  const bf16_t* src = S.v_cache + (long)hkv * D;
  const bf16_t* src_new = S.v + (long)hkv * D;   // tail row key - L_keep
  _Float16* dst = P.vt + ((long)hkv * P.head_tiles + kt) * (D * kVtRow);
  uint32_t big = 0;   // largest |bf16| bit pattern converted (two per word)
  for (int w = threadIdx.x; w < 8 * M; w += kRopeThreads) {
    const int c = w & 7;        // key chunk 0..7 (consecutive threads)
    const int m = w >> 3;       // 8-dim block
    u32x4 rowv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int key = key0 + key_slot(8 * c + j);
      const bf16_t* row = (key < L_keep ? src + (long)key * rs : src_new + (long)(key - L_keep) * rs) + 8 * m;
      rowv[j] = key < n_valid ? *(const u32x4*)row : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int e = 0; e < 4; ++e) big = max(big, max(rowv[j][e] & 0x7FFFu, (rowv[j][e] >> 16) & 0x7FFFu));
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      f16x8 h;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t word = rowv[j][d >> 1];
        h[j] = (_Float16)bf16_to_f32((d & 1) ? (word >> 16) : (word & 0xFFFFu));
      }
      *(f16x8*)(dst + ((8 * m + d) * CPR + c) * 8) = h;
      if (c == 7) *(u32x4*)(dst + ((8 * m + d) * CPR + 8) * 8) = u32x4{0, 0, 0, 0};
    }
  }
  if (big >= 0x4780u) status_raise(pa.status, kFaultRange);   // 0x4780: bf16 bits of 2^16
}

template <int D>
__global__ __launch_bounds__(kRopeThreads) void k_stage(RopeArgs r, PackArgs p, int rope_tokens) {
  status_mark(p.status);
  const int b = blockIdx.x;
  if (b < rope_tokens) {
    rope_token(r, b);
    return;
  }
  if (b - rope_tokens < p.pack_items) vt_pack_tile<D>(r, p, b - rope_tokens);
}

// Key relocation (Section 5.2, tail-and-relocate): one workgroup per moved row. The
// row's shift delta gives the angles delta * theta^(-2j/r), formed in float64 once per
// rotary pair into LDS; every key buffer's row is then turned pair by pair in place
// (float64 rotation of the stored bf16 values, rounded to bf16 nearest even), and the
// row's position label moves by delta.
__global__ __launch_bounds__(kRopeThreads) void k_relocate(RelocArgs a) {
  __shared__ double s_cos[kMaxHalf];
  __shared__ double s_sin[kMaxHalf];
  const int b = blockIdx.x;
  int s = 0;
  while (s + 1 < a.n_spans && a.block_begin[s + 1] <= b) ++s;
  const long row = (long)a.row[s] + (b - a.block_begin[s]);
  const int delta = a.delta[s];
  const int D = a.head_dim, Hkv = a.n_kv_heads, r = a.rotary_dim, half = r >> 1;
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    const double w = pow(a.theta, -2.0 * (double)j / (double)r);
    double sn, cs;
    sincos((double)delta * w, &sn, &cs);
    s_cos[j] = cs;
    s_sin[j] = sn;
  }
  __syncthreads();
  for (int bi = 0; bi < a.n_bufs; ++bi) {
    bf16_t* x = a.bufs[bi] + row * Hkv * D;
    for (int w = threadIdx.x; w < Hkv * half; w += blockDim.x) {
      const int h = w / half, j = w - h * half;
      bf16_t* y = x + (long)h * D;
      const double av = (double)bf16_to_f32(y[j]);
      const double bv = (double)bf16_to_f32(y[j + half]);
      y[j] = (bf16_t)f64_to_bf16_rne(av * s_cos[j] - bv * s_sin[j]);
      y[j + half] = (bf16_t)f64_to_bf16_rne(bv * s_cos[j] + av * s_sin[j]);
    }
  }
  if (threadIdx.x == 0 && a.pos) a.pos[row] += delta;
}

}  // namespace

hipError_t launch_relocate(const RelocArgs& a, hipStream_t s) {
  const int blocks = a.block_begin[a.n_spans];
  if (blocks <= 0) return hipSuccess;
  if (a.n_bufs > 0 && a.rotary_dim > 2 * kMaxHalf) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_relocate, dim3(blocks), dim3(kRopeThreads), 0, s, a);
  return hipGetLastError();
}

static_assert(sizeof(RopeArgs) + sizeof(PackArgs) + sizeof(int) <= kMaxKernargBytes, "stage launch record");
static_assert(sizeof(RelocArgs) <= kMaxKernargBytes, "relocation launch record");

hipError_t launch_stage(const RopeArgs& r, int rope_tokens, const PackArgs& a, int head_dim, hipStream_t s) {
  const int blocks = rope_tokens + a.pack_items;
  if (blocks <= 0) return hipSuccess;
  if (r.rotary_dim > 2 * kMaxHalf) return hipErrorInvalidValue;
  if (head_dim == 256)
    hipLaunchKernelGGL(k_stage<256>, dim3(blocks), dim3(kRopeThreads), 0, s, r, a, rope_tokens);
  else if (head_dim == 128)
    hipLaunchKernelGGL(k_stage<128>, dim3(blocks), dim3(kRopeThreads), 0, s, r, a, rope_tokens);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_stage<64>, dim3(blocks), dim3(kRopeThreads), 0, s, r, a, rope_tokens);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tu
