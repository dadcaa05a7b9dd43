// Gated delta-rule continuation (paper Section 4.1, Eq. 3: the recurrent state
// continues from its previous value over the replacement tokens; the layers are
// Gated DeltaNet layers, Yang et al. 2025). Per value head the state S (d_v x d_k)
// follows
//     S_t = g_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,   o_t = scale S_t q_t.
//
// The tail is cut into chunks of C tokens starting at its first token. Inside a
// chunk (rows r, i), with lg_r = sum_{s<=r} log2 g_s and G[r][i] = 2^(lg_r - lg_i):
//     M = strictly-lower(diag(beta) (G .* K K^T)),   T = (I + M)^-1
//     W = T diag(beta 2^lg) K,   U~ = T diag(beta) V                     (k_delta_prep)
//     U = U~ - W S^T
//     O = scale (diag(2^lg) Q S^T + lower(G .* Q K^T) U)
//     S <- 2^lg_last S + U^T diag(2^(lg_last - lg)) K                      (k_delta_chain)
// Only decay ratios <= 1 are formed. A ragged last chunk is padded with k = q = v = 0,
// beta = 0, g = 1, which leaves the recurrence unchanged.
//
// k_delta_prep: one workgroup per (chunk, value head), all chunks in parallel.
//   K K^T and Q K^T on v_mfma_f32_16x16x32_bf16 (exact bf16 products, fp32 sums);
//   T by blocked forward substitution in fp32 (16x16 diagonal blocks by one lane per
//   column, then off-diagonal blocks level by level); W and U~ on
//   v_mfma_f32_16x16x32_f16 with T and the scaled K, V rounded to f16. Writes W (f16),
//   U~ (fp32), P = scale * lower(G .* Q K^T) (f16) and lg (fp32) to the workspace.
// k_delta_chain: one workgroup per (context, value head, slice of DVS rows of S). Rows
//   of S evolve independently (row i only needs U[:, i]), so slicing d_v spreads a
//   head over several workgroups. The fp32 state slice lives in MFMA accumulators
//   for the whole tail, is read from HBM once and written once; each chunk it is
//   rounded to f16 into LDS to serve as the MFMA operand of W S^T and Q S^T.
//   f16 (10 stored mantissa bits) keeps the operands of these fp32-intermediate
//   products accurate enough for the error bound where bf16 would not.
#include "common.h"

namespace tu {

namespace {

typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;

__device__ __forceinline__ f16x8 ld_f16x8(const _Float16* p) { return __builtin_bit_cast(f16x8, *(const u32x4*)p); }
__device__ __forceinline__ bf16x8 ld_bf16x8(const bf16_t* p) { return __builtin_bit_cast(bf16x8, *(const u32x4*)p); }
__device__ __forceinline__ f16x8 zero_f16x8() { return __builtin_bit_cast(f16x8, u32x4{0, 0, 0, 0}); }

__device__ __forceinline__ f32x4 mfma_f16(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Operands rounded to f16 must stay within its range: a larger magnitude rounds to
// infinity, and the kernels then set kFaultRange in the call's status.
constexpr float kF16Max = 65504.f;
__device__ __forceinline__ float max_abs4(f32x4 v) {
  return fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3])));
}

__device__ __forceinline__ int find_seq_by_chunk(const DeltaArgs& a, int c) {
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].chunk_begin <= c) ++si;
  return si;
}

constexpr int cmax(size_t x, size_t y) { return (int)(x > y ? x : y); }

// ------------------------------------------------------------------ prep
constexpr int kPrepThreads = 512;   // 8 waves
template <int DK, int C>
__global__ __launch_bounds__(kPrepThreads) void k_delta_prep(DeltaArgs a) {
  constexpr int NT = kPrepThreads;
  constexpr int NW = NT / 64;
  constexpr int DV = DK;
  constexpr int NB = C / 16;     // 16-row blocks of the chunk
  constexpr int KP = DK + 8;     // pitch of [C][DK] bf16 tiles
  constexpr int CP = C + 4;      // pitch of [C][C] fp32 tiles
  constexpr int CH = C + 8;      // pitch of [*][C] f16 tiles
  // LDS regions shared by arrays whose lifetimes do not overlap, so that two workgroups
  // fit a CU: K (phases 0-5a) then (beta 2^lg K)^T (5b-6); Q (0-5a) then (beta V)^T
  // (5b-6); M (1-4) then T in f16 (5a-6). A barrier separates 5a (the last reads of K,
  // Q and T in fp32) from 5b (the first writes of the transposed copies).
  constexpr int R1 = cmax(sizeof(bf16_t) * C * KP, sizeof(_Float16) * DK * CH);
  constexpr int R2 = cmax(sizeof(bf16_t) * C * KP, sizeof(_Float16) * DV * CH);
  constexpr int R3 = cmax(sizeof(float) * C * CP, sizeof(_Float16) * C * CH);
  __shared__ __attribute__((aligned(16))) char r1[R1];
  __shared__ __attribute__((aligned(16))) char r2[R2];
  __shared__ __attribute__((aligned(16))) char r3[R3];
  __shared__ __attribute__((aligned(16))) float Tf[C][CP];
  __shared__ __attribute__((aligned(16))) float Xs[3][16][20];
  __shared__ __attribute__((aligned(16))) float lg[C];
  __shared__ __attribute__((aligned(16))) float bt[C];
  auto& Ks = *reinterpret_cast<bf16_t(*)[C][KP]>(r1);
  auto& Bt = *reinterpret_cast<_Float16(*)[DK][CH]>(r1);
  auto& Qs = *reinterpret_cast<bf16_t(*)[C][KP]>(r2);
  auto& Vt = *reinterpret_cast<_Float16(*)[DV][CH]>(r2);
  auto& Mf = *reinterpret_cast<float(*)[C][CP]>(r3);
  auto& Th = *reinterpret_cast<_Float16(*)[C][CH]>(r3);

  const int Hk = a.n_k_heads, Hv = a.n_v_heads;
  const int c = blockIdx.x / Hv;          // global chunk
  const int h = blockIdx.x - c * Hv;      // value head
  const int si = find_seq_by_chunk(a, c);
  const DeltaSeq S = a.seq[si];
  const int t0 = (c - S.chunk_begin) * C;
  const int Cr = min(C, S.T - t0);
  const int kh = h / (Hv / Hk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g4 = lane >> 4;
  float big = 0.f;   // largest magnitude this thread rounds to f16
  status_mark(a.status);

  // ---- phase 0: stage K, Q (bf16), beta, log2 g
  for (int e = tid; e < C * (DK / 8); e += NT) {
    const int r = e / (DK / 8), cc = e - r * (DK / 8);
    u32x4 kw = {0, 0, 0, 0}, qw = {0, 0, 0, 0};
    if (r < Cr) {
      const long off = ((long)(t0 + r) * Hk + kh) * DK + cc * 8;
      kw = *(const u32x4*)(S.k + off);
      qw = *(const u32x4*)(S.q + off);
    }
    *(u32x4*)&Ks[r][cc * 8] = kw;
    *(u32x4*)&Qs[r][cc * 8] = qw;
  }
  // the values this thread converts in phase 5, fetched now so their latency overlaps
  // phases 1-4 ((C / 4) * (DK / 8) <= NT: one item per thread at most)
  constexpr int NE5 = (C / 4) * (DK / 8);
  static_assert(NE5 <= NT, "phase 5 maps one item per thread");
  u32x4 vw[4];
  if (tid < NE5) {
    const int s4 = (tid % (C / 4)) * 4, d0 = (tid / (C / 4)) * 8;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      vw[j] = (s4 + j < Cr) ? *(const u32x4*)(S.v + ((long)(t0 + s4 + j) * Hv + h) * DV + d0) : u32x4{0, 0, 0, 0};
  }
  if (tid < C) {
    const bool ok = tid < Cr;
    bt[tid] = ok ? S.beta[(long)(t0 + tid) * Hv + h] : 0.f;
    // log2 g, held at -100 or above: a gate of exactly 0 would give -inf and, in the
    // differences of the cumulative sums below, NaN; 2^-100 of the state is far below
    // fp32 rounding of any other term
    lg[tid] = ok ? fmaxf(__log2f(S.g[(long)(t0 + tid) * Hv + h]), -100.f) : 0.f;
  }
  lds_barrier();

  // ---- phase 1: cumulative log-decay (wave 0) and K K^T, Q K^T lower blocks (MFMA)
  if (wave == 0) {
    float x = lane < C ? lg[lane] : 0.f;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const float y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane < C) lg[lane] = x;
  }
  constexpr int NLB = NB * (NB + 1) / 2;   // lower blocks incl. diagonal
  constexpr int NPW = (2 * NLB + NW - 1) / NW;   // blocks per wave (KK and QK together)
  f32x4 acc[NPW];
  int blk_of[NPW];
#pragma unroll
  for (int j = 0; j < NPW; ++j) {
    const int idx = wave + NW * j;
    blk_of[j] = idx;
    acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (idx < 2 * NLB) {
      const int li = idx % NLB;
      const bool is_q = idx >= NLB;
      int bi = 0;
      while ((bi + 1) * (bi + 2) / 2 <= li) ++bi;
      const int bj = li - bi * (bi + 1) / 2;
      // transposed product: the lane ends up with row 16 bi + l16 and the 4 consecutive
      // columns 16 bj + 4 g4 .. (K K^T is symmetric; Q K^T is formed as (K Q^T)^T)
#pragma unroll
      for (int kk = 0; kk < DK / 32; ++kk) {
        const bf16x8 av = ld_bf16x8(&Ks[16 * bj + l16][32 * kk + 8 * g4]);
        const bf16x8 bv = is_q ? ld_bf16x8(&Qs[16 * bi + l16][32 * kk + 8 * g4])
                               : ld_bf16x8(&Ks[16 * bi + l16][32 * kk + 8 * g4]);
        acc[j] = mfma_bf16(av, bv, acc[j]);
      }
    }
  }
  lds_barrier();   // lg ready

  // ---- phase 2: M (fp32, LDS) and P (f16, workspace) from the MFMA results
  const long slot = (long)c * Hv + h;
  _Float16* Pg = a.ws_p + slot * C * C;
#pragma unroll
  for (int j = 0; j < NPW; ++j) {
    const int idx = blk_of[j];
    if (idx >= 2 * NLB) continue;
    const int li = idx % NLB;
    const bool is_q = idx >= NLB;
    int bi = 0;
    while ((bi + 1) * (bi + 2) / 2 <= li) ++bi;
    const int bj = li - bi * (bi + 1) / 2;
    const int r = 16 * bi + l16, i0 = 16 * bj + 4 * g4;   // row, first of 4 columns
    const float lr = lg[r];
    const f32x4 li4 = *(const f32x4*)&lg[i0];
    if (is_q) {
      f16x4 pv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = i0 + e <= r ? a.scale * __builtin_amdgcn_exp2f(fminf(lr - li4[e], 0.f)) * acc[j][e] : 0.f;
        big = fmaxf(big, fabsf(x));
        pv[e] = (_Float16)x;
      }
      *(f16x4*)&Pg[r * C + i0] = pv;
    } else {
      const float br = bt[r];
      f32x4 mv;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        mv[e] = i0 + e < r ? br * __builtin_amdgcn_exp2f(fminf(lr - li4[e], 0.f)) * acc[j][e] : 0.f;
      *(f32x4*)&Mf[r][i0] = mv;
    }
  }
  // zero the upper blocks of P
  for (int e = tid; e < C * C / 8; e += NT) {
    const int r = e / (C / 8), i = (e - r * (C / 8)) * 8;
    if ((i >> 4) > (r >> 4)) *(u32x4*)&Pg[r * C + i] = u32x4{0, 0, 0, 0};
  }
  if (tid < C) a.ws_lg[slot * C + tid] = lg[tid];
  lds_barrier();

  // ---- phase 3: diagonal 16x16 blocks of T = (I + M)^-1, one lane per column
  if (wave == 0 && g4 < NB) {
    const int b = g4, cc = l16;
    float x[16];
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < rr; ++i) s += Mf[16 * b + rr][16 * b + i] * x[i];
      x[rr] = rr < cc ? 0.f : (rr == cc ? 1.f : -s);
    }
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) Tf[16 * b + rr][16 * b + cc] = x[rr];
  }
  lds_barrier();

  // ---- phase 4: off-diagonal blocks, level by level: T_ij = -T_ii sum_{m=j}^{i-1} M_im T_mj.
  // One wave per block of the level, 16x16x16 products on v_mfma_f32_16x16x4_f32 (fp32
  // operands and sums); the sum X is staged through the wave's own LDS tile to serve as
  // the B operand of the second product.
#pragma unroll
  for (int lev = 1; lev < NB; ++lev) {
    const int nblk = NB - lev;
    if (wave < nblk) {
      const int j = wave, i = wave + lev;
      f32x4 x = {0.f, 0.f, 0.f, 0.f};
      for (int m = j; m < i; ++m)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          x = __builtin_amdgcn_mfma_f32_16x16x4f32(Mf[16 * i + l16][16 * m + 4 * s + g4],
                                                   Tf[16 * m + 4 * s + g4][16 * j + l16], x, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) Xs[wave][4 * g4 + e][l16] = x[e];
      __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // this wave's LDS writes are done
      f32x4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        y = __builtin_amdgcn_mfma_f32_16x16x4f32(Tf[16 * i + l16][16 * i + 4 * s + g4], Xs[wave][4 * s + g4][l16], y,
                                                 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) Tf[16 * i + 4 * g4 + e][16 * j + l16] = -y[e];
    }
    lds_barrier();
  }

  // ---- phase 5a: T to f16 (lower, zero upper; M is dead), this thread's K rows into
  // registers, and scale * 2^lg Q as f16 (the chain's Q S^T operand, row decay folded in)
  for (int e = tid; e < C * C; e += NT) {
    const int r = e / C, i = e - r * C;
    const float x = (i >> 4) <= (r >> 4) ? Tf[r][i] : 0.f;
    big = fmaxf(big, fabsf(x));
    Th[r][i] = (_Float16)x;
  }
  u32x4 kw[4];
  if (tid < NE5) {
    const int s4 = (tid % (C / 4)) * 4, d0 = (tid / (C / 4)) * 8;
#pragma unroll
    for (int j = 0; j < 4; ++j) kw[j] = *(const u32x4*)&Ks[s4 + j][d0];
  }
  for (int e = tid; e < C * (DK / 8); e += NT) {
    const int r = e / (DK / 8), cc = e - r * (DK / 8);
    const float w = a.scale * __builtin_amdgcn_exp2f(lg[r]);
    const u32x4 qw = *(const u32x4*)&Qs[r][cc * 8];
    f16x8 hq;
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const uint32_t qb = (d & 1) ? (qw[d >> 1] & 0xFFFF0000u) : (qw[d >> 1] << 16);
      const float x = w * __uint_as_float(qb);
      big = fmaxf(big, fabsf(x));
      hq[d] = (_Float16)x;
    }
    *(f16x8*)(a.ws_q + slot * C * DK + (long)r * DK + cc * 8) = hq;
  }
  lds_barrier();   // K and Q are no longer read: their regions take the transposed copies

  // ---- phase 5b: (beta 2^lg K)^T and (beta V)^T in f16, and the decayed K^T for the chain
  if (tid < NE5) {
    const int s4 = (tid % (C / 4)) * 4, d0 = (tid / (C / 4)) * 8;
    float wk[4], wv[4], wd[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int s = s4 + j;
      wv[j] = bt[s];
      wk[j] = bt[s] * __builtin_amdgcn_exp2f(lg[s]);
      wd[j] = __builtin_amdgcn_exp2f(lg[C - 1] - lg[s]);
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      f16x4 hk, hv, hd;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t kb = (d & 1) ? (kw[j][d >> 1] & 0xFFFF0000u) : (kw[j][d >> 1] << 16);
        const uint32_t vb = (d & 1) ? (vw[j][d >> 1] & 0xFFFF0000u) : (vw[j][d >> 1] << 16);
        const float xk = wk[j] * __uint_as_float(kb), xv = wv[j] * __uint_as_float(vb);
        const float xd = wd[j] * __uint_as_float(kb);
        big = fmaxf(big, fmaxf(fabsf(xk), fmaxf(fabsf(xv), fabsf(xd))));
        hk[j] = (_Float16)xk;
        hv[j] = (_Float16)xv;
        hd[j] = (_Float16)xd;
      }
      *(f16x4*)&Bt[d0 + d][s4] = hk;
      *(f16x4*)&Vt[d0 + d][s4] = hv;
      *(f16x4*)(a.ws_kt + slot * DK * C + (long)(d0 + d) * C + s4) = hd;
    }
  }
  lds_barrier();

  // ---- phase 6: W = T (beta 2^lg K), U~ = T (beta V) on MFMA; write to workspace
  _Float16* Wg = a.ws_w + slot * C * DK;
  float* Ug = a.ws_u + slot * C * DV;
  constexpr int NOB = NB * (DK / 16);   // output blocks per matrix
  for (int idx = wave; idx < 2 * NOB; idx += NW) {
    const bool is_u = idx >= NOB;
    const int b = idx % NOB;
    const int rb = b / (DK / 16), db = b % (DK / 16);
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    // transposed product (X^T T^T): the lane ends up with row 16 rb + l16 and the 4
    // consecutive columns 16 db + 4 g4 .. of W (or U~), stored as one vector
#pragma unroll
    for (int kk = 0; kk < (C + 31) / 32; ++kk) {
      f16x8 av = zero_f16x8(), bv = zero_f16x8();
      if (C >= 32 || g4 < 2) {
        av = is_u ? ld_f16x8(&Vt[16 * db + l16][32 * kk + 8 * g4]) : ld_f16x8(&Bt[16 * db + l16][32 * kk + 8 * g4]);
        bv = ld_f16x8(&Th[16 * rb + l16][32 * kk + 8 * g4]);
      }
      o = mfma_f16(av, bv, o);
    }
    const int r = 16 * rb + l16, d0 = 16 * db + 4 * g4;
    if (is_u) {
      *(f32x4*)&Ug[r * DV + d0] = o;
    } else {
      big = fmaxf(big, fmaxf(fmaxf(fabsf(o[0]), fabsf(o[1])), fmaxf(fabsf(o[2]), fabsf(o[3]))));
      const f16x4 wv = {(_Float16)o[0], (_Float16)o[1], (_Float16)o[2], (_Float16)o[3]};
      *(f16x4*)&Wg[r * DK + d0] = wv;
    }
  }
  if (big > kF16Max) status_raise(a.status, kFaultRange);
}

// ------------------------------------------------------------------ chain
constexpr int kChainThreads = 1024;  // 16 waves: four per SIMD interleave their latencies
template <int DK, int C, int DVS>
__global__ __launch_bounds__(kChainThreads) void k_delta_chain(DeltaArgs a) {
  constexpr int NT = kChainThreads;
  constexpr int NW = NT / 64;
  constexpr int DV = DK;
  constexpr int KP = DK + 8;
  constexpr int CH = C + 8;
  constexpr int NCB = DVS / 16;                 // column blocks of the slice
  constexpr int NXB = (C / 16) * NCB;           // blocks of W S^T / Q S^T / O
  constexpr int NXW = (NXB + NW - 1) / NW;      // per wave
  constexpr int NSB = (DK / 16) * NCB;          // blocks of S^T
  constexpr int NSW = (NSB + NW - 1) / NW;      // per wave (the last ones may own none)
  // per-chunk operands staged from the workspace (all f16 except U~)
  constexpr int VQ = C * DK / 8;                // 16-byte vectors of W and of Qg
  constexpr int VK = DK * C / 8;                // of Kd^T
  constexpr int VP = C * C / 8;                 // of P
  constexpr int VU = C * DVS / 4;               // 16-byte vectors of the U~ slice (fp32)
  constexpr int RQ = (VQ + NT - 1) / NT, RK = (VK + NT - 1) / NT, RP = (VP + NT - 1) / NT, RU = (VU + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) _Float16 Ws[C][KP];
  __shared__ __attribute__((aligned(16))) _Float16 Qs[C][KP];
  __shared__ __attribute__((aligned(16))) _Float16 Kdt[DK][CH];
  __shared__ __attribute__((aligned(16))) _Float16 Ph[C][CH];
  __shared__ __attribute__((aligned(16))) float Us[C][DVS + 4];
  __shared__ __attribute__((aligned(16))) _Float16 Ut[DVS][CH];
  __shared__ __attribute__((aligned(16))) _Float16 Sh[DVS][KP];
  __shared__ float s_glast;

  const int Hv = a.n_v_heads;
  const int per_seq = Hv * a.n_slices;
  int si, h, sl;
  if ((Hv & 7) == 0) {
    // workgroup b runs on XCD b % 8 (round-robin dispatch); the prep workgroup of
    // (chunk, head h) ran on XCD h % 8, so every slice of head h is placed there too and
    // finds the head's chunk operands in that XCD's L2
    const int b = blockIdx.x;
    const int hx = b & 7;                     // h % 8
    const int rest = b >> 3;                  // (seq, h / 8, slice)
    sl = rest % a.n_slices;
    const int hq = (rest / a.n_slices) % (Hv >> 3);
    si = rest / a.n_slices / (Hv >> 3);
    h = 8 * hq + hx;
  } else {
    const int item = xcd_remap(blockIdx.x, gridDim.x);   // slices of one head share an XCD
    si = item / per_seq;
    const int rem = item - si * per_seq;
    h = rem / a.n_slices;
    sl = rem - h * a.n_slices;
  }
  if (si >= a.n_seq) return;
  const int i0 = sl * DVS;
  const DeltaSeq S = a.seq[si];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g4 = lane >> 4;
  const bool kpart = (C >= 32) || (g4 < 2);     // lanes that carry chunk-dim K elements
  float big = 0.f;   // largest magnitude this thread rounds to f16 (S copy, U)

  // ---- load the state slice: S^T blocks (d rows, i cols) in accumulators, f16 copy in LDS
  float* Sg = S.state + (long)h * DV * DK;
  f32x4 st[NSW];
#pragma unroll
  for (int j = 0; j < NSW; ++j) {
    const int b = wave + NW * j;
    if (b >= NSB) continue;
    const int db = b / NCB, cb = b % NCB;
    const int i = 16 * cb + l16, d = 16 * db + 4 * g4;
    st[j] = *(const f32x4*)(Sg + (long)(i0 + i) * DK + d);
    big = fmaxf(big, max_abs4(st[j]));
    f16x4 hv = {(_Float16)st[j][0], (_Float16)st[j][1], (_Float16)st[j][2], (_Float16)st[j][3]};
    *(f16x4*)&Sh[i][d] = hv;
  }

  // ---- next chunk's operands are fetched into registers while the current one is computed
  u32x4 rw[RQ], rq[RQ], rk[RK], rp[RP], ru[RU];
  float rg = 0.f;
  auto prefetch = [&](int lc) {
    const long slot = (long)(S.chunk_begin + lc) * Hv + h;
    const u32x4* W4 = (const u32x4*)(a.ws_w + slot * C * DK);
    const u32x4* Q4 = (const u32x4*)(a.ws_q + slot * C * DK);
    const u32x4* K4 = (const u32x4*)(a.ws_kt + slot * DK * C);
    const u32x4* P4 = (const u32x4*)(a.ws_p + slot * C * C);
    const float* U = a.ws_u + slot * C * DV + i0;
#pragma unroll
    for (int j = 0; j < RQ; ++j) {
      const int e = tid + NT * j;
      if (e < VQ) {
        rw[j] = W4[e];
        rq[j] = Q4[e];
      }
    }
#pragma unroll
    for (int j = 0; j < RK; ++j)
      if (tid + NT * j < VK) rk[j] = K4[tid + NT * j];
#pragma unroll
    for (int j = 0; j < RP; ++j)
      if (tid + NT * j < VP) rp[j] = P4[tid + NT * j];
#pragma unroll
    for (int j = 0; j < RU; ++j) {
      const int e = tid + NT * j;
      if (e < VU) {
        const int r = e / (DVS / 4), c4 = e - r * (DVS / 4);
        ru[j] = *(const u32x4*)(U + (long)r * DV + 4 * c4);
      }
    }
    rg = a.ws_lg[slot * C + C - 1];
  };
  auto stage = [&]() {
#pragma unroll
    for (int j = 0; j < RQ; ++j) {
      const int e = tid + NT * j;
      if (e < VQ) {
        const int r = e / (DK / 8), c8 = e - r * (DK / 8);
        *(u32x4*)&Ws[r][8 * c8] = rw[j];
        *(u32x4*)&Qs[r][8 * c8] = rq[j];
      }
    }
#pragma unroll
    for (int j = 0; j < RK; ++j) {
      const int e = tid + NT * j;
      if (e < VK) {
        const int d = e / (C / 8), c8 = e - d * (C / 8);
        *(u32x4*)&Kdt[d][8 * c8] = rk[j];
      }
    }
#pragma unroll
    for (int j = 0; j < RP; ++j) {
      const int e = tid + NT * j;
      if (e < VP) {
        const int r = e / (C / 8), c8 = e - r * (C / 8);
        *(u32x4*)&Ph[r][8 * c8] = rp[j];
      }
    }
#pragma unroll
    for (int j = 0; j < RU; ++j) {
      const int e = tid + NT * j;
      if (e < VU) {
        const int r = e / (DVS / 4), c4 = e - r * (DVS / 4);
        *(u32x4*)&Us[r][4 * c4] = ru[j];
      }
    }
    if (tid == 0) s_glast = __builtin_amdgcn_exp2f(rg);
  };

  prefetch(0);
  for (int lc = 0; lc < S.n_chunks; ++lc) {
    const int t0 = lc * C;
    const int Cr = min(C, S.T - t0);
    stage();
    lds_barrier();
    if (lc + 1 < S.n_chunks) prefetch(lc + 1);
    const float g_last = s_glast;

    // ---- X = W S^T -> U = U~ - X (to LDS as U^T);  Y = Qg S^T starts O
    f32x4 oacc[NXW];
#pragma unroll
    for (int j = 0; j < NXW; ++j) {
      const int b = wave + NW * j;
      oacc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (b >= NXB) continue;
      const int rb = b / NCB, cb = b % NCB;
      f32x4 x = {0.f, 0.f, 0.f, 0.f}, y = {0.f, 0.f, 0.f, 0.f};
      // X in (rows, slice columns) layout for U; Y transposed (S Qg^T) so that the lane
      // holds one row and 4 consecutive columns of O
#pragma unroll
      for (int kk = 0; kk < DK / 32; ++kk) {
        const f16x8 sv = ld_f16x8(&Sh[16 * cb + l16][32 * kk + 8 * g4]);
        x = mfma_f16(ld_f16x8(&Ws[16 * rb + l16][32 * kk + 8 * g4]), sv, x);
        y = mfma_f16(sv, ld_f16x8(&Qs[16 * rb + l16][32 * kk + 8 * g4]), y);
      }
      f16x4 uh;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float u = Us[16 * rb + 4 * g4 + e][16 * cb + l16] - x[e];
        big = fmaxf(big, fabsf(u));
        uh[e] = (_Float16)u;
      }
      *(f16x4*)&Ut[16 * cb + l16][16 * rb + 4 * g4] = uh;
      oacc[j] = y;
    }
    lds_barrier();

    // ---- O += P U, written out; S^T <- 2^lg_last S^T + Kd^T U; refresh the f16 copy of S
#pragma unroll
    for (int j = 0; j < NXW; ++j) {
      const int b = wave + NW * j;
      if (b >= NXB) continue;
      const int rb = b / NCB, cb = b % NCB;
      f32x4 o = oacc[j];
      // (P U)^T = U^T P^T: row 16 rb + l16, columns 16 cb + 4 g4 .. + 3 of O
#pragma unroll
      for (int kk = 0; kk < (C + 31) / 32; ++kk) {
        f16x8 av = zero_f16x8(), bv = zero_f16x8();
        if (kpart) {
          av = ld_f16x8(&Ut[16 * cb + l16][32 * kk + 8 * g4]);
          bv = ld_f16x8(&Ph[16 * rb + l16][32 * kk + 8 * g4]);
        }
        o = mfma_f16(av, bv, o);
      }
      const int r = 16 * rb + l16;
      if (r < Cr) *(f32x4*)(S.out + ((long)(t0 + r) * Hv + h) * DV + i0 + 16 * cb + 4 * g4) = o;
    }
#pragma unroll
    for (int j = 0; j < NSW; ++j) {
      const int b = wave + NW * j;
      if (b >= NSB) continue;
      const int db = b / NCB, cb = b % NCB;
      f32x4 sacc = st[j] * g_last;
#pragma unroll
      for (int kk = 0; kk < (C + 31) / 32; ++kk) {
        f16x8 av = zero_f16x8(), bv = zero_f16x8();
        if (kpart) {
          av = ld_f16x8(&Kdt[16 * db + l16][32 * kk + 8 * g4]);
          bv = ld_f16x8(&Ut[16 * cb + l16][32 * kk + 8 * g4]);
        }
        sacc = mfma_f16(av, bv, sacc);
      }
      st[j] = sacc;
      big = fmaxf(big, max_abs4(sacc));
      // every read of Sh for this chunk happened before the barrier above
      f16x4 hv = {(_Float16)sacc[0], (_Float16)sacc[1], (_Float16)sacc[2], (_Float16)sacc[3]};
      *(f16x4*)&Sh[16 * cb + l16][16 * db + 4 * g4] = hv;
    }
    lds_barrier();   // staged tiles, U^T and S are free for the next chunk
  }
#pragma unroll
  for (int j = 0; j < NSW; ++j) {
    const int b = wave + NW * j;
    if (b >= NSB) continue;
    const int db = b / NCB, cb = b % NCB;
    *(f32x4*)(Sg + (long)(i0 + 16 * cb + l16) * DK + 16 * db + 4 * g4) = st[j];
  }
  if (big > kF16Max) status_raise(a.status, kFaultRange);
}

static_assert(sizeof(DeltaArgs) <= kMaxKernargBytes, "delta launch record");

template <int DK, int C>
hipError_t prep_for(const DeltaArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_delta_prep<DK, C>), dim3(a.total_chunks * a.n_v_heads), dim3(kPrepThreads), 0, s, a);
  return hipGetLastError();
}

template <int DK, int C>
hipError_t chain_for(const DeltaArgs& a, hipStream_t s) {
  const int blocks = (a.n_seq * a.n_v_heads * a.n_slices + 7) & ~7;   // XCD remap needs a multiple of 8
  const int dvs = DK / a.n_slices;
  if (dvs == 32)
    hipLaunchKernelGGL((k_delta_chain<DK, C, 32>), dim3(blocks), dim3(kChainThreads), 0, s, a);
  else if (dvs == 64)
    hipLaunchKernelGGL((k_delta_chain<DK, C, 64>), dim3(blocks), dim3(kChainThreads), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_delta_prep(const DeltaArgs& a, int d, int chunk, hipStream_t s) {
  if (a.total_chunks <= 0) return hipSuccess;
  if (d == 128 && chunk == 64) return prep_for<128, 64>(a, s);
  if (d == 128 && chunk == 32) return prep_for<128, 32>(a, s);
  if (d == 128 && chunk == 16) return prep_for<128, 16>(a, s);
  if (d == 64 && chunk == 64) return prep_for<64, 64>(a, s);
  if (d == 64 && chunk == 32) return prep_for<64, 32>(a, s);
  if (d == 64 && chunk == 16) return prep_for<64, 16>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_delta_chain(const DeltaArgs& a, int d, int chunk, hipStream_t s) {
  if (a.total_chunks <= 0) return hipSuccess;
  if (d == 128 && chunk == 64) return chain_for<128, 64>(a, s);
  if (d == 128 && chunk == 32) return chain_for<128, 32>(a, s);
  if (d == 128 && chunk == 16) return chain_for<128, 16>(a, s);
  if (d == 64 && chunk == 64) return chain_for<64, 64>(a, s);
  if (d == 64 && chunk == 32) return chain_for<64, 32>(a, s);
  if (d == 64 && chunk == 16) return chain_for<64, 16>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace tu
