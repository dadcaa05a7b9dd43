// Gated delta-rule continuation (paper Section 4.1, Eq. 3: the recurrent state
// continues from its previous value over the replacement tokens; the layers are
// Gated DeltaNet layers, Yang et al. 2025). Per value head the state S (d_v x d_k)
// follows
//     S_t = g_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,   o_t = scale S_t q_t.
//
// The tail is cut into chunks of C tokens starting at its first token. Inside a
// chunk (rows r, i), with lg_r = sum_{s<=r} log2 g_s and G[r][i] = 2^(lg_r - lg_i):
//     M = strictly-lower(diag(beta) (G .* K K^T)),   T = (I + M)^-1
//     W = T diag(beta 2^lg) K,   T_v = T diag(beta),   P = scale lower(G .* Q K^T)
//                                                                       (k_delta_prep)
//     U = T_v V - W S^T
//     O = scale diag(2^lg) Q S^T + P U
//     S <- 2^lg_last S + U^T diag(2^(lg_last - lg)) K                      (k_delta_chain)
// (W and T_v V are the WY factors of the chunk.) Only decay ratios <= 1 are formed. A
// ragged last chunk is padded with k = q = v = 0, beta = 0, g = 1, which leaves the
// recurrence unchanged.
//
// k_delta_prep: one workgroup per (chunk, value head), all chunks in parallel: the
//   work of a chunk that does not depend on the state. K K^T and Q K^T on
//   v_mfma_f32_16x16x32_bf16 (exact bf16 products, fp32 sums); T by blocked forward
//   substitution in fp32 (16x16 diagonal blocks by one lane per column, then
//   off-diagonal blocks level by level); W on v_mfma_f32_16x16x32_f16. Writes W, T_v
//   and P (f16) and the decay factors 2^(lg_last - lg) and 2^lg (fp32) to the
//   workspace, and, once per key head, q and k^T in f16; W, P, q and k^T with their
//   contracted index in the chain's operand order (below).
// k_delta_chain: one workgroup per (context, value head, slice of DVS rows of S); rows
//   of S evolve independently (row i only needs U[:, i]). Each 16 rows of the slice
//   belong to one "owner" wave that keeps them, fp32, in MFMA accumulators for the
//   whole tail (read from HBM once, written once). An accumulator lane holds 4
//   consecutive rows of one column of a 16x16 block; two such blocks side by side
//   supply the 8 values one lane feeds to a 16x16x32 product, when the contracted
//   index runs through each group of 32 in the order perm32 below. So S (as f16), U
//   and its decayed copy serve as MFMA operands straight from registers, and the
//   state step of a chunk needs no LDS round trip and no barrier. The other waves
//   ("producers") stage the next chunk's operands into the second of two LDS buffers:
//   q, k^T, W, P, T_v and the decay factors as the prep wrote them, and the v slice
//   transposed to f16 (with two or four owners, the owners copy P and T_v, or W, P and
//   T_v, themselves once their products are issued). One barrier per chunk. f16 (10 stored mantissa bits) keeps the operands of
//   these fp32-intermediate products accurate enough for the error bound where bf16
//   would not; bf16 inputs convert to f16 exactly inside its range.
#include "common.h"

namespace tu {

namespace {


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

// Position of index x inside its group of 32 in the chain's operand order: the group
// of 4 a = x / 4 goes to 8 (a % 4) + 4 (a / 4), so that lane group g reads indices
// 4g .. 4g + 3 and 16 + 4g .. 16 + 4g + 3 as 8 contiguous values.
__device__ __forceinline__ int perm32(int x) {
  const int a = (x >> 2) & 7;
  return (x & ~31) | (8 * (a & 3) + 4 * (a >> 2) + (x & 3));
}

// The last sequence whose first chunk is at or before c (chunk_begin is non-decreasing
// and starts at 0): a binary search, about log2(n_seq) dependent loads.
__device__ __forceinline__ int find_seq_by_chunk(const DeltaArgs& a, int c) {
  int lo = 0, hi = a.n_seq - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.seq[mid].chunk_begin <= c) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

constexpr int cmax(size_t x, size_t y) { return (int)(x > y ? x : y); }

// Lower-block-triangular C x C fp32 matrix (M, then T): 16x16 blocks (bi, bj), bj <= bi,
// stored one after another with rows of 20 floats
constexpr int kTriPitch = 20;
__device__ __forceinline__ int tri(int r, int c) {
  const int bi = r >> 4, bj = c >> 4;
  return ((bi * (bi + 1) / 2 + bj) * 16 + (r & 15)) * kTriPitch + (c & 15);
}

// ------------------------------------------------------------------ prep
constexpr int kPrepThreads = 512;   // 8 waves
template <int DK, int C>
__global__ __launch_bounds__(kPrepThreads) void k_delta_prep(DeltaArgs a) {
  constexpr int NT = kPrepThreads;
  constexpr int NW = NT / 64;
  constexpr int NB = C / 16;     // 16-row blocks of the chunk
  constexpr int KP = DK + 8;     // pitch of [C][DK] bf16 tiles
  constexpr int CT = C + 8;      // pitch of f16 tiles with the chunk index contiguous
  constexpr int CC = C < 32 ? 32 : C;   // row length of P in the workspace (padded)
  constexpr int TRI = NB * (NB + 1) / 2 * 16 * kTriPitch;   // floats of a lower-block-triangular matrix
  // Three regions whose arrays have disjoint lifetimes (barriers separate the last reads
  // of one from the first writes of the next), 48 KB at C = 64, d = 128, so that three
  // workgroups fit a CU: k rows (phases 0-1), M (2-4), k^T in f16 (5-6); q rows (0-1),
  // T (3-5); T diag(beta 2^lg) in f16 (5-6).
  constexpr int RA = cmax(cmax(sizeof(bf16_t) * C * KP, sizeof(float) * TRI), sizeof(_Float16) * DK * CT);
  constexpr int RB = cmax(sizeof(bf16_t) * C * KP, sizeof(float) * TRI);
  __shared__ __attribute__((aligned(16))) char ra[RA];
  __shared__ __attribute__((aligned(16))) char rb_[RB];
  __shared__ __attribute__((aligned(16))) _Float16 Twh[C][CT];
  __shared__ __attribute__((aligned(16))) float Xs[3][16][20];
  __shared__ __attribute__((aligned(16))) float lg[C];
  __shared__ __attribute__((aligned(16))) float bt[C];
  auto& Ks = *reinterpret_cast<bf16_t(*)[C][KP]>(ra);
  float* Mt = reinterpret_cast<float*>(ra);
  auto& Kt = *reinterpret_cast<_Float16(*)[DK][CT]>(ra);
  auto& Qs = *reinterpret_cast<bf16_t(*)[C][KP]>(rb_);
  float* Tt = reinterpret_cast<float*>(rb_);

  const int Hk = a.n_k_heads, Hv = a.n_v_heads;
  // work item (chunk, value head); consecutive items, and so the value heads that share
  // a key head's q and k, run on one XCD and share its L2
  const int item = xcd_remap(blockIdx.x, gridDim.x);
  if (item >= a.total_chunks * Hv) return;
  const int c = item / Hv;                // global chunk
  const int h = item - c * Hv;            // value head
  const int si = find_seq_by_chunk(a, c);
  const DeltaSeq S = a.seq[si];
  const int t0 = (c - S.chunk_begin) * C;
  const int Cr = min(C, S.T - t0);
  const int kh = h / (Hv / Hk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g4 = lane >> 4;
  float big = 0.f;   // largest magnitude this thread rounds to f16
  status_mark(a.status);

  // ---- phase 0: stage K, Q (bf16), beta, log2 g. Every load is issued before the first
  // LDS write; rows past the chunk's end load its last row (Cr >= 1) and are stored as 0.
  {
    constexpr int NE = C * (DK / 8);
    constexpr int PER = (NE + NT - 1) / NT;
    u32x4 kw[PER], qw[PER];
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = min(tid + p * NT, NE - 1);
      const int r = min(e / (DK / 8), Cr - 1);
      const long off = ((long)(t0 + r) * Hk + kh) * DK + (e % (DK / 8)) * 8;
      kw[p] = *(const u32x4*)(S.k + off);
      qw[p] = *(const u32x4*)(S.q + off);
    }
    const long tr = (long)(t0 + min(tid, Cr - 1)) * Hv + h;
    const float bv = tid < C ? S.beta[tr] : 0.f;
    const float gv = tid < C ? S.g[tr] : 1.f;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = tid + p * NT;
      if (NE % NT == 0 || e < NE) {
        const int r = e / (DK / 8), cc = e - r * (DK / 8);
        const u32x4 z = {0, 0, 0, 0};
        *(u32x4*)&Ks[r][cc * 8] = r < Cr ? kw[p] : z;
        *(u32x4*)&Qs[r][cc * 8] = r < Cr ? qw[p] : z;
      }
    }
    if (tid < C) {
      const bool ok = tid < Cr;
      bt[tid] = ok ? bv : 0.f;
      // log2 g, held at -100 or above: a gate of exactly 0 would give -inf and, in the
      // differences of the cumulative sums below, NaN; 2^-100 of the state is far below
      // fp32 rounding of any other term
      lg[tid] = ok ? fmaxf(__log2f(gv), -100.f) : 0.f;
    }
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
  _Float16* Pg = a.ws_p + slot * C * CC;
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
      *(f16x4*)&Pg[r * CC + perm32(i0)] = pv;
    } else {
      const float br = bt[r];
      f32x4 mv;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        mv[e] = i0 + e < r ? br * __builtin_amdgcn_exp2f(fminf(lr - li4[e], 0.f)) * acc[j][e] : 0.f;
      *(f32x4*)&Mt[tri(r, i0)] = mv;
    }
  }
  // q in f16 for the chain, d in its operand order, written by the first value head of
  // each key head (k^T by the last): output vector v8 of a row holds the natural
  // d0 .. d0 + 3 and d0 + 16 .. d0 + 19 of its group of 32 (the inverse of perm32)
  const int G = Hv / Hk;
  if (h % G == 0) {
    _Float16* Qg = a.ws_q + ((long)c * Hk + kh) * C * DK;
    for (int e = tid; e < C * (DK / 8); e += NT) {
      const int r = e / (DK / 8), v8 = e - r * (DK / 8);
      const int d0 = 32 * (v8 >> 2) + 4 * (v8 & 3);
      const uint2 w[2] = {*(const uint2*)&Qs[r][d0], *(const uint2*)&Qs[r][d0 + 16]};
      f16x8 hq;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t wq = w[q >> 1][q & 1];
        const float x0 = __uint_as_float(wq << 16), x1 = __uint_as_float(wq & 0xFFFF0000u);
        big = fmaxf(big, fmaxf(fabsf(x0), fabsf(x1)));
        hq[2 * q] = (_Float16)x0;
        hq[2 * q + 1] = (_Float16)x1;
      }
      *(f16x8*)&Qg[r * DK + 8 * v8] = hq;
    }
  }
  // zero the upper blocks of P and the padding of its rows
  for (int e = tid; e < C * CC / 4; e += NT) {
    const int r = e / (CC / 4), i = (e - r * (CC / 4)) * 4;
    if (i >= C || (i >> 4) > (r >> 4)) *(uint2*)&Pg[r * CC + perm32(i)] = uint2{0, 0};
  }
  // the chain's decay factors: to the chunk's end, and from its start
  if (tid < C) {
    a.ws_dec[(2 * slot) * C + tid] = __builtin_amdgcn_exp2f(lg[C - 1] - lg[tid]);
    a.ws_dec[(2 * slot + 1) * C + tid] = __builtin_amdgcn_exp2f(lg[tid]);
  }
  lds_barrier();

  // ---- phase 3: diagonal 16x16 blocks of T = (I + M)^-1, one lane per column: forward
  // substitution, with the next row of M read while the current one is summed
  if (wave == 0 && g4 < NB) {
    const int b = g4, cc = l16;
    const float* Mrow = &Mt[tri(16 * b, 16 * b)];
    float x[16];
    f32x4 cur[4], nxt[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) cur[q] = *(const f32x4*)(Mrow + 4 * q);
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      if (rr + 1 < 16) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (4 * q < rr + 1) nxt[q] = *(const f32x4*)(Mrow + (rr + 1) * kTriPitch + 4 * q);
      }
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < rr; ++i) acc[i & 3] += cur[i >> 2][i & 3] * x[i];
      const float sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
      x[rr] = rr < cc ? 0.f : (rr == cc ? 1.f : -sum);
#pragma unroll
      for (int q = 0; q < 4; ++q) cur[q] = nxt[q];
    }
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) Tt[tri(16 * b + rr, 16 * b + cc)] = x[rr];
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
          x = __builtin_amdgcn_mfma_f32_16x16x4f32(Mt[tri(16 * i + l16, 16 * m + 4 * s + g4)],
                                                   Tt[tri(16 * m + 4 * s + g4, 16 * j + l16)], x, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) Xs[wave][4 * g4 + e][l16] = x[e];
      __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));   // this wave's LDS writes are done
      f32x4 y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        y = __builtin_amdgcn_mfma_f32_16x16x4f32(Tt[tri(16 * i + l16, 16 * i + 4 * s + g4)], Xs[wave][4 * s + g4][l16],
                                                 y, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) Tt[tri(16 * i + 4 * g4 + e, 16 * j + l16)] = -y[e];
    }
    lds_barrier();
  }

  // ---- phase 5: T diag(beta 2^lg) (f16, LDS) and T_v = T diag(beta) (f16, workspace),
  // zero above the diagonal blocks (whose entries of T were never written); k^T in f16
  _Float16* Tvg = a.ws_tv + slot * C * C;
  for (int e = tid; e < C * C / 4; e += NT) {
    const int r = e / (C / 4), i0 = (e - r * (C / 4)) * 4;
    f16x4 hw, hv;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + q;
      const float x = (i >> 4) <= (r >> 4) ? Tt[tri(r, (i >> 4) <= (r >> 4) ? i : 0)] : 0.f;
      const float xw = x * (bt[i] * __builtin_amdgcn_exp2f(lg[i])), xv = x * bt[i];
      big = fmaxf(big, fmaxf(fabsf(xw), fabsf(xv)));
      hw[q] = (_Float16)xw;
      hv[q] = (_Float16)xv;
    }
    *(f16x4*)&Twh[r][i0] = hw;
    *(f16x4*)&Tvg[r * C + i0] = hv;
  }
  // k^T in f16 over the dead M, from the k rows read again (from L2: phase 0 read them)
  for (int e = tid; e < (C / 2) * (DK / 8); e += NT) {
    const int s2 = (e % (C / 2)) * 2, d0 = (e / (C / 2)) * 8;
    const u32x4 z4 = {0, 0, 0, 0};
    const u32x4 k0 = s2 < Cr ? *(const u32x4*)(S.k + ((long)(t0 + s2) * Hk + kh) * DK + d0) : z4;
    const u32x4 k1 = s2 + 1 < Cr ? *(const u32x4*)(S.k + ((long)(t0 + s2 + 1) * Hk + kh) * DK + d0) : z4;
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const uint32_t b0 = (d & 1) ? (k0[d >> 1] & 0xFFFF0000u) : (k0[d >> 1] << 16);
      const uint32_t b1 = (d & 1) ? (k1[d >> 1] & 0xFFFF0000u) : (k1[d >> 1] << 16);
      const float x0 = __uint_as_float(b0), x1 = __uint_as_float(b1);
      big = fmaxf(big, fmaxf(fabsf(x0), fabsf(x1)));
      const f16x2 hk = {(_Float16)x0, (_Float16)x1};
      *(f16x2*)&Kt[d0 + d][s2] = hk;
    }
  }
  lds_barrier();

  // ---- phase 6: W = T diag(beta 2^lg) K on MFMA, to the workspace with d in the
  // chain's operand order; k^T (last value head of each key head) with s in that order,
  // its chunk index padded with zeros to a whole MFMA step
  if (h % G == G - 1) {
    _Float16* Kg = a.ws_kt + ((long)c * Hk + kh) * DK * CC;
    for (int e = tid; e < DK * (CC / 8); e += NT) {
      const int d = e / (CC / 8), v8 = e - d * (CC / 8);
      const int s0 = 32 * (v8 >> 2) + 4 * (v8 & 3);
      const uint2 z2 = {0, 0};
      const uint2 lo = s0 < C ? *(const uint2*)&Kt[d][s0] : z2;
      const uint2 hi = s0 + 16 < C ? *(const uint2*)&Kt[d][s0 + 16] : z2;
      *(u32x4*)&Kg[d * CC + 8 * v8] = u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
  }
  _Float16* Wg = a.ws_w + slot * C * DK;
  constexpr int NOB = NB * (DK / 16);
  for (int idx = wave; idx < NOB; idx += NW) {
    const int rb = idx / (DK / 16), db = idx % (DK / 16);
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    // transposed product (K^T W'^T): the lane ends up with row 16 rb + l16 and the 4
    // consecutive columns 16 db + 4 g4 .. of W
#pragma unroll
    for (int kk = 0; kk < (C + 31) / 32; ++kk) {
      f16x8 av = zero_f16x8(), bv = zero_f16x8();
      if (C >= 32 || g4 < 2) {
        av = ld_f16x8(&Kt[16 * db + l16][32 * kk + 8 * g4]);
        bv = ld_f16x8(&Twh[16 * rb + l16][32 * kk + 8 * g4]);
      }
      o = mfma_f16(av, bv, o);
    }
    big = fmaxf(big, max_abs4(o));
    const f16x4 wv = {(_Float16)o[0], (_Float16)o[1], (_Float16)o[2], (_Float16)o[3]};
    *(f16x4*)&Wg[(16 * rb + l16) * DK + perm32(16 * db + 4 * g4)] = wv;
  }
  if (big > kF16Max) status_raise(a.status, kFaultRange);
}

// ------------------------------------------------------------------ chain
constexpr int kChainThreads = 512;   // 8 waves: DVS / 16 owners, the rest producers

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One chunk's operands in LDS (two of these alternate)
template <int DK, int C, int DVS>
struct ChainStage {
  static constexpr int KP = DK + 8;                  // pitch of rows over d
  static constexpr int CC = C < 32 ? 32 : C;         // chunk index padded to a whole MFMA step
  static constexpr int CK = CC + 8;                  // pitch of rows over the chunk index
  _Float16 W[C][KP];      // W, d in operand order
  _Float16 Q[C][KP];      // q in f16, d in operand order
  _Float16 Kt[DK][CK];    // k^T in f16, s in operand order
  _Float16 P[C][CK];      // P, s in operand order
  _Float16 Tv[C][CK];     // T_v, natural order
  _Float16 Vt[DVS][CK];   // the v slice transposed, natural order
  float dec[2][C];        // 2^(lg_last - lg_s), 2^lg_s
};

template <int DK, int C, int DVS>
__global__ __launch_bounds__(kChainThreads) void k_delta_chain(DeltaArgs a) {
  using Stage = ChainStage<DK, C, DVS>;
  constexpr int NT = kChainThreads;
  constexpr int DV = DK;
  constexpr int CC = Stage::CC;
  constexpr int NO = DVS / 16;                  // owner waves
  constexpr int NP = NT - 64 * NO;              // producer threads
  static_assert(NP >= 2 * C, "one decay factor per producer thread");
  constexpr int NRB = C / 16;                   // 16-row blocks of a chunk
  constexpr int NDB = DK / 16;                  // 16-row blocks of S^T
  constexpr int NKD = DK / 32;                  // MFMA steps over d
  constexpr int NKS = CC / 32;                  // MFMA steps over the chunk index
  // producer work per chunk: 16-byte vectors of q, k^T, W, P, T_v (copied as the prep
  // wrote them); 2-row x 8-column items of the v slice (converted and transposed)
  constexpr int VQ = C * DK / 8, VK = DK * CC / 8, VW = C * DK / 8, VP = C * CC / 8, VT = C * C / 8;
  constexpr int NVI = (C / 2) * (DVS / 8);
  // The owners finish their part of a chunk first, so with four owners they copy W, P
  // and T_v of the next chunk (loads issued before their products, stores after), with
  // two P and T_v; the producers copy the rest.
  constexpr bool OW = NO >= 4, OPT = NO >= 2;
  constexpr int NOT = 64 * NO;                  // owner threads
  constexpr int RQ = (VQ + NP - 1) / NP, RK = (VK + NP - 1) / NP, RV = (NVI + NP - 1) / NP;
  constexpr int RW = OW ? (VW + NOT - 1) / NOT : (VW + NP - 1) / NP;
  constexpr int RP = OPT ? (VP + NOT - 1) / NOT : (VP + NP - 1) / NP;
  constexpr int RT = OPT ? (VT + NOT - 1) / NOT : (VT + NP - 1) / NP;
  __shared__ __attribute__((aligned(16))) Stage stg[2];

  // work item: (context, key head, value head of the group, slice), ordered so that the
  // workgroups reading one key head's q and k share an XCD
  const int Hv = a.n_v_heads, Hk = a.n_k_heads, G = Hv / Hk;
  const int item = xcd_remap(blockIdx.x, gridDim.x);
  const int per_seq = Hv * a.n_slices;
  const int si = item / per_seq;
  if (si >= a.n_seq) return;
  const int rem = item - si * per_seq;
  const int kh = rem / (G * a.n_slices);
  const int rem2 = rem - kh * G * a.n_slices;
  const int h = kh * G + rem2 / a.n_slices;
  const int i0 = (rem2 % a.n_slices) * DVS;
  const DeltaSeq S = a.seq[si];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g4 = lane >> 4;
  const bool owner = wave < NO;
  const int p = tid - 64 * NO;                  // producer thread index
  float big = 0.f;   // largest magnitude this thread rounds to f16

  // chunk-index padding of T_v and the v slice (C = 16 only) stays zero for the whole
  // kernel (k^T comes padded from the workspace)
  if (C < 32) {
    for (int e = tid; e < 2 * (C + DVS) * 16; e += NT) {
      const int b = e / ((C + DVS) * 16), rest = e - b * (C + DVS) * 16;
      const int row = rest / 16, x = C + (rest % 16);
      if (row < C) stg[b].Tv[row][x] = (_Float16)0.f;
      else stg[b].Vt[row - C][x] = (_Float16)0.f;
    }
  }

  // ---- producers: registers of one chunk, then their conversion into a stage
  const u32x4 z4 = {0, 0, 0, 0};
  u32x4 rq[RQ], rw[RW], rp[RP], rt[RT], rk[RK], rv[RV][2];
  float rdec = 0.f;   // one of the chunk's 2C decay factors
  // W, and P and T_v, of chunk lc by thread x of the n that copy them
  auto fetch_w = [&](int lc, int x, int n) {
    const u32x4* W4 = (const u32x4*)(a.ws_w + ((long)(S.chunk_begin + lc) * Hv + h) * C * DK);
#pragma unroll
    for (int j = 0; j < RW; ++j) rw[j] = x + n * j < VW ? W4[x + n * j] : z4;
  };
  auto fetch_pt = [&](int lc, int x, int n) {
    const long slot = (long)(S.chunk_begin + lc) * Hv + h;
    const u32x4* P4 = (const u32x4*)(a.ws_p + slot * C * CC);
    const u32x4* T4 = (const u32x4*)(a.ws_tv + slot * C * C);
#pragma unroll
    for (int j = 0; j < RP; ++j) rp[j] = x + n * j < VP ? P4[x + n * j] : z4;
#pragma unroll
    for (int j = 0; j < RT; ++j) rt[j] = x + n * j < VT ? T4[x + n * j] : z4;
  };
  auto put_w = [&](Stage& B, int x, int n) {
#pragma unroll
    for (int j = 0; j < RW; ++j) {
      const int e = x + n * j;
      if (e < VW) *(u32x4*)&B.W[e / (DK / 8)][8 * (e % (DK / 8))] = rw[j];
    }
  };
  auto put_pt = [&](Stage& B, int x, int n) {
#pragma unroll
    for (int j = 0; j < RP; ++j) {
      const int e = x + n * j;
      if (e < VP) *(u32x4*)&B.P[e / (CC / 8)][8 * (e % (CC / 8))] = rp[j];
    }
#pragma unroll
    for (int j = 0; j < RT; ++j) {
      const int e = x + n * j;
      if (e < VT) *(u32x4*)&B.Tv[e / (C / 8)][8 * (e % (C / 8))] = rt[j];
    }
  };
  auto fetch = [&](int lc) {
    const int t0 = lc * C;
    const int Cr = min(C, S.T - t0);
    const long slot = (long)(S.chunk_begin + lc) * Hv + h;
    const long slot_k = (long)(S.chunk_begin + lc) * Hk + kh;
    const u32x4* Q4 = (const u32x4*)(a.ws_q + slot_k * C * DK);
    const u32x4* K4 = (const u32x4*)(a.ws_kt + slot_k * DK * CC);
#pragma unroll
    for (int j = 0; j < RQ; ++j) rq[j] = p + NP * j < VQ ? Q4[p + NP * j] : z4;
#pragma unroll
    for (int j = 0; j < RK; ++j) rk[j] = p + NP * j < VK ? K4[p + NP * j] : z4;
#pragma unroll
    for (int j = 0; j < RV; ++j) {
      const int e = p + NP * j;
      const int s2 = (e % (C / 2)) * 2, d0 = (e / (C / 2)) * 8;
#pragma unroll
      for (int q = 0; q < 2; ++q)
        rv[j][q] = (e < NVI && s2 + q < Cr) ? *(const u32x4*)(S.v + ((long)(t0 + s2 + q) * Hv + h) * DV + i0 + d0) : z4;
    }
    if (!OW) fetch_w(lc, p, NP);
    if (!OPT) fetch_pt(lc, p, NP);
    if (p < 2 * C) rdec = a.ws_dec[2 * slot * C + p];
  };
  auto put = [&](Stage& B) {
#pragma unroll
    for (int j = 0; j < RQ; ++j) {
      const int e = p + NP * j;
      if (e < VQ) *(u32x4*)&B.Q[e / (DK / 8)][8 * (e % (DK / 8))] = rq[j];
    }
#pragma unroll
    for (int j = 0; j < RK; ++j) {
      const int e = p + NP * j;
      if (e < VK) *(u32x4*)&B.Kt[e / (CC / 8)][8 * (e % (CC / 8))] = rk[j];
    }
#pragma unroll
    for (int j = 0; j < RV; ++j) {
      const int e = p + NP * j;
      if (e < NVI) {
        const int s2 = (e % (C / 2)) * 2, d0 = (e / (C / 2)) * 8;
#pragma unroll
        for (int d = 0; d < 8; ++d) {
          const float x0 = (d & 1) ? bf16_hi(rv[j][0][d >> 1]) : bf16_lo(rv[j][0][d >> 1]);
          const float x1 = (d & 1) ? bf16_hi(rv[j][1][d >> 1]) : bf16_lo(rv[j][1][d >> 1]);
          big = fmaxf(big, fmaxf(fabsf(x0), fabsf(x1)));
          const f16x2 hx = {(_Float16)x0, (_Float16)x1};
          *(f16x2*)&B.Vt[d0 + d][s2] = hx;
        }
      }
    }
    if (!OW) put_w(B, p, NP);
    if (!OPT) put_pt(B, p, NP);
    if (p < 2 * C) B.dec[p / C][p % C] = rdec;
  };

  // ---- owners: S^T rows 16 db + 4 g4 + e, column 16 wave + l16 of the slice, in
  // accumulators; their negated f16 copy as operands over d (blocks 2 kk and 2 kk + 1),
  // so that -W S^T accumulates onto T_v V in place
  float* Sg = S.state + (long)h * DV * DK + (long)(i0 + 16 * wave + l16) * DK;
  f32x4 st[NDB];
  f16x8 sh[NKD];
  auto refresh_sh = [&]() {
#pragma unroll
    for (int kk = 0; kk < NKD; ++kk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sh[kk][e] = (_Float16)(-st[2 * kk][e]);
        sh[kk][4 + e] = (_Float16)(-st[2 * kk + 1][e]);
      }
      big = fmaxf(big, fmaxf(max_abs4(st[2 * kk]), max_abs4(st[2 * kk + 1])));
    }
  };
  if (owner) {
    if (OW) fetch_w(0, tid, NOT);
    if (OPT) fetch_pt(0, tid, NOT);
#pragma unroll
    for (int db = 0; db < NDB; ++db) st[db] = *(const f32x4*)(Sg + 16 * db + 4 * g4);
    refresh_sh();
    if (OW) put_w(stg[0], tid, NOT);
    if (OPT) put_pt(stg[0], tid, NOT);
  } else {
    fetch(0);
    put(stg[0]);
    if (S.n_chunks > 1) fetch(1);
  }
  lds_barrier();

  for (int lc = 0; lc < S.n_chunks; ++lc) {
    if (owner) {
      const bool next = lc + 1 < S.n_chunks;
      if (OW && next) fetch_w(lc + 1, tid, NOT);
      if (OPT && next) fetch_pt(lc + 1, tid, NOT);
      const Stage& B = stg[lc & 1];
      const int t0 = lc * C;
      const int Cr = min(C, S.T - t0);
      // -Y^T = (-S) Q^T (columns 16 wave + 4 g4 .., row 16 rb + l16) and
      // U = T_v V + W (-S)^T (rows 16 rb + 4 g4 .., column 16 wave + l16)
      f32x4 y[NRB], u[NRB];
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) y[rb] = u[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < NKS; ++kk)
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
          u[rb] = mfma_f16(ld_f16x8(&B.Tv[16 * rb + l16][32 * kk + 8 * g4]),
                           ld_f16x8(&B.Vt[16 * wave + l16][32 * kk + 8 * g4]), u[rb]);
#pragma unroll
      for (int kk = 0; kk < NKD; ++kk)
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
          y[rb] = mfma_f16(sh[kk], ld_f16x8(&B.Q[16 * rb + l16][32 * kk + 8 * g4]), y[rb]);
          u[rb] = mfma_f16(ld_f16x8(&B.W[16 * rb + l16][32 * kk + 8 * g4]), sh[kk], u[rb]);
        }
      // U and its decayed copy, as operands over the chunk index
      f16x8 uh[NKS], ud[NKS];
#pragma unroll
      for (int kk = 0; kk < NKS; ++kk) uh[kk] = ud[kk] = zero_f16x8();
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float uu = u[rb][e];
          const float dd = B.dec[0][16 * rb + 4 * g4 + e] * uu;
          big = fmaxf(big, fabsf(uu));
          uh[rb >> 1][4 * (rb & 1) + e] = (_Float16)uu;
          ud[rb >> 1][4 * (rb & 1) + e] = (_Float16)dd;
        }
      // O^T = scale 2^lg Y^T + U^T P^T, written out
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        y[rb] = y[rb] * (-a.scale * B.dec[1][16 * rb + l16]);
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk) y[rb] = mfma_f16(uh[kk], ld_f16x8(&B.P[16 * rb + l16][32 * kk + 8 * g4]), y[rb]);
        const int r = 16 * rb + l16;
        if (r < Cr) *(f32x4*)(S.out + ((long)(t0 + r) * Hv + h) * DV + i0 + 16 * wave + 4 * g4) = y[rb];
      }
      // S^T <- 2^lg_last S^T + K^T (decayed U)
      const float g_last = B.dec[1][C - 1];
#pragma unroll
      for (int db = 0; db < NDB; ++db) st[db] = st[db] * g_last;
#pragma unroll
      for (int kk = 0; kk < NKS; ++kk)
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          st[db] = mfma_f16(ld_f16x8(&B.Kt[16 * db + l16][32 * kk + 8 * g4]), ud[kk], st[db]);
      refresh_sh();
      if (OW && next) put_w(stg[(lc + 1) & 1], tid, NOT);
      if (OPT && next) put_pt(stg[(lc + 1) & 1], tid, NOT);
    } else if (lc + 1 < S.n_chunks) {
      put(stg[(lc + 1) & 1]);
      if (lc + 2 < S.n_chunks) fetch(lc + 2);
    }
    lds_barrier();   // the next stage is complete; this one may be refilled
  }
  if (owner) {
#pragma unroll
    for (int db = 0; db < NDB; ++db) *(f32x4*)(Sg + 16 * db + 4 * g4) = st[db];
  }
  if (big > kF16Max) status_raise(a.status, kFaultRange);
}

static_assert(sizeof(DeltaArgs) <= kMaxKernargBytes, "delta launch record");

template <int DK, int C>
hipError_t prep_for(const DeltaArgs& a, hipStream_t s) {
  const int blocks = (a.total_chunks * a.n_v_heads + 7) & ~7;   // xcd_remap wants a multiple of 8
  hipLaunchKernelGGL((k_delta_prep<DK, C>), dim3(blocks), dim3(kPrepThreads), 0, s, a);
  return hipGetLastError();
}

template <int DK, int C>
hipError_t chain_for(const DeltaArgs& a, hipStream_t s) {
  const int blocks = (a.n_seq * a.n_v_heads * a.n_slices + 7) & ~7;   // xcd_remap wants a multiple of 8
  const int dvs = DK / a.n_slices;
  if (dvs == 16)
    hipLaunchKernelGGL((k_delta_chain<DK, C, 16>), dim3(blocks), dim3(kChainThreads), 0, s, a);
  else if (dvs == 32)
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
