// Short causal convolution continued from its carried state (paper Section 4.1 and
// Fig. 2: the recurrent layers' convolution state continues over the replacement
// tokens without rollback). Per channel c of a projected tensor x [T][C]:
//     y_t[c] = act( sum_{j<W} w[c][j] * xt[t + j][c] ),   xt = (W-1 carried rows, then x)
// act = SiLU or identity; the carried state becomes the last W-1 rows of xt.
//
// One thread per 8 channels (16-byte loads and stores) and a block of kConvTokens
// tokens: it requests the block's rows and the W-1 rows before it all at once (one
// memory round trip), then forms each output from a window of W rows in registers. Products are accumulated in
// fp32 in tap order and rounded to bf16 (round to nearest even). Only the first
// token block of a channel group touches the state: it reads the old rows, keeps
// them, and writes the new rows after its own reads, so the update is in place
// without any other block depending on it.
#include "common.h"

namespace tu {

namespace {

constexpr int kConvThreads = 256;
constexpr int kConvTokens = 8;    // tokens per block (>= W - 1, so only block 0 reads the state)

__device__ __forceinline__ void unpack8(u32x4 w, float (&f)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = bf16_to_f32(w[e] & 0xFFFFu);
    f[2 * e + 1] = bf16_to_f32(w[e] >> 16);
  }
}

template <int W>
__global__ __launch_bounds__(kConvThreads) void k_short_conv(ConvArgs a) {
  int ji = 0;
  while (ji + 1 < a.n_jobs && a.job[ji + 1].block_begin <= (int)blockIdx.x) ++ji;
  const ConvJob& J = a.job[ji];
  const int local = blockIdx.x - J.block_begin;
  const int tb = local / J.n_cblocks;                        // token block
  const int cg = (local - tb * J.n_cblocks) * kConvThreads + threadIdx.x;   // 8-channel group
  if (8 * cg >= J.C) return;
  const int C = J.C;
  const int t0 = tb * kConvTokens;
  const int t1 = min(J.T, t0 + kConvTokens);

  float wf[W][8];
  {
    const u32x4* wp = (const u32x4*)(J.w + (long)8 * cg * W);   // taps of 8 channels: 8W bf16
    float tmp[8];
#pragma unroll
    for (int q = 0; q < W; ++q) {
      unpack8(wp[q], tmp);
      // vector q holds channels 8cg + (8q + e) / W, taps (8q + e) % W
#pragma unroll
      for (int e = 0; e < 8; ++e) wf[(8 * q + e) % W][(8 * q + e) / W] = tmp[e];
    }
  }
  // rows t0 .. t0 + kConvTokens + W - 2 of xt (this thread's 8 channels), all requested
  // before any is used
  const bf16_t* __restrict__ xs = J.x;
  const bf16_t* __restrict__ ss = J.state;
  constexpr int R = kConvTokens + W - 1;
  u32x4 raw[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = t0 + r;   // row of xt
    if (i < W - 1)
      raw[r] = *(const u32x4*)(ss + (long)i * C + 8 * cg);
    else if (i - (W - 1) < J.T)
      raw[r] = *(const u32x4*)(xs + (long)(i - (W - 1)) * C + 8 * cg);
    else
      raw[r] = u32x4{0, 0, 0, 0};
  }
  u32x4 old[W > 1 ? W - 1 : 1];
#pragma unroll
  for (int r = 0; r < W - 1; ++r) old[r] = raw[r];   // the carried rows when t0 == 0
#pragma unroll
  for (int k = 0; k < kConvTokens; ++k) {
    const int t = t0 + k;
    if (t >= t1) break;
    float win[W][8];
#pragma unroll
    for (int j = 0; j < W; ++j) unpack8(raw[k + j], win[j]);
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < W; ++j) acc = __builtin_fmaf(wf[j][2 * e + h], win[j][2 * e + h], acc);
        if (J.act) acc = acc / (1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * acc));
        v[h] = acc;
      }
      o[e] = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
    }
    *(u32x4*)(J.out + (long)t * C + 8 * cg) = o;
  }
  // the first block writes the new state: rows T .. T + W - 2 of xt
  if (tb == 0) {
#pragma unroll
    for (int r = 0; r < W - 1; ++r) {
      const int i = J.T + r;
      u32x4 v;
      if (i < W - 1) {
#pragma unroll
        for (int q = 0; q < W - 1; ++q)   // old[i] without a runtime index (kept in registers)
          if (q == i) v = old[q];
      } else {
        v = *(const u32x4*)(J.x + (long)(i - (W - 1)) * C + 8 * cg);
      }
      *(u32x4*)(J.state + (long)r * C + 8 * cg) = v;
    }
  }
}

}  // namespace

int conv_blocks(ConvJob& j, int block_begin) {
  j.block_begin = block_begin;
  j.n_cblocks = (j.C / 8 + kConvThreads - 1) / kConvThreads;
  return (int)((j.T + kConvTokens - 1) / kConvTokens) * j.n_cblocks;
}

hipError_t launch_short_conv(const ConvArgs& a, int blocks, int width, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  switch (width) {
    case 1: hipLaunchKernelGGL(k_short_conv<1>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 2: hipLaunchKernelGGL(k_short_conv<2>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 3: hipLaunchKernelGGL(k_short_conv<3>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 4: hipLaunchKernelGGL(k_short_conv<4>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 5: hipLaunchKernelGGL(k_short_conv<5>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 6: hipLaunchKernelGGL(k_short_conv<6>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 7: hipLaunchKernelGGL(k_short_conv<7>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    case 8: hipLaunchKernelGGL(k_short_conv<8>, dim3(blocks), dim3(kConvThreads), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tu
