// Causal grouped-query attention of the tail over the surviving + new KV (paper
// Section 4.1, Eq. 3; Section 4.3: attending to the surviving context is the
// work that remains after unchanged records are no longer recomputed).
//
// Tail row i of query head h attends to cache rows 0 .. L_keep + i of KV head
// h / G (G = Hq / Hkv). The G query heads that share a KV head are packed as
// rows (token-major: packed row = t * G + (h mod G)), so one workgroup tile of
// 128 packed rows reads each K/V tile once for all of them.
//
// Workgroup: 4 waves x 32 packed rows, key tiles of 64 rows staged in LDS.
// The scores are formed transposed, S^T = K Q^T, on v_mfma_f32_32x32x16_bf16:
// A = 32 keys x 16 dims of K (LDS), B = 16 dims x 32 queries of Q (registers).
// A lane's accumulator then holds 16 keys of ONE query (lane % 32), so the
// online-softmax state (running max, running sum) is per lane; the two lanes
// sharing a query (l and l ^ 32) exchange their maxima once per tile. The output
// is accumulated transposed too, O^T += V^T P^T, on v_mfma_f32_32x32x16_f16: V is
// written into LDS transposed ([dim][key]) and converted to f16, and the
// probabilities P (in [0, 1]) are rounded to f16, whose 10 stored mantissa bits
// keep the result within the accuracy bound where bf16's 7 would not. Within each
// 16-key group the LDS key order is permuted so that a lane's 8 keys of a B
// fragment are contiguous (one 16-byte read).
//
// For occupancy the key range of a tile is split over `n_splits` workgroups; each
// writes an unnormalised partial (O, running max, sum) and k_attn_merge combines
// them. Workgroups are ordered (kv head, split, tile) and remapped so that the
// tiles of one (head, split) key range share an XCD and its L2.
#include "common.h"

namespace tu {

namespace {

constexpr int kBM = 128;   // packed query rows per workgroup
constexpr int kBN = 64;    // keys per tile
constexpr int kKPad = 8;   // bf16 padding per K row in LDS
constexpr int kVPad = 8;   // f16 padding per V^T row in LDS
constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units): P < 2^8 fits f16

__device__ __forceinline__ int key_slot(int k) {
  // swap bits 2 and 3 of the key index within its 16-key group
  return (k & ~0xC) | ((k & 4) << 1) | ((k & 8) >> 1);
}

// Scales an MFMA accumulator that lives in AGPRs. Going through explicit AGPR
// reads/writes keeps the accumulator out of the VALU register class, so the
// compiler does not shuttle it between AGPRs and VGPRs on every key tile.
__device__ __forceinline__ void scale_acc(f32x16& acc, float s) {
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    float v;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(acc[e]));
    v *= s;
    asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(acc[e]) : "v"(v));
  }
}

__device__ __forceinline__ _Float16 bf16_lo_to_f16(uint32_t w) { return (_Float16)__uint_as_float(w << 16); }
__device__ __forceinline__ _Float16 bf16_hi_to_f16(uint32_t w) { return (_Float16)__uint_as_float(w & 0xFFFF0000u); }

template <int D>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  constexpr int NS = D / 16;   // 16-dim steps of Q K^T
  constexpr int NDB = D / 32;  // 32-dim blocks of O^T
  __shared__ __attribute__((aligned(16))) bf16_t Ks[kBN][D + kKPad];
  __shared__ __attribute__((aligned(16))) _Float16 Vt[D][kBN + kVPad];

  const int item = xcd_remap(blockIdx.x, gridDim.x);
  if (item >= a.total_items) return;
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].item_begin <= item) ++si;
  const AttnSeq S = a.seq[si];
  int local = item - S.item_begin;
  const int tile = local % S.n_tiles;
  local /= S.n_tiles;
  const int split = local % S.n_splits;
  const int hkv = local / S.n_splits;

  const int Hq = a.n_q_heads;
  const int Hkv = a.n_kv_heads;
  const int G = Hq / Hkv;
  const int rows_total = S.T * G;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int hl = lane >> 5;     // half of the wave
  const int col = lane & 31;    // query column of this lane

  const int r = tile * kBM + wave * 32 + col;
  const bool row_ok = r < rows_total;
  const int t = row_ok ? r / G : S.T - 1;
  const int qh = hkv * G + (row_ok ? r - (r / G) * G : 0);
  const int r_last = min(rows_total, (tile + 1) * kBM) - 1;
  const int t_hi = r_last / G;
  const int t_lo = (tile * kBM) / G;
  const int n_keys = S.L_keep + t_hi + 1;
  const int n_kt = (n_keys + kBN - 1) / kBN;
  const int tps = (n_kt + S.n_splits - 1) / S.n_splits;
  const int kt_begin = split * tps;
  const int kt_end = min(n_kt, kt_begin + tps);
  const int my_limit = S.L_keep + t;  // last key this query may see

  // Q fragments stay in registers for the whole key loop
  bf16x8 qf[NS];
  {
    const bf16_t* qrow = S.q_hat + ((long)t * Hq + qh) * D + 8 * hl;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      u32x4 w = row_ok ? *(const u32x4*)(qrow + 16 * s) : u32x4{0, 0, 0, 0};
      qf[s] = __builtin_bit_cast(bf16x8, w);
    }
  }

  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] = 0.f;
  // Online softmax in the log2 domain with a lazily moved reference max: the
  // probabilities are 2^(s*c - m_run) with m_run raised (and O, l rescaled) only
  // when a tile's max exceeds it by more than kTau, so P stays below 2^kTau.
  float m_run = -__builtin_inff();
  float l_run = 0.f;
  const float c2 = a.scale_log2;

  const long rs = (long)Hkv * D;  // elements per cache row
  const bf16_t* kbase = S.k_cache + (long)hkv * D;
  const bf16_t* vbase = S.v_cache + (long)hkv * D;

  // staging: K rows are copied as 16-byte vectors, V as (4 keys x 8 dims) blocks
  constexpr int KIT = kBN * D / 8 / 256;
  constexpr int KROWS = 256 / (D / 8);
  constexpr int VTASK = (kBN / 4) * (D / 8);
  constexpr int VIT = (VTASK + 255) / 256;
  const int k_kr = threadIdx.x / (D / 8);
  const int k_kc = threadIdx.x % (D / 8);
  u32x4 kreg[KIT];
  u32x4 vreg[VIT][4];

  // per-thread source addresses of the first tile; later tiles add a uniform offset
  const bf16_t* kthr = kbase + (long)k_kr * rs + k_kc * 8;
  const bf16_t* vthr[VIT];
#pragma unroll
  for (int it = 0; it < VIT; ++it) {
    const int c = threadIdx.x + 256 * it;
    vthr[it] = vbase + (long)((c % (kBN / 4)) * 4) * rs + (c / (kBN / 4)) * 8;
  }
  auto load_tile = [&](int kt) {
    const int key0 = kt * kBN;
    const long toff = (long)key0 * rs;
    if (key0 + kBN <= n_keys) {
#pragma unroll
      for (int it = 0; it < KIT; ++it) kreg[it] = *(const u32x4*)(kthr + toff + (long)(KROWS * it) * rs);
#pragma unroll
      for (int it = 0; it < VIT; ++it)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          vreg[it][j] = (threadIdx.x + 256 * it < VTASK) ? *(const u32x4*)(vthr[it] + toff + j * rs)
                                                          : u32x4{0, 0, 0, 0};
    } else {
#pragma unroll
      for (int it = 0; it < KIT; ++it) {
        const int key = key0 + k_kr + KROWS * it;
        kreg[it] = key < n_keys ? *(const u32x4*)(kthr + toff + (long)(KROWS * it) * rs) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int it = 0; it < VIT; ++it) {
        const int c = threadIdx.x + 256 * it;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int key = key0 + (c % (kBN / 4)) * 4 + j;
          vreg[it][j] = (c < VTASK && key < n_keys) ? *(const u32x4*)(vthr[it] + toff + j * rs)
                                                     : u32x4{0, 0, 0, 0};
        }
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int it = 0; it < KIT; ++it) *(u32x4*)&Ks[k_kr + KROWS * it][k_kc * 8] = kreg[it];
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int c = threadIdx.x + 256 * it;
      if (c < VTASK) {
        const int kq = c % (kBN / 4);
        const int dc = c / (kBN / 4);
        const int slot = key_slot(kq * 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          f16x4 h4;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            h4[j] = (e & 1) ? bf16_hi_to_f16(vreg[it][j][e >> 1]) : bf16_lo_to_f16(vreg[it][j][e >> 1]);
          *(f16x4*)&Vt[dc * 8 + e][slot] = h4;
        }
      }
    }
  };

  if (kt_begin < kt_end) load_tile(kt_begin);
  for (int kt = kt_begin; kt < kt_end; ++kt) {
    const int key0 = kt * kBN;
    store_tile();
    __syncthreads();
    if (kt + 1 < kt_end) load_tile(kt + 1);   // in flight while this tile is computed

    // ---- S^T = K Q^T for the 64 keys: two 32x32 blocks
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kb][e] = 0.f;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 ka = __builtin_bit_cast(bf16x8, *(const u32x4*)&Ks[kb * 32 + col][16 * s + 8 * hl]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[s], sacc[kb], 0, 0, 0);
      }
    }

    // ---- causal mask (only on tiles that cross the tail diagonal) and tile max
    if (key0 + kBN - 1 > S.L_keep + t_lo) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + kb * 32 + 8 * (e >> 2) + 4 * hl + (e & 3);
          if (key > my_limit) sacc[kb][e] = -__builtin_inff();
        }
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[kb][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c2;
    if (__any(mx > m_run + kTau)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = (m_new == -__builtin_inff()) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) scale_acc(o[db], alpha);
    }
    const float m_use = (m_run == -__builtin_inff()) ? 0.f : m_run;
    float psum = 0.f;
    f16x8 pf[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][e], c2, -m_use));
        psum += p;
        pf[kb * 2 + (e >> 3)][e & 7] = (_Float16)p;
      }
    l_run += psum;

    // ---- O^T += V^T P^T over 4 steps of 16 keys
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const f16x8 va = __builtin_bit_cast(f16x8, *(const u32x4*)&Vt[db * 32 + col][ks * 16 + 8 * hl]);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, pf[ks], o[db], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (!row_ok) return;
  if (S.n_splits == 1) {
    const float inv = 1.f / l_tot;
    float* orow = S.out + ((long)t * Hq + qh) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 v = {o[db][4 * i] * inv, o[db][4 * i + 1] * inv, o[db][4 * i + 2] * inv, o[db][4 * i + 3] * inv};
        *(f32x4*)(orow + db * 32 + 8 * i + 4 * hl) = v;
      }
  } else {
    const long prow = (long)split * S.T * Hq + (long)t * Hq + qh;
    float* orow = S.part_o + prow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 v = {o[db][4 * i], o[db][4 * i + 1], o[db][4 * i + 2], o[db][4 * i + 3]};
        *(f32x4*)(orow + db * 32 + 8 * i + 4 * hl) = v;
      }
    if (hl == 0) {
      S.part_ml[prow * 2] = m_run;
      S.part_ml[prow * 2 + 1] = l_tot;
    }
  }
}

// One thread per 4 output dims of one (token, head) row.
template <int D>
__global__ __launch_bounds__(256) void k_attn_merge(MergeArgs a) {
  constexpr int TPR = D / 4;  // threads per row
  const int g = blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
  const int d4 = threadIdx.x % TPR;
  if (g >= a.row_begin[a.n_seq]) return;
  int si = 0;
  while (si + 1 < a.n_seq && a.row_begin[si + 1] <= g) ++si;
  const AttnSeq S = a.seq[si];
  const long row = g - a.row_begin[si];
  const long R = (long)S.T * a.n_q_heads;
  float M = -__builtin_inff();
  for (int s = 0; s < S.n_splits; ++s) M = fmaxf(M, S.part_ml[(s * R + row) * 2]);
  float L = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < S.n_splits; ++s) {
    const float m = S.part_ml[(s * R + row) * 2];
    if (m == -__builtin_inff()) continue;
    const float w = __builtin_amdgcn_exp2f(m - M);
    L += w * S.part_ml[(s * R + row) * 2 + 1];
    const f32x4 v = *(const f32x4*)(S.part_o + (s * R + row) * D + 4 * d4);
    acc += w * v;
  }
  const float inv = 1.f / L;
  *(f32x4*)(S.out + row * D + 4 * d4) = acc * inv;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int head_dim, hipStream_t s) {
  if (a.total_items <= 0) return hipSuccess;
  // round the grid up to a multiple of 8 so the XCD remap is a bijection
  const int blocks = (a.total_items + 7) & ~7;
  if (head_dim == 256)
    hipLaunchKernelGGL(k_attn<256>, dim3(blocks), dim3(256), 0, s, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn<64>, dim3(blocks), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_merge(const MergeArgs& a, int total_rows, int head_dim, hipStream_t s) {
  if (total_rows <= 0) return hipSuccess;
  const int rows_per_block = 256 / (head_dim / 4);
  const int blocks = (total_rows + rows_per_block - 1) / rows_per_block;
  if (head_dim == 256)
    hipLaunchKernelGGL(k_attn_merge<256>, dim3(blocks), dim3(256), 0, s, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn_merge<64>, dim3(blocks), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tu
