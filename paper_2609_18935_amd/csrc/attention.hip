// Causal grouped-query attention of the tail over the surviving + new KV (paper
// Section 4.1, Eq. 3; Section 4.3: attending to the surviving context is the
// work that remains after unchanged records are no longer recomputed).
//
// Tail row i of query head h attends to cache rows 0 .. L_keep + i of KV head
// h / G (G = Hq / Hkv). The G query heads that share a KV head are packed as
// rows (token-major: packed row = t * G + (h mod G)), so one workgroup tile of
// 256 packed rows reads each K/V tile once for all of them.
//
// Workgroup: 8 waves of 32 packed rows each, two waves per SIMD; key tiles of 64
// rows in LDS, processed as two 32-key units. Scores are formed transposed,
// S^T = K Q^T, on v_mfma_f32_32x32x16_bf16 (A = 32 keys x 16 dims of K from LDS,
// B = 16 dims x 32 queries of Q held in registers), so a lane's accumulator holds
// 16 keys of ONE query and the online-softmax state is per lane; the two lanes of a
// query (l and l ^ 32) exchange their maxima once per unit. The output is accumulated
// transposed too, O^T += V^T P^T, on v_mfma_f32_32x32x16_f16 with P in [0, 2^8) rounded to f16
// (10 stored mantissa bits keep the result inside the accuracy bound; bf16's 7 do
// not). V^T comes pre-packed per 64-key tile as f16 by k_vt_pack, in exactly the LDS
// layout, so staging it is a plain copy (a copy kept beside the cache, or one packed for
// this call in the workspace).
//
// Tiles move HBM/L2 -> LDS with buffer_load_dwordx4 ... lds (no staging registers;
// the buffer resource of a tile ends at the cache's data, so rows past it read as
// zeros), double-buffered with one barrier per tile: after it, every wave is done with
// the previous tile, whose stage then receives the next tile while this one is
// computed. Loads are issued on every tile (zero bytes past the split's end), so the
// wait counts never change. Each unit runs its score MFMAs, the softmax and the P.V
// MFMAs in order; the other wave of the SIMD, at another point of its own units, keeps
// the matrix core fed meanwhile. A wave holds 256 registers: O^T for 32 rows x 256
// dims (128), the Q fragments (64), the scores and the rest, all in ordinary vector
// registers (the build asks for the VGPR form of the MFMAs, so the budget is not split
// in equal accumulator and vector halves, which would spill Q). The lane-pair
// exchanges use v_permlane32_swap instead of an LDS round trip.
//
// For occupancy the key range is split over `n_splits` workgroups; each writes a
// normalised f16 partial (O / l) with its reference max and sum, and k_attn_merge
// combines them. Workgroups are ordered (context, kv head, split, tile); the query
// tiles of one (context, head, split) key range go to one die (XCD) and share its L2.
// A launch of one context gives every die an equal share of the items in this order;
// a launch of several contexts, whose key ranges differ in length, places the groups
// by a table: longest first, each on the die with the least work so far.
#include "common.h"

namespace tu {

namespace {

typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;

constexpr int kBM = kAttnRows;
constexpr int kBN = kAttnKeys;
constexpr float kTau = 8.f;  // lazy-rescale threshold (log2 units): P < 2^8 fits f16

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt immediate that waits on the vector-memory counter only
constexpr int vm_wait(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// Fourth word of a raw buffer resource (32-bit data, no swizzle) on CDNA
constexpr int kBufWord3 = 0x00020000;

// Copies 16 bytes per lane from base + voff + soff to LDS (lane i writes lds + 16 i).
// The resource covers `bytes` from base; lanes past it write zeros. base and bytes are
// wave-uniform; reading them through readfirstlane lets the compiler see that, so the
// resource stays in scalar registers (no per-lane loop around the load).
__device__ __forceinline__ void dma16(const void* base, int bytes, uint32_t voff, uint32_t soff, void* lds) {
  const uint64_t b = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  void* ub = (void*)(((uint64_t)hi << 32) | lo);
  const __amdgpu_buffer_rsrc_t res =
      __builtin_amdgcn_make_buffer_rsrc(ub, 0, __builtin_amdgcn_readfirstlane(bytes), kBufWord3);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(res, (lds_void*)lds, 16, voff, soff, 0, 0);
}

// s_waitcnt immediate that waits on the LDS counter only
constexpr int kLgkmWait0 = 15 | (7 << 4) | (0 << 8) | (3 << 14);

// Workgroup barrier without the memory fence of __syncthreads: the fence would also
// wait for the tile prefetches still in flight. LDS hazards are covered by the
// explicit vm waits plus this barrier; the wave's own LDS reads have returned before
// it arrives, and the empty asm keeps the compiler from moving memory accesses
// across it.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(kLgkmWait0);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Two stages of K (bf16 [64 keys][D + 8]) and V^T (f16 [D][64 + 8], packed layout),
// sized for D = 256. Every row carries one 16-byte pad so that 16 consecutive rows
// read at the same column fall in 16 distinct bank groups while fragment addresses
// stay affine (one base register plus immediates). A stage is rounded up to whole
// rounds of 16-byte loads by the workgroup, so every wave issues the same number of
// loads per tile. Separate arrays, so the compiler sees that a prefetch into one stage
// does not alias reads of the other.
constexpr int kThreads = 512;       // 8 waves x 32 packed rows
constexpr int kVRow = kVtRow;       // f16 elements per V^T row
template <int D>
struct StageGeom {
  static constexpr int RC = D / 8;                            // data chunks per K row
  static constexpr int KRC = RC + 1;                          // chunks per K row in LDS
  static constexpr int NLK = (kBN * KRC + kThreads - 1) / kThreads;  // K loads per thread
  static constexpr int NLV = (D * (kVRow / 8) + kThreads - 1) / kThreads;
  static constexpr int NCV = D * (kVRow / 8);                 // V^T data chunks
};
constexpr int kKStage = StageGeom<256>::NLK * kThreads * 8;   // bf16 per K stage
constexpr int kVStage = StageGeom<256>::NLV * kThreads * 8;   // f16 per V^T stage
__shared__ __attribute__((aligned(16))) bf16_t g_ks0[kKStage];
__shared__ __attribute__((aligned(16))) bf16_t g_ks1[kKStage];
__shared__ __attribute__((aligned(16))) _Float16 g_vt0[kVStage];
__shared__ __attribute__((aligned(16))) _Float16 g_vt1[kVStage];

// Scales an MFMA accumulator (the rare move of the softmax reference max).
__device__ __forceinline__ void scale_acc(f32x16& acc, float s) {
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] *= s;
}

template <int B>
struct IntC {
  static constexpr int value = B;
};

// The item of this workgroup: by the launch's die table when it has one, else equal
// shares of the item order per die.
__device__ __forceinline__ int attn_item(const AttnOrder& o) {
  if (o.n_groups == 0) return xcd_remap(blockIdx.x, gridDim.x);
  const int x = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int g0 = o.die_begin[x], g1 = o.die_begin[x + 1];
  int g = g0;
  while (g < g1 && o.grp_end[g] <= slot) ++g;
  if (g == g1) return 0x7fffffff;   // the die's share ends before this slot
  return (int)o.grp_item0[g] + slot - (g > g0 ? (int)o.grp_end[g - 1] : 0);
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_attn(AttnArgs a,
                                                                                               AttnOrder ord) {
  constexpr int NS = D / 16;                // 16-dim steps of S^T = K Q^T
  constexpr int NDB = D / 32;               // 32-dim blocks of O^T
  constexpr int RC = D / 8;                 // 16-byte chunks of data per K row

  const int item = attn_item(ord);
  if (item >= a.total_items) return;
  int si = 0;
  while (si + 1 < a.n_seq && a.seq[si + 1].item_begin <= item) ++si;
  const AttnSeq& S = a.seq[si];
  int local = item - S.item_begin;
  const int tile = __builtin_amdgcn_readfirstlane(local % S.n_tiles);
  local /= S.n_tiles;
  const int split = __builtin_amdgcn_readfirstlane(local % S.n_splits);
  const int hkv = __builtin_amdgcn_readfirstlane(local / S.n_splits);

  const int Hq = a.n_q_heads;
  const int Hkv = a.n_kv_heads;
  const int G = Hq / Hkv;
  const int T = S.T;
  const int L_keep = S.L_keep;
  const int rows_total = T * G;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hl = lane >> 5;     // half of the wave
  const int col = lane & 31;    // query column of this lane

  const int r = tile * kBM + wave * 32 + col;
  const bool row_ok = r < rows_total;
  const int t = row_ok ? r / G : T - 1;
  const int qh = hkv * G + (row_ok ? r - (r / G) * G : 0);
  const int my_limit = L_keep + t;  // last key this query may see
  const int r_last = min(rows_total, (tile + 1) * kBM) - 1;
  const int t_hi = r_last / G;
  const int t_lo = __builtin_amdgcn_readfirstlane((tile * kBM) / G);
  const int n_keys = L_keep + t_hi + 1;
  const int n_kt = (n_keys + kBN - 1) / kBN;
  const int tps = (n_kt + S.n_splits - 1) / S.n_splits;
  const int kt_begin = __builtin_amdgcn_readfirstlane(split * tps);
  const int kt_end = __builtin_amdgcn_readfirstlane(min(n_kt, kt_begin + tps));
  const int n_valid = L_keep + T;   // cache rows holding data

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
  // when a unit's max exceeds it by more than kTau, so P stays below 2^kTau.
  float m_run = -__builtin_inff();
  float l_run = 0.f;
  const float c2 = a.scale_log2;

  const long rs = (long)Hkv * D;  // elements per cache row
  const bf16_t* kbase = S.k_cache + (long)hkv * D;
  const _Float16* vtbase = S.vt + (long)hkv * S.head_tiles * (D * kVRow);

  // ---- tile prefetch. A stage holds K as rows of RC + 1 chunks (16 B each; the last
  // is padding) and V^T as D rows of 9 chunks. LDS chunk q = i * kThreads + tid is
  // written by load i of thread tid (a wave's 64 lanes fill 64 consecutive chunks).
  // Loads go through a buffer resource per tile whose size ends at the cache's data:
  // lanes past it (the last tile's missing rows, the round-up tail of a stage) read
  // zeros. Padding chunks receive a copy of their row's first chunk (never read). V^T
  // tiles come from k_vt_pack in this exact layout and are copied chunk for chunk.
  using GM = StageGeom<D>;
  constexpr int KRC = GM::KRC;
  constexpr int NLK = GM::NLK;
  constexpr int NLV = GM::NLV;
  // lane byte offsets of the K loads within a tile
  uint32_t koff[NLK];
#pragma unroll
  for (int i = 0; i < NLK; ++i) {
    const int q = i * kThreads + tid;
    const int row = q / KRC;
    const int c = q - row * KRC;
    koff[i] = (uint32_t)(row * rs * 2 + (c < RC ? c : 0) * 16);
  }
  auto load_k = [&](auto bc, int kt) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    bf16_t* dst = B ? g_ks1 : g_ks0;
    const int key0 = kt * kBN;
    // bytes from this head's part of row key0 to the end of its part of the last data
    // row (zero past the split's last tile)
    const int rows = min(n_valid - key0, 2 * kBN);
    const int bytes = max(rows * (int)rs * 2 - ((int)rs - D) * 2, 0) * (int)(kt < kt_end);
    const bf16_t* base = kbase + (long)key0 * rs;
#pragma unroll
    for (int i = 0; i < NLK; ++i) dma16(base, bytes, koff[i], 0, dst + (i * kThreads + wave * 64) * 8);
  };
  const uint32_t voff = (uint32_t)tid * 16;
  auto load_v = [&](auto bc, int kt) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    _Float16* dst = B ? g_vt1 : g_vt0;
    const _Float16* base = vtbase + (long)kt * (D * kVRow);
    const int bytes = kt < kt_end ? GM::NCV * 16 : 0;
#pragma unroll
    for (int i = 0; i < NLV; ++i) dma16(base, bytes, voff, i * kThreads * 16, dst + (i * kThreads + wave * 64) * 8);
  };

  // ---- LDS fragment addresses: K row 32 * half + col, chunk 2s + hl; V^T row
  // 32 db + col, chunk 2u + hl (16-key group u of the tile)
  const uint32_t ka_base = (uint32_t)(col * KRC * 16 + hl * 16);
  const uint32_t va_base = (uint32_t)(col * kVRow * 2 + hl * 16);

  // ---- S^T for the 32 keys of unit `half` of the tile in stage B, dim steps [S0, S1)
  auto qk_part = [&](auto bc, int half, f32x16& sacc, auto s0c, auto s1c) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    constexpr int S0 = decltype(s0c)::value, S1 = decltype(s1c)::value;
    const char* ks = (const char*)(B ? g_ks1 : g_ks0) + ka_base + half * 32 * KRC * 16;
    if constexpr (S0 == 0) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
    }
#pragma unroll
    for (int s = S0; s < S1; ++s) {
      const bf16x8 ka = __builtin_bit_cast(bf16x8, *(const u32x4*)(ks + s * 32));
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[s], sacc, 0, 0, 0);
    }
  };
  // ---- causal mask of a unit crossing the tail diagonal (a uniform branch)
  auto mask = [&](int kb0, f32x16& sacc) __attribute__((always_inline)) {
    if (kb0 + 31 > L_keep + t_lo) {
      // element e holds key kb0 + 4 hl + 8 (e >> 2) + (e & 3); comparing its constant
      // part against one per-unit difference keeps the offsets as immediates
      const int room = my_limit - kb0 - 4 * hl;
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (8 * (e >> 2) + (e & 3) > room) sacc[e] = -__builtin_inff();
    }
  };
  // ---- the unit's max over the query's 32 keys (lanes l and l ^ 32 hold 16 each)
  auto rowmax = [&](const f32x16& sacc) __attribute__((always_inline)) -> float {
    float mx = -__builtin_inff();
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[e]);
    const auto sw = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, mx),
                                                     __builtin_bit_cast(uint32_t, mx), false, false);
    return fmaxf(__builtin_bit_cast(float, (uint32_t)sw[0]), __builtin_bit_cast(float, (uint32_t)sw[1])) * c2;
  };
  // ---- lazy move of the reference max (rare: O and l rescaled)
  auto rescale_if = [&](float mx) __attribute__((always_inline)) {
    if (__any(mx > m_run + kTau)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = (m_new == -__builtin_inff()) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) scale_acc(o[db], alpha);
    }
  };
  // ---- probabilities, rounded to f16 in the key order of the P^T fragments
  auto sexp = [&](const f32x16& sacc, f16x8 (&pf)[2]) __attribute__((always_inline)) {
    const float m_use = (m_run == -__builtin_inff()) ? 0.f : m_run;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[e], c2, -m_use));
      ps[e & 3] += p;
      pf[e >> 3][e & 7] = (_Float16)p;
    }
    l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
  };
  // ---- O^T += V^T P^T for the 32 keys of unit `half` of the tile in stage B
  auto pv = [&](auto bc, int half, const f16x8 (&pf)[2]) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    const char* vt = (const char*)(B ? g_vt1 : g_vt0) + va_base;
#pragma unroll
    for (int ks16 = 0; ks16 < 2; ++ks16) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const f16x8 va = __builtin_bit_cast(
            f16x8, *(const u32x4*)(vt + db * 32 * kVRow * 2 + (half * 2 + ks16) * 32));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, pf[ks16], o[db], 0, 0, 0);
      }
    }
  };

  // Keep n MFMAs fed by their LDS fragment reads, two reads ahead: bounds the fragment
  // registers in flight (the compiler would otherwise issue every read up front).
  constexpr int kMfma = 0x008, kDsRead = 0x100;
  auto sched_reads = [&](auto nc) __attribute__((always_inline)) {
    constexpr int N = decltype(nc)::value;
    __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
      if (i < N - 1) __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
    }
  };

  f32x16 sa;
  f16x8 pf[2];
  // One 32-key unit of the tile in stage B: scores, softmax, P.V.
  auto unit = [&](auto bc, int half, int kb0) __attribute__((always_inline)) {
    qk_part(bc, half, sa, IntC<0>{}, IntC<NS>{});
    sched_reads(IntC<NS>{});
    mask(kb0, sa);
    const float mx = rowmax(sa);
    rescale_if(mx);
    sexp(sa, pf);
    pv(bc, half, pf);
    sched_reads(IntC<2 * NDB>{});
  };
  // One key tile kt in stage B. Only this tile's loads are in flight on entry: once they
  // have landed and every wave has passed the barrier, every wave is also done with
  // tile kt - 1, so the loads of tile kt + 1 go to the other stage at once and land
  // while this tile is computed (one barrier per tile). Loads are issued
  // unconditionally (past the split's last tile they have zero bytes), so the wait
  // counts are the same on every tile.
  auto step = [&](auto bc, int kt) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    __builtin_amdgcn_s_waitcnt(vm_wait(0));   // this wave's loads of tile kt have landed
    wg_barrier();                              // everyone's have; stage B ^ 1 is free
    load_k(IntC<B ^ 1>{}, kt + 1);
    load_v(IntC<B ^ 1>{}, kt + 1);
    unit(bc, 0, kt * kBN);
    unit(bc, 1, kt * kBN + 32);
  };

  if (kt_begin < kt_end) {
    load_k(IntC<0>{}, kt_begin);
    load_v(IntC<0>{}, kt_begin);
    for (int kt = kt_begin; kt < kt_end; kt += 2) {
      step(IntC<0>{}, kt);
      if (kt + 1 < kt_end) step(IntC<1>{}, kt + 1);
    }
    __builtin_amdgcn_s_waitcnt(vm_wait(0));  // no tile write may outlive the workgroup
  }

  const auto lsw = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, l_run),
                                                    __builtin_bit_cast(uint32_t, l_run), false, false);
  const float l_tot = __builtin_bit_cast(float, (uint32_t)lsw[0]) + __builtin_bit_cast(float, (uint32_t)lsw[1]);
  if (!row_ok) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (S.n_splits == 1) {
    float* orow = S.out + ((long)t * Hq + qh) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 v = {o[db][4 * i] * inv, o[db][4 * i + 1] * inv, o[db][4 * i + 2] * inv, o[db][4 * i + 3] * inv};
        *(f32x4*)(orow + db * 32 + 8 * i + 4 * hl) = v;
      }
  } else {
    const long prow = (long)split * T * Hq + (long)t * Hq + qh;
    _Float16* orow = S.part_o + prow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f16x4 v = {(_Float16)(o[db][4 * i] * inv), (_Float16)(o[db][4 * i + 1] * inv),
                   (_Float16)(o[db][4 * i + 2] * inv), (_Float16)(o[db][4 * i + 3] * inv)};
        *(f16x4*)(orow + db * 32 + 8 * i + 4 * hl) = v;
      }
    if (hl == 0) {
      S.part_ml[prow * 2] = l_tot > 0.f ? m_run : -__builtin_inff();
      S.part_ml[prow * 2 + 1] = l_tot;
    }
  }
}

// Log-sum-exp merge of the split partials: `split_lanes` (1, 2, 4 or 8) consecutive
// lanes per 8 output dims of one (token, head) row. Lane l of a row's group takes the
// splits l, l + split_lanes, ... in batches of 8 whose loads are all in flight
// together (the running max and sums move between batches); the lanes' partial
// results are then combined by shuffles and the first lane writes the row's 8 outputs.
template <int D>
__global__ __launch_bounds__(256) void k_attn_merge(MergeArgs a) {
  constexpr int TPR = D / 8;  // 8-dim pieces per row
  const int SL = a.split_lanes;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int g = t / (TPR * SL);
  const int d8 = (t / SL) % TPR;
  const int sl = t % SL;
  const bool live = g < a.row_begin[a.n_seq];
  float M = -__builtin_inff(), L = 0.f;
  f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  // (no pointer into the argument struct outlives this block: that would make the
  // compiler copy the struct to scratch memory)
  float* orow = nullptr;
  if (live) {
    int si = 0;
    while (si + 1 < a.n_seq && a.row_begin[si + 1] <= g) ++si;
    const AttnSeq& S = a.seq[si];
    const long row = g - a.row_begin[si];
    orow = S.out + row * D + 8 * d8;
    const long R = (long)S.T * a.n_q_heads;
    for (int s0 = sl; s0 < S.n_splits; s0 += 8 * SL) {
      f32x2 ml[8];
      f16x8 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int sp = s0 + j * SL;
        const long at = (long)sp * R + row;
        if (sp < S.n_splits) {
          ml[j] = *(const f32x2*)(S.part_ml + at * 2);
          v[j] = *(const f16x8*)(S.part_o + at * D + 8 * d8);
        } else {
          ml[j] = f32x2{-__builtin_inff(), 0.f};
          v[j] = f16x8{};
        }
      }
      float Mb = M;
#pragma unroll
      for (int j = 0; j < 8; ++j) Mb = fmaxf(Mb, ml[j][0]);
      if (Mb == -__builtin_inff()) continue;
      const float c = M == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(M - Mb);
      L *= c;
      acc0 *= c;
      acc1 *= c;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (ml[j][0] == -__builtin_inff()) continue;
        const float w = __builtin_amdgcn_exp2f(ml[j][0] - Mb) * ml[j][1];
        L += w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc0[e] += w * (float)v[j][e];
          acc1[e] += w * (float)v[j][4 + e];
        }
      }
      M = Mb;
    }
  }
  // combine the lanes of a row group (every lane of the wave takes part in the shuffles)
  for (int x = 1; x < SL; x <<= 1) {
    const float M2 = __shfl_xor(M, x, 64);
    const float L2 = __shfl_xor(L, x, 64);
    f32x4 b0, b1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      b0[e] = __shfl_xor(acc0[e], x, 64);
      b1[e] = __shfl_xor(acc1[e], x, 64);
    }
    const float Mn = fmaxf(M, M2);
    if (Mn == -__builtin_inff()) continue;
    const float c1 = M == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    const float c2 = M2 == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(M2 - Mn);
    L = L * c1 + L2 * c2;
    acc0 = acc0 * c1 + b0 * c2;
    acc1 = acc1 * c1 + b1 * c2;
    M = Mn;
  }
  if (!live || sl != 0) return;
  const float inv = 1.f / L;
  *(f32x4*)orow = acc0 * inv;
  *(f32x4*)(orow + 4) = acc1 * inv;
}

}  // namespace

static_assert(sizeof(AttnArgs) + sizeof(AttnOrder) <= kMaxKernargBytes, "attention launch record");
static_assert(sizeof(MergeArgs) <= kMaxKernargBytes, "merge launch record");

hipError_t launch_attention(const AttnArgs& a, const AttnOrder& o, int head_dim, hipStream_t s) {
  if (a.total_items <= 0) return hipSuccess;
  // without a die table the grid is rounded up to a multiple of 8 so the remap is a bijection
  const int blocks = o.n_groups > 0 ? o.blocks : (a.total_items + kXcds - 1) / kXcds * kXcds;
  if (head_dim == 256)
    hipLaunchKernelGGL(k_attn<256>, dim3(blocks), dim3(kThreads), 0, s, a, o);
  else if (head_dim == 128)
    hipLaunchKernelGGL(k_attn<128>, dim3(blocks), dim3(kThreads), 0, s, a, o);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn<64>, dim3(blocks), dim3(kThreads), 0, s, a, o);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_merge(const MergeArgs& a, int total_rows, int head_dim, hipStream_t s) {
  if (total_rows <= 0) return hipSuccess;
  if (a.split_lanes != 1 && a.split_lanes != 2 && a.split_lanes != 4 && a.split_lanes != 8) return hipErrorInvalidValue;
  const long threads = (long)total_rows * (head_dim / 8) * a.split_lanes;
  const int blocks = (int)((threads + 255) / 256);
  if (head_dim == 256)
    hipLaunchKernelGGL(k_attn_merge<256>, dim3(blocks), dim3(256), 0, s, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL(k_attn_merge<128>, dim3(blocks), dim3(256), 0, s, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(k_attn_merge<64>, dim3(blocks), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tu
