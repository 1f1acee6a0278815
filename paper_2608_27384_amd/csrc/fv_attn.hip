// Chunk-wise causal attention of action tokens over [prefix ; buffer].
//
// The mask of the paper (Sec. 3.1: a noisier, later chunk attends to the
// cleaner, earlier chunks, never the reverse, at chunk granularity; every
// action token sees the cached observation) becomes two key ranges here:
// the QKV epilogue writes buffer token j of stream b at arena row P0_b + j,
// P0_b = buffer_row0(P_b) >= P_b the first multiple of 8 at or after the P_b
// valid prefix rows, so a query of chunk k sees the rows [0, P_b) and
// [P0_b + C lo, P0_b + C hi) with (lo, hi) = (first valid slot,
// k + 1).  The other mask modes and cold-start padding only change (lo, hi)
// (visible_chunks).  Keys outside a query's ranges are scored -inf, giving
// probability exactly 0; tiles outside every row's ranges are not visited.
//
// Work split: the query rows of one (stream, kv head) are the (token, head)
// pairs of its query-head group, flattened token-major; a block takes
// consecutive rows, 16 per wave (bf16: 8 waves, 128 rows; fp32: 4 waves, 64
// rows, RG groups of 16 rows per wave sharing every K and V fragment read
// from LDS), so rows of all heads that share the kv head reuse one K/V tile.
// For bf16 head dims 128 and 256 (attn16d_kernel) the K/V tiles go from
// memory straight into a ring of LDS stages, three tiles ahead; otherwise the
// next K/V tile is loaded into registers while the current one is
// multiplied.  Rows of a block may straddle a chunk
// boundary; each lane masks with its own row's limit.  Optionally the key
// tiles of a block are split over gridDim.z blocks whose normalised partial
// outputs (in the element type) and (max, sum) are merged in a fixed order
// by attn_combine.
//
// Per key tile (KT keys): K [KT][dh] and V^T [dh][KT] are staged in LDS;
// each wave forms S^T = K Q^T with MFMA, so a lane holds the scores of one
// query for 4 keys per 16-key subtile; the row max and row sum need only two
// cross-lane exchanges (lanes l, l^16, l^32, l^48); the probabilities are
// then, without any data movement, the B operand of O^T += V^T P^T.
#include <algorithm>
#include <vector>

#include "fv_internal.h"

namespace fv {

namespace {

constexpr float kSlack = 8.0f;  // lazy softmax reference slack (log2 units)
constexpr float kHeadroom = 64.0f;  // fixed-reference headroom of the bf16 kernel (log2 units)
constexpr int kRG = 1;          // 16-row MFMA groups per wave
constexpr int kRowsPerBlock = 4 * 16 * kRG;
constexpr int kAttn16Waves = 8;  // bf16 kernel: 8 waves x 16 rows
constexpr int kAttnStages = 4;  // K/V tile stages of the direct-load kernel (3-5 measured equal)
template <int DH>
constexpr int attn16d_lds() {
  return kAttnStages * 2 * (32 * DH * 2);
}

template <typename T>
constexpr int rows_per_block() {
  return sizeof(T) == 2 ? 16 * kAttn16Waves : kRowsPerBlock;
}

// Key tiles a block visits: the prefix tiles [0, nA), then the tiles of the
// buffer span [P0 + C lo_min, P0 + C hi_max) (the rows' visible chunk ranges
// are monotone in the chunk index, so the first and last row of the block
// bound them), without the masked gap between the two.
struct KeyTiles {
  int nA, tB0, n;
  __device__ int tile(int vt) const { return vt < nA ? vt : tB0 + (vt - nA); }
};
__device__ __forceinline__ KeyTiles key_tiles(int P, int C, int K, int first, int mode,
                                              int tok_first, int tok_last, int KT) {
  const int P0 = buffer_row0(P);  // arena row of the first buffer token
  int lo0, hi0, lo1, hi1;
  visible_chunks(tok_first / C, K, first, mode, lo0, hi0);
  visible_chunks(tok_last / C, K, first, mode, lo1, hi1);
  KeyTiles r;
  r.nA = (P + KT - 1) / KT;
  r.tB0 = max((P0 + C * lo0) / KT, r.nA);
  const int tB1 = (P0 + C * hi1 + KT - 1) / KT;
  r.n = r.nA + max(0, tB1 - r.tB0);
  return r;
}

template <typename T, int DH, int KT, int RG>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int kRowsPerWave = 16 * RG;
  constexpr int kRowsPerBlock = 4 * kRowsPerWave;
  using MF = Mfma<T>;
  constexpr int EPV = 16 / (int)sizeof(T);
  constexpr int LDK = DH + EPV;
  constexpr int LDV = KT + EPV;
  constexpr int NST = KT / 16;
  constexpr int NKS = DH / MF::KM;
  constexpr int NDT = DH / 16;
  constexpr int VK = KT * DH / EPV, VV = DH * KT / EPV;  // 16-byte vectors per tile
  constexpr int NVK = (VK + 255) / 256, NVV = (VV + 255) / 256;
  constexpr bool kBF16 = sizeof(T) == 2;
  static_assert(!kBF16 || NST % 2 == 0, "bf16 path pairs 16-key subtiles");

  __shared__ __attribute__((aligned(16))) T sK[KT * LDK];
  __shared__ __attribute__((aligned(16))) T sV[DH * LDV];

  const int G = a.n_q_heads / a.n_kv_heads;
  const int rows_bg = a.tokens * G;
  const int tile0 = blockIdx.x * kRowsPerBlock;
  const int b = blockIdx.y / a.n_kv_heads, g = blockIdx.y - b * a.n_kv_heads;
  const int split = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int P = a.len[b];
  const int C = a.chunk_len;
  const int l16 = lane & 15, lg = lane >> 4;

  const int K = a.tokens / C;
  const int first = K - a.n_valid[b];
  // this lane's query rows (one per 16-row group) and their buffer key ranges
  int tok[RG], head[RG], klo[RG], khi[RG];
  bool valid[RG];
#pragma unroll
  for (int q = 0; q < RG; ++q) {
    const int rq = tile0 + kRowsPerWave * wave + 16 * q + l16;
    valid[q] = rq < rows_bg;
    const int rqc = valid[q] ? rq : rows_bg - 1;
    tok[q] = rqc / G;
    head[q] = g * G + (rqc - tok[q] * G);
    int lo, hi;
    visible_chunks(tok[q] / C, K, first, a.mask_mode, lo, hi);
    klo[q] = buffer_row0(P) + C * lo;
    khi[q] = buffer_row0(P) + C * hi;
  }
  const int rlast = min(tile0 + kRowsPerBlock - 1, rows_bg - 1);
  const KeyTiles kts = key_tiles(P, C, K, first, a.mask_mode, tile0 / G, rlast / G, KT);
  const int kt_begin = (split * kts.n) / a.n_split, kt_end = ((split + 1) * kts.n) / a.n_split;

  typename MF::frag qf[RG][NKS];
#pragma unroll
  for (int q = 0; q < RG; ++q) {
    const T* qrow = reinterpret_cast<const T*>(a.q) +
                    ((size_t)(b * a.tokens + tok[q]) * a.n_q_heads + head[q]) * DH;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[q][ks] = MF::load(qrow + ks * MF::KM + MF::KG * lg);
  }

  f32x4 acc[RG][NDT];
  float m_run[RG], l_run[RG];
#pragma unroll
  for (int q = 0; q < RG; ++q) {
    m_run[q] = -INFINITY;
    l_run[q] = 0.f;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) acc[q][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const T* kbase = reinterpret_cast<const T*>(a.karena) +
                   ((size_t)b * a.n_kv_heads + g) * (size_t)a.S * DH;
  const T* vbase = reinterpret_cast<const T*>(a.vtarena) +
                   ((size_t)b * a.n_kv_heads + g) * (size_t)DH * a.S;
  const float sl2 = 1.4426950408889634f / sqrtf((float)DH);

  // register stage of one K / V^T tile (loads issued unconditionally; a
  // clamped tile index keeps the addresses in bounds)
  u32x4 rk[NVK], rv[NVV];
  auto load_tile = [&](int kt) __attribute__((always_inline)) {
    const int key0 = kt * KT;
#pragma unroll
    for (int i = 0; i < NVK; ++i) {
      const int vi = tid + 256 * i;
      if (VK % 256 == 0 || vi < VK) {
        const int r = vi / (DH / EPV), c = vi - r * (DH / EPV);
        rk[i] = *reinterpret_cast<const u32x4*>(kbase + (size_t)(key0 + r) * DH + c * EPV);
      }
    }
#pragma unroll
    for (int i = 0; i < NVV; ++i) {
      const int vi = tid + 256 * i;
      if (VV % 256 == 0 || vi < VV) {
        const int r = vi / (KT / EPV), c = vi - r * (KT / EPV);
        rv[i] = *reinterpret_cast<const u32x4*>(vbase + (size_t)r * a.S + key0 + c * EPV);
      }
    }
  };
  auto store_tile = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NVK; ++i) {
      const int vi = tid + 256 * i;
      if (VK % 256 == 0 || vi < VK) {
        const int r = vi / (DH / EPV), c = vi - r * (DH / EPV);
        *reinterpret_cast<u32x4*>(&sK[r * LDK + c * EPV]) = rk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < NVV; ++i) {
      const int vi = tid + 256 * i;
      if (VV % 256 == 0 || vi < VV) {
        const int r = vi / (KT / EPV), c = vi - r * (KT / EPV);
        *reinterpret_cast<u32x4*>(&sV[r * LDV + c * EPV]) = rv[i];
      }
    }
  };

  const int kt_clamp = max(kt_begin, kt_end - 1);
  load_tile(kts.tile(min(kt_begin, kt_clamp)));
  for (int vt = kt_begin; vt < kt_end; ++vt) {
    const int key0 = kts.tile(vt) * KT;
    __syncthreads();  // previous tile fully consumed
    store_tile();
    __syncthreads();
    load_tile(kts.tile(min(vt + 1, kt_clamp)));  // overlaps the MFMA work below

    // S^T = K Q^T for every row group; K fragments are shared
    f32x4 s[RG][NST];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
#pragma unroll
      for (int q = 0; q < RG; ++q) s[q][st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const typename MF::frag kf =
            MF::load(&sK[(16 * st + l16) * LDK + ks * MF::KM + MF::KG * lg]);
#pragma unroll
        for (int q = 0; q < RG; ++q) s[q][st] = MF::mma(kf, qf[q][ks], s[q][st]);
      }
    }
    // Online softmax per query row (a lane owns one row of each group) with
    // a lazily moved reference: exponents are taken against m_run, which
    // only moves when a row's tile maximum exceeds it by more than kSlack
    // (log2 units), so probabilities stay below 2^kSlack and the costly
    // rescale of the accumulators runs only when some row of the wave moved.
    bool moved = false;
    float alpha[RG];
#pragma unroll
    for (int q = 0; q < RG; ++q) {
      float mt = -INFINITY;
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = key0 + 16 * st + 4 * lg + r;
          const bool vis = key < P || (key >= klo[q] && key < khi[q]);
          const float x = vis ? s[q][st][r] * sl2 : -INFINITY;
          s[q][st][r] = x;
          mt = fmaxf(mt, x);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = mt > m_run[q] + kSlack ? mt : m_run[q];
      alpha[q] = 1.f;
      if (m_new != m_run[q]) {
        // acc and l are still zero while m_run is -inf
        alpha[q] = m_run[q] == -INFINITY ? 0.f : exp2f(m_run[q] - m_new);
        moved = true;
      }
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      float ls = 0.f;
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = exp2f(s[q][st][r] - m_use);
          s[q][st][r] = p;
          ls += p;
        }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      l_run[q] = l_run[q] * alpha[q] + ls;
      m_run[q] = m_new;
    }
    if (__any(moved)) {
#pragma unroll
      for (int q = 0; q < RG; ++q)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[q][dt] *= alpha[q];
    }

    // O^T += V^T P^T; V^T fragments are shared by both row groups
    if constexpr (kBF16) {
#pragma unroll
      for (int kc = 0; kc < NST / 2; ++kc) {
        bf16x8 pf[RG];
#pragma unroll
        for (int q = 0; q < RG; ++q) {
          u16x8 pb;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            pb[r] = f32_to_bf16(s[q][2 * kc][r]);
            pb[4 + r] = f32_to_bf16(s[q][2 * kc + 1][r]);
          }
          pf[q] = __builtin_bit_cast(bf16x8, pb);
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const T* vr = &sV[(16 * dt + l16) * LDV + 32 * kc + 4 * lg];
          const u16x4 lo = *reinterpret_cast<const u16x4*>(vr);
          const u16x4 hi = *reinterpret_cast<const u16x4*>(vr + 16);
          const bf16x8 vf = __builtin_bit_cast(
              bf16x8, u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
#pragma unroll
          for (int q = 0; q < RG; ++q)
            acc[q][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[q], acc[q][dt], 0, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) {
            const float vf = (float)sV[(16 * dt + l16) * LDV + 16 * st + 4 * lg + r];
#pragma unroll
            for (int q = 0; q < RG; ++q)
              acc[q][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf, (float)s[q][st][r], acc[q][dt],
                                                                0, 0, 0);
          }
    }
  }

  const size_t R = (size_t)a.B * a.tokens * a.n_q_heads;
#pragma unroll
  for (int q = 0; q < RG; ++q) {
    if (!valid[q]) continue;
    const size_t grow = (size_t)(b * a.tokens + tok[q]) * a.n_q_heads + head[q];
    // normalised output (a split with no visible key stores zeros)
    const float inv = l_run[q] > 0.f ? 1.0f / l_run[q] : 0.f;
    T* orow = a.n_split == 1
                  ? reinterpret_cast<T*>(a.o) + grow * DH
                  : reinterpret_cast<T*>(a.part_o) + ((size_t)split * R + grow) * DH;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) orow[16 * dt + 4 * lg + r] = from_f32<T>(acc[q][dt][r] * inv);
    if (a.n_split > 1 && lg == 0) {
      a.part_ml[((size_t)split * R + grow) * 2 + 0] = m_run[q];
      a.part_ml[((size_t)split * R + grow) * 2 + 1] = l_run[q];
    }
  }
}

// bf16 path with 16x16x32 MFMAs and 16 query rows per wave: 8 waves share
// each K/V tile of a 128-row block.  A wave's state (O^T 256 x 16 in 64
// registers, Q^T fragments in 32) lets two waves share a SIMD, so one
// wave's softmax arithmetic and fixed costs overlap the other's MFMAs (a
// 32-row wave needs 128 + 64 registers for the same and runs alone).  S^T = K Q^T per 16-key half h gives lane l
// the scores of query l % 16 for keys 16 h + 4 g + 0..3 (g = l / 16); the 8
// scores of both halves, rounded to bf16, are the B operand of
// O^T += V^T P^T with the MFMA's k index 8 g + e standing for key
// 4 g + e (e < 4) or 16 + 4 g + e - 4 (e >= 4), and the V^T fragment reads
// the same two 4-key runs.
// Reductions over the lanes l, l ^ 16, l ^ 32, l ^ 48 of a wave with the
// gfx950 lane swaps (VALU, no LDS): swapping a value with itself across
// 16-lane rows (32-lane halves) hands each lane the pair {x[l], x[l ^ 16]}
// ({x[l], x[l ^ 32]}) in its two results.
__device__ __forceinline__ float max_xor16_32(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum_xor16_32(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// (a plain function: the load builtin written directly in a kernel template
// body loses the template's host-side launch stub)
__device__ __forceinline__ void lds_dma16_attn(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
}
template <int N>
__device__ __forceinline__ void wait_vmcnt_attn() {  // at most N vector memory ops outstanding
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void wait_lgkmcnt0_attn() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}

// (row tile, stream x kv head) of this block.  Block b runs on die b % 8 of
// the chip (each die has its own L2); on large grids without key splits the
// blocks of a die take a contiguous range of the (stream-major) work list,
// so the row tiles of one stream, which read the same keys and values, run
// together on one die instead of being spread over all eight.
// The list is walked in die_order, which gives every die about the same
// total prefix length (ragged prefixes otherwise leave some dies a seventh
// more work than others), and a stream's row tiles from the last.
__device__ __forceinline__ void attn_block_of(int& rtile, int& bg, const int* __restrict__ order) {
  const int nx = gridDim.x, nb = nx * gridDim.y;
  if (gridDim.z > 1 || nb < 64) {
    rtile = blockIdx.x;
    bg = blockIdx.y;
    return;
  }
  const int blk = blockIdx.y * nx + blockIdx.x;
  const int per = nb >> 3, rem = nb & 7;
  const int x = blk & 7, slot = blk >> 3;
  const int L = x * per + min(x, rem) + slot;
  const int pos = L / nx;
  bg = order[pos];
  // a stream's last row tiles see the most buffer keys: they go first
  rtile = nx - 1 - (L - pos * nx);
}

template <int DH, int NWV>
__global__ __launch_bounds__(64 * NWV) void attn16_kernel(AttnArgs a) {
  using T = bf16_t;
  constexpr int KT = 32;                 // keys per tile
  constexpr int NT = 64 * NWV;           // threads
  constexpr int RB = 16 * NWV;           // query rows per block
  constexpr int LDK = DH + 8, LDV = KT + 4;
  constexpr int NKS = DH / 32;           // 32-wide k steps of Q K^T
  constexpr int NDT = DH / 16;           // 16-row tiles of O^T
  constexpr int VK = KT * DH / 8, VV = DH * KT / 8;  // 16-byte vectors per tile
  constexpr int NVK = (VK + NT - 1) / NT, NVV = (VV + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) T sK[KT * LDK];
  __shared__ __attribute__((aligned(16))) T sV[DH * LDV];
  __shared__ __attribute__((aligned(16))) T sO[NWV][16 * LDK];  // output staging

  const int G = a.n_q_heads / a.n_kv_heads;
  const int rows_bg = a.tokens * G;
  int rtile, bg;
  attn_block_of(rtile, bg, a.bg_order);
  const int tile0 = rtile * RB;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int split = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int P = a.len[b];
  const int C = a.chunk_len;
  const int l16 = lane & 15, lg = lane >> 4;

  const int K = a.tokens / C;
  const int first = K - a.n_valid[b];
  const int rq = tile0 + 16 * wave + l16;
  const bool valid = rq < rows_bg;
  const int rqc = valid ? rq : rows_bg - 1;
  const int tok = rqc / G;
  const int head = g * G + (rqc - tok * G);
  int klo, khi;  // this row's visible buffer keys [klo, khi); prefix keys [0, P)
  visible_chunks(tok / C, K, first, a.mask_mode, klo, khi);
  klo = buffer_row0(P) + C * klo;
  khi = buffer_row0(P) + C * khi;
  const int rlast = min(tile0 + RB - 1, rows_bg - 1);
  const KeyTiles kts = key_tiles(P, C, K, first, a.mask_mode, tile0 / G, rlast / G, KT);
  const int kt_begin = (split * kts.n) / a.n_split, kt_end = ((split + 1) * kts.n) / a.n_split;

  // Q^T fragments (B operand): query l16, dh 32 ks + 8 lg .. + 8
  bf16x8 qf[NKS];
  {
    const T* qrow = reinterpret_cast<const T*>(a.q) +
                    ((size_t)(b * a.tokens + tok) * a.n_q_heads + head) * DH;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(qrow + 32 * ks + 8 * lg));
  }
  f32x4 acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const T* kbase = reinterpret_cast<const T*>(a.karena) +
                   ((size_t)b * a.n_kv_heads + g) * (size_t)a.S * DH;
  const T* vbase = reinterpret_cast<const T*>(a.vtarena) +
                   ((size_t)b * a.n_kv_heads + g) * (size_t)DH * a.S;
  const float sl2 = 1.4426950408889634f / sqrtf((float)DH);

  u32x4 rk[NVK], rv[NVV];
  auto load_tile = [&](int kt) __attribute__((always_inline)) {
    const int key0 = kt * KT;
#pragma unroll
    for (int i = 0; i < NVK; ++i) {
      const int vi = tid + NT * i;
      if (VK % NT == 0 || vi < VK) {
        const int r = vi / (DH / 8), c = vi - r * (DH / 8);
        rk[i] = *reinterpret_cast<const u32x4*>(kbase + (size_t)(key0 + r) * DH + c * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < NVV; ++i) {
      const int vi = tid + NT * i;
      if (VV % NT == 0 || vi < VV) {
        const int r = vi / (KT / 8), c = vi - r * (KT / 8);
        rv[i] = *reinterpret_cast<const u32x4*>(vbase + (size_t)r * a.S + key0 + c * 8);
      }
    }
  };
  auto store_tile = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NVK; ++i) {
      const int vi = tid + NT * i;
      if (VK % NT == 0 || vi < VK) {
        const int r = vi / (DH / 8), c = vi - r * (DH / 8);
        *reinterpret_cast<u32x4*>(&sK[r * LDK + c * 8]) = rk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < NVV; ++i) {
      const int vi = tid + NT * i;
      if (VV % NT == 0 || vi < VV) {
        const int r = vi / (KT / 8), c = vi - r * (KT / 8);
        u32x2* dst = reinterpret_cast<u32x2*>(&sV[r * LDV + c * 8]);  // 8-byte aligned rows
        dst[0] = u32x2{rv[i][0], rv[i][1]};
        dst[1] = u32x2{rv[i][2], rv[i][3]};
      }
    }
  };

  // Softmax with a fixed per-row reference m_ref: probabilities are
  // exp2(s - m_ref) and may exceed 1 by up to 2^kHeadroom, which fp32 sums
  // and bf16 probabilities represent exactly as well as values below 1.  The
  // inner loop touches the accumulators only through MFMAs; when a row's
  // score would pass the headroom (always on the first tile, rarely later)
  // the loop stops, the accumulators are rescaled once and the same tile is
  // processed again against the raised reference.
  const int kt_clamp = max(kt_begin, kt_end - 1);
  load_tile(kts.tile(min(kt_begin, kt_clamp)));
  int kt = kt_begin;
  bool staged = false;
  float m_pending = -INFINITY;
  while (kt < kt_end) {
    for (; kt < kt_end; ++kt) {
      const int key0 = kts.tile(kt) * KT;
      if (!staged) {
        __syncthreads();  // previous tile fully consumed
        store_tile();
        __syncthreads();
        load_tile(kts.tile(min(kt + 1, kt_clamp)));  // overlaps the MFMA work below
      }
      staged = false;

      // S^T per 16-key half: two chains each (even / odd k steps)
      f32x4 s[2][2] = {{f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}},
                       {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}}};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const bf16x8 kf = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u16x8*>(&sK[(16 * h + l16) * LDK + 32 * ks + 8 * lg]));
          s[h][ks & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], s[h][ks & 1], 0, 0, 0);
        }
      // sc[e] (e < 4): key 4 lg + e;  sc[4 + e]: key 16 + 4 lg + e
      float sc[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sc[e] = s[0][0][e] + s[0][1][e];
        sc[4 + e] = s[1][0][e] + s[1][1][e];
      }
      const bool inside = key0 + KT <= P || (key0 >= klo && key0 + KT <= khi);
      if (!__all(inside)) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int key = key0 + 16 * (e >> 2) + 4 * lg + (e & 3);
          if (!(key < P || (key >= klo && key < khi))) sc[e] = -INFINITY;
        }
      }
      float mt = sc[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) mt = fmaxf(mt, sc[e]);
      mt = max_xor16_32(mt) * sl2;
      if (m_run == -INFINITY) m_run = mt;
      if (__any(mt > m_run + kHeadroom)) {
        m_pending = mt;
        staged = true;
        break;
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      float ls = 0.f;
      u16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[e], sl2, -m_use));  // see attn16d_kernel
        ls += p;
        pb[e] = f32_to_bf16(p);
      }
      l_run += sum_xor16_32(ls);
      const bf16x8 pf = __builtin_bit_cast(bf16x8, pb);
      // O^T (dh x queries) += V^T P^T: dh row 16 dt + l16, keys 4 lg + 0..3
      // and 16 + 4 lg + 0..3
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const T* vr = &sV[(16 * dt + l16) * LDV + 4 * lg];
        const u16x4 lo = *reinterpret_cast<const u16x4*>(vr);
        const u16x4 hi = *reinterpret_cast<const u16x4*>(vr + 16);
        const bf16x8 vf = __builtin_bit_cast(
            bf16x8, u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, acc[dt], 0, 0, 0);
      }
    }
    if (staged) {
      const float m_new = m_pending > m_run + kHeadroom ? m_pending : m_run;
      const float alpha = m_run == -INFINITY ? 0.f : exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[dt] *= alpha;
      m_run = m_new;
    }
  }

  // Normalised output through LDS: lane (query l16, group lg) holds dh
  // 16 dt + 4 lg + 0..3; rows then go out whole, 16 bytes per lane.
  const size_t R = (size_t)a.B * a.tokens * a.n_q_heads;
  {
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
    T* so = sO[wave];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      u16x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = f32_to_bf16(acc[dt][i] * inv);
      *reinterpret_cast<u16x4*>(so + l16 * LDK + 16 * dt + 4 * lg) = w;
    }
    if (a.n_split > 1 && lg == 0 && valid) {
      const size_t grow = (size_t)(b * a.tokens + tok) * a.n_q_heads + head;
      a.part_ml[((size_t)split * R + grow) * 2 + 0] = m_run;
      a.part_ml[((size_t)split * R + grow) * 2 + 1] = l_run;
    }
  }
  __syncthreads();
  {
    constexpr int CPR = DH / 8;  // 16-byte chunks per row
    const T* so = sO[wave];
    for (int idx = lane; idx < 16 * CPR; idx += 64) {
      const int row = idx / CPR, c = idx - row * CPR;
      const int rq2 = tile0 + 16 * wave + row;
      if (rq2 < rows_bg) {
        const int tok2 = rq2 / G;
        const int head2 = g * G + (rq2 - tok2 * G);
        const size_t grow2 = (size_t)(b * a.tokens + tok2) * a.n_q_heads + head2;
        T* orow = a.n_split == 1
                      ? reinterpret_cast<T*>(a.o) + grow2 * DH
                      : reinterpret_cast<T*>(a.part_o) + ((size_t)split * R + grow2) * DH;
        *reinterpret_cast<u32x4*>(orow + 8 * c) =
            *reinterpret_cast<const u32x4*>(so + row * LDK + 8 * c);
      }
    }
  }
}

// bf16 kernel for head dims 128 and 256 with the K and V^T tiles brought
// straight from memory into LDS (direct-to-LDS loads, no staging registers)
// through a ring of NS tile stages: NS - 1 tiles are in flight while one is
// multiplied, and one barrier per tile (after which the stage of the
// previous tile is refilled) replaces the two of the register-staged kernel.
// Same rows, softmax, masking and output as attn16_kernel, with two layout
// changes that the direct loads need (they write 1 KB runs of LDS, so rows
// cannot be padded):
//  * The score MFMA's A-operand row i of half h holds key 8 (i / 4) + 4 h +
//    i % 4, so a lane's 8 probabilities are keys 8 lg .. 8 lg + 7 in order
//    and its V^T operand is one 16-byte piece of a V^T row.
//  * 16-byte piece c of K row r is stored at c ^ ((r % 4) + 4 ((r / 8) % 4))
//    and piece c of V^T row r at c ^ ((r / 4) % 4); the 16 rows one
//    fragment read touches then fall on 16 different bank groups.
template <int DH, int NWV, int NS>
__global__ __launch_bounds__(64 * NWV) void attn16d_kernel(AttnArgs a) {
  using T = bf16_t;
  constexpr int KT = 32;                     // keys per tile
  constexpr int NT = 64 * NWV;               // threads
  constexpr int RB = 16 * NWV;               // query rows per block
  constexpr int NKS = DH / 32, NDT = DH / 16;
  constexpr int NKF = 2 * NKS;               // K fragments per tile
  constexpr int DK = NKF < 8 ? NKF : 8, DV = NDT < 8 ? NDT : 8;  // read-ahead depths
  constexpr int KCH = DH / 8;                // 16-byte pieces per K row
  constexpr int KBYTES = KT * DH * 2, VBYTES = DH * KT * 2;
  constexpr int STAGE = KBYTES + VBYTES;
  constexpr int NI = STAGE / 16 / NT;        // direct loads per thread per stage
  constexpr int LDO = DH + 8;                // output staging pitch (elements)
  static_assert(DH == 128 || DH == 256, "swizzle is laid out for 16 or 32 pieces per K row");
  static_assert(NI * NT * 16 == STAGE && KBYTES % 1024 == 0, "stage split");
  static_assert(NWV * 16 * LDO * 2 <= NS * STAGE, "output staging fits in the ring");
  extern __shared__ __attribute__((aligned(16))) T attn_ring[];
  unsigned char* ring = reinterpret_cast<unsigned char*>(attn_ring);

  Prefetch<2, NT> pre;  // the output projection's weights, into the memory-side cache
  pre.issue(a.pf, a.pf_bytes, a.len);
  const int G = a.n_q_heads / a.n_kv_heads;
  const int rows_bg = a.tokens * G;
  int rtile, bg;
  attn_block_of(rtile, bg, a.bg_order);
  const int tile0 = rtile * RB;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int split = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int P = a.len[b];
  const int C = a.chunk_len;
  const int l16 = lane & 15, lg = lane >> 4;

  const int K = a.tokens / C;
  const int first = K - a.n_valid[b];
  const int rq = tile0 + 16 * wave + l16;
  const bool valid = rq < rows_bg;
  const int rqc = valid ? rq : rows_bg - 1;
  const int tok = rqc / G;
  const int head = g * G + (rqc - tok * G);
  int klo, khi;  // this row's visible buffer keys [klo, khi); prefix keys [0, P)
  visible_chunks(tok / C, K, first, a.mask_mode, klo, khi);
  klo = buffer_row0(P) + C * klo;
  khi = buffer_row0(P) + C * khi;
  const int rlast = min(tile0 + RB - 1, rows_bg - 1);
  const KeyTiles kts = key_tiles(P, C, K, first, a.mask_mode, tile0 / G, rlast / G, KT);
  const int kt_begin = (split * kts.n) / a.n_split, kt_end = ((split + 1) * kts.n) / a.n_split;

  bf16x8 qf[NKS];
  {
    const T* qrow = reinterpret_cast<const T*>(a.q) +
                    ((size_t)(b * a.tokens + tok) * a.n_q_heads + head) * DH;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(qrow + 32 * ks + 8 * lg));
  }
  f32x4 acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const T* kbase = reinterpret_cast<const T*>(a.karena) +
                   ((size_t)b * a.n_kv_heads + g) * (size_t)a.S * DH;
  const T* vbase = reinterpret_cast<const T*>(a.vtarena) +
                   ((size_t)b * a.n_kv_heads + g) * (size_t)DH * a.S;
  const float sl2 = 1.4426950408889634f / sqrtf((float)DH);

  // The thread's piece of each of its direct loads: unit u of a stage is K
  // (row, piece) for u < KBYTES / 16, else V^T (row, piece); offsets exclude
  // the tile's first key.  Every load instruction is all-K or all-V^T.
  int off[NI];
  bool isk[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int u = 64 * (NI * wave + i) + lane;
    isk[i] = u < KBYTES / 16;
    if (isk[i]) {
      const int r = u / KCH, c = (u % KCH) ^ ((r & 3) | (((r >> 3) & 3) << 2));
      off[i] = r * DH + 8 * c;
    } else {
      const int v = u - KBYTES / 16;
      const int r = v >> 2, c = (v & 3) ^ ((r >> 2) & 3);
      off[i] = r * a.S + 8 * c;
    }
  }
  auto issue = [&](int vt, int stage) __attribute__((always_inline)) {
    const int key0 = kts.tile(vt) * KT;
    unsigned char* st = ring + stage * STAGE + 1024 * NI * wave;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const T* src = isk[i] ? kbase + (size_t)key0 * DH + off[i] : vbase + key0 + off[i];
      lds_dma16_attn(src, st + 1024 * i);
    }
  };
  // fragment addresses within a stage
  const int krow = 8 * (l16 >> 2) + (l16 & 3);  // K row of A-operand row l16, half 0
  // its piece swizzle is l16 for both halves; V^T rows 16 dt + l16 share (l16 / 4) % 4
  const int vpiece = lg ^ ((l16 >> 2) & 3);

  for (int p = 0; p < NS - 1; ++p)
    if (kt_begin + p < kt_end) issue(kt_begin + p, p);
  // the query loads, issued before the tiles, have landed once at most the
  // tiles' loads are outstanding (vector memory counts retire in order)
  if (kt_end - kt_begin >= NS - 1)
    wait_vmcnt_attn<(NS - 1) * NI>();
  else
    wait_vmcnt_attn<0>();
  int kt = kt_begin, stage = 0;
  bool staged = false;
  float m_pending = -INFINITY;
  while (kt < kt_end) {
    for (; kt < kt_end; ++kt) {
      const int key0 = kts.tile(kt) * KT;
      if (!staged) {
        // this wave's loads of tile kt landed (later tiles may still fly) and
        // its reads of tile kt - 1 completed; after the barrier both hold for
        // every wave, so tile kt - 1's stage takes tile kt + NS - 1
        if (kt + NS - 2 < kt_end)
          wait_vmcnt_attn<(NS - 2) * NI>();
        else
          wait_vmcnt_attn<0>();
        wait_lgkmcnt0_attn();
        __builtin_amdgcn_s_barrier();
        if (kt + NS - 1 < kt_end) issue(kt + NS - 1, stage == 0 ? NS - 1 : stage - 1);
      }
      staged = false;
      const unsigned char* sk = ring + stage * STAGE;
      const unsigned char* sv = sk + KBYTES;

      // K fragment idx = 2 ks + h and V^T fragment dt are read DK / DV ahead
      // of their MFMA from register rings; the first V^T reads are issued
      // before the softmax arithmetic, which hides their latency
      auto kread = [&](int idx) __attribute__((always_inline)) {
        return __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u16x8*>(sk + (krow + 4 * (idx & 1)) * (2 * DH) +
                                                    16 * ((4 * (idx >> 1) + lg) ^ l16)));
      };
      auto vread = [&](int dt) __attribute__((always_inline)) {
        return __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u16x8*>(sv + (16 * dt + l16) * 64 + 16 * vpiece));
      };
      bf16x8 kf[DK];
#pragma unroll
      for (int i = 0; i < DK; ++i) kf[i] = kread(i);
      f32x4 s[2][2] = {{f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}},
                       {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}}};
#pragma unroll
      for (int idx = 0; idx < NKF; ++idx) {
        const int ks = idx >> 1, h = idx & 1;
        s[h][ks & 1] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[idx % DK], qf[ks], s[h][ks & 1], 0, 0, 0);
        if (idx + DK < NKF) kf[idx % DK] = kread(idx + DK);
      }
      bf16x8 vf[DV];
#pragma unroll
      for (int i = 0; i < DV; ++i) vf[i] = vread(i);
      // issue order: DK reads, then one read (K, then the first V^T) after
      // each score MFMA
      static_assert(NKF - DK + DV == NKF, "one read per score MFMA");
      __builtin_amdgcn_sched_group_barrier(0x100, DK, 0);
#pragma unroll
      for (int i = 0; i < NKF; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      // sc[e]: key key0 + 8 lg + e
      float sc[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sc[e] = s[0][0][e] + s[0][1][e];
        sc[4 + e] = s[1][0][e] + s[1][1][e];
      }
      const bool inside = key0 + KT <= P || (key0 >= klo && key0 + KT <= khi);
      if (!__all(inside)) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int key = key0 + 8 * lg + e;
          if (!(key < P || (key >= klo && key < khi))) sc[e] = -INFINITY;
        }
      }
      float mt = sc[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) mt = fmaxf(mt, sc[e]);
      mt = max_xor16_32(mt) * sl2;
      if (m_run == -INFINITY) m_run = mt;
      if (__any(mt > m_run + kHeadroom)) {
        m_pending = mt;
        staged = true;
        break;
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      float ls = 0.f;
      u16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // raw hardware exp2: a probability below 2^-126 (flushed to 0) is
        // negligible against the row's sum
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[e], sl2, -m_use));
        ls += p;
        pb[e] = f32_to_bf16(p);
      }
      l_run += sum_xor16_32(ls);
      const bf16x8 pf = __builtin_bit_cast(bf16x8, pb);
      // O^T (dh x queries) += V^T P^T: dh row 16 dt + l16, keys 8 lg .. 8 lg + 7
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[dt % DV], pf, acc[dt], 0, 0, 0);
        if (dt + DV < NDT) vf[dt % DV] = vread(dt + DV);
      }
      stage = stage + 1 == NS ? 0 : stage + 1;
    }
    if (staged) {
      const float m_new = m_pending > m_run + kHeadroom ? m_pending : m_run;
      const float alpha = m_run == -INFINITY ? 0.f : exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[dt] *= alpha;
      m_run = m_new;
    }
  }

  // Normalised output through LDS (the ring, free once every wave is past
  // its last tile): lane (query l16, group lg) holds dh 16 dt + 4 lg + 0..3;
  // rows then go out whole, 16 bytes per lane.
  const size_t R = (size_t)a.B * a.tokens * a.n_q_heads;
  __syncthreads();
  T* so = attn_ring + wave * 16 * LDO;
  {
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      u16x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = f32_to_bf16(acc[dt][i] * inv);
      *reinterpret_cast<u16x4*>(so + l16 * LDO + 16 * dt + 4 * lg) = w;
    }
    if (a.n_split > 1 && lg == 0 && valid) {
      const size_t grow = (size_t)(b * a.tokens + tok) * a.n_q_heads + head;
      a.part_ml[((size_t)split * R + grow) * 2 + 0] = m_run;
      a.part_ml[((size_t)split * R + grow) * 2 + 1] = l_run;
    }
  }
  wait_lgkmcnt0_attn();  // the wave reads back only its own rows
  {
    constexpr int CPR = DH / 8;  // 16-byte chunks per row
    for (int idx = lane; idx < 16 * CPR; idx += 64) {
      const int row = idx / CPR, c = idx - row * CPR;
      const int rq2 = tile0 + 16 * wave + row;
      if (rq2 < rows_bg) {
        const int tok2 = rq2 / G;
        const int head2 = g * G + (rq2 - tok2 * G);
        const size_t grow2 = (size_t)(b * a.tokens + tok2) * a.n_q_heads + head2;
        T* orow = a.n_split == 1
                      ? reinterpret_cast<T*>(a.o) + grow2 * DH
                      : reinterpret_cast<T*>(a.part_o) + ((size_t)split * R + grow2) * DH;
        *reinterpret_cast<u32x4*>(orow + 8 * c) =
            *reinterpret_cast<const u32x4*>(so + row * LDO + 8 * c);
      }
    }
  }
  pre.retire();
}

// Merge of split partials in split order.  Partial z holds o_z = acc_z / l_z
// (stored in the element type) with its reference m_z and sum l_z:
// o = sum_z 2^(m_z - M) l_z o_z / sum_z 2^(m_z - M) l_z.  One wave per row; a
// lane owns 4 consecutive features.
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_combine(const T* __restrict__ part_o,
                                                    const float* __restrict__ part_ml,
                                                    T* __restrict__ o, int R, int n_split) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= R) return;
  // every load of the row is issued before any is used (n_split <= 8), with
  // no condition on the loads themselves: slots z >= n_split re-read split
  // n_split - 1 and get weight 0, features past DH re-read the last group and
  // are not stored (a conditional load makes the compiler wait for each one)
  float mz[8], lz[8];
  f32x2 ml[8];
#pragma unroll
  for (int z = 0; z < 8; ++z)
    ml[z] = *reinterpret_cast<const f32x2*>(part_ml + ((size_t)min(z, n_split - 1) * R + row) * 2);
  constexpr int NV = (DH + 255) / 256;  // 4-feature groups per lane
  f32x4 pv[8][NV];
#pragma unroll
  for (int z = 0; z < 8; ++z)
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int d = min(4 * lane + 256 * v, DH - 4);
      pv[z][v] = load4_f32(part_o + ((size_t)min(z, n_split - 1) * R + row) * DH + d);
    }
#pragma unroll
  for (int z = 0; z < 8; ++z) {
    mz[z] = ml[z][0];
    lz[z] = z < n_split ? ml[z][1] : 0.f;
  }
  float M = -INFINITY;
#pragma unroll
  for (int z = 0; z < 8; ++z) M = fmaxf(M, mz[z]);
  float den = 0.f;
#pragma unroll
  for (int z = 0; z < 8; ++z) {
    mz[z] = lz[z] > 0.f ? exp2f(mz[z] - M) * lz[z] : 0.f;  // weight of split z
    den += mz[z];
  }
  const float inv = 1.0f / den;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int d = 4 * lane + 256 * v;
    if (d >= DH) continue;
    f32x4 num = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int z = 0; z < 8; ++z) num += mz[z] * pv[z][v];
    store4<T>(o + (size_t)row * DH + d, num[0] * inv, num[1] * inv, num[2] * inv, num[3] * inv);
  }
}

template <typename T, int DH>
void launch_dh(const AttnArgs& a, hipStream_t s, int parts) {
  // 32-key tiles keep wide heads (and fp32) within the register file
  constexpr int KT = (sizeof(T) == 2 && DH < 192) ? 64 : 32;
  const int G = a.n_q_heads / a.n_kv_heads;
  constexpr int RB = rows_per_block<T>();
  dim3 grid((a.tokens * G + RB - 1) / RB, a.B * a.n_kv_heads, a.n_split);
  if (parts & 1) {
    if constexpr (sizeof(T) == 2 && (DH == 128 || DH == 256))
      hipLaunchKernelGGL((attn16d_kernel<DH, kAttn16Waves, kAttnStages>), grid,
                         dim3(64 * kAttn16Waves), (attn16d_lds<DH>()), s, a);
    else if constexpr (sizeof(T) == 2)
      hipLaunchKernelGGL((attn16_kernel<DH, kAttn16Waves>), grid, dim3(64 * kAttn16Waves), 0, s, a);
    else
      hipLaunchKernelGGL((attn_kernel<T, DH, KT, kRG>), grid, dim3(256), 0, s, a);
  }
  if (a.n_split > 1 && (parts & 2)) {
    const int R = a.B * a.tokens * a.n_q_heads;
    hipLaunchKernelGGL((attn_combine<T, DH>), dim3((R + 3) / 4), dim3(256), 0, s,
                       reinterpret_cast<const T*>(a.part_o), a.part_ml,
                       reinterpret_cast<T*>(a.o), R, a.n_split);
  }
}

}  // namespace

void die_order(const int* len, int B, int Hkv, int* order) {
  const int n = B * Hkv;
  for (int i = 0; i < n; ++i) order[i] = i;
  if (n % 8 || n < 8) return;
  // longest first, each to the least-loaded die with room left
  std::vector<int> byl(order, order + n);
  std::stable_sort(byl.begin(), byl.end(),
                   [&](int x, int y) { return len[x / Hkv] > len[y / Hkv]; });
  const int cap = n / 8;
  std::vector<std::vector<int>> die(8);
  std::vector<long> load(8, 0);
  for (int bg : byl) {
    int best = -1;
    for (int d = 0; d < 8; ++d)
      if ((int)die[d].size() < cap && (best < 0 || load[d] < load[best])) best = d;
    die[best].push_back(bg);
    load[best] += len[bg / Hkv];
  }
  int k = 0;
  for (int d = 0; d < 8; ++d)
    for (int bg : die[d]) order[k++] = bg;
}

template <typename T>
int attention_row_tiles(int tokens, int n_q_heads, int n_kv_heads) {
  constexpr int RB = rows_per_block<T>();
  return (tokens * (n_q_heads / n_kv_heads) + RB - 1) / RB;
}

template <typename T>
void launch_attention(const AttnArgs& a, hipStream_t s, int parts) {
  switch (a.head_dim) {
    case 64: launch_dh<T, 64>(a, s, parts); break;
    case 128: launch_dh<T, 128>(a, s, parts); break;
    case 192: launch_dh<T, 192>(a, s, parts); break;
    case 256: launch_dh<T, 256>(a, s, parts); break;
    default: break;  // rejected at fv_create
  }
}

// The direct-load kernels' dynamic LDS exceeds the default limit.
hipError_t attention_prepare() {
  hipError_t e = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&attn16d_kernel<128, kAttn16Waves, kAttnStages>),
      hipFuncAttributeMaxDynamicSharedMemorySize, attn16d_lds<128>());
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(
      reinterpret_cast<const void*>(&attn16d_kernel<256, kAttn16Waves, kAttnStages>),
      hipFuncAttributeMaxDynamicSharedMemorySize, attn16d_lds<256>());
}

template void launch_attention<bf16_t>(const AttnArgs&, hipStream_t, int);
template void launch_attention<float>(const AttnArgs&, hipStream_t, int);
template int attention_row_tiles<bf16_t>(int, int, int);
template int attention_row_tiles<float>(int, int, int);

}  // namespace fv
