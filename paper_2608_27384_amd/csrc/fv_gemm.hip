// MFMA GEMMs of the action expert with fused epilogues.
//
// Every linear layer of the expert (time-MLP, FiLM maps, packed QKV, output
// projection, packed gate/up, down projection) is C = A * W with A the
// activations [M][K] (row-major) and W stored output-major as Bt [N][K].
//
// Two main loops.  The bf16 tiles 256x256, 128x128 and 64x128 use
// gemm_dma_kernel: k-tiles go from memory straight into a ring of LDS stages
// with the direct-to-LDS loads (see there).  The fp32 tiles and the small-M
// 32x128 tile use gemm_kernel, described here, and M <= 16 time-MLP layers a
// GEMV.
//
// gemm_kernel block: NW waves (2, 4 or 8).  Tile BM x BN; k is staged through
// LDS 128 bytes per row (64 bf16 / 32 fp32) at a time in two buffers.  While a wave
// multiplies the tile in one buffer with 32x32 MFMA instructions, the
// registers holding the next tile are written to the other buffer piece by
// piece between k-steps, and every freed register piece immediately issues
// its global load of the tile after that; the MFMA operands of the next
// k-step are read from LDS while the current k-step's MFMAs run, and the
// instruction order interleaves MFMAs with those reads, stores and loads.
// One barrier per k-tile.  Rows of A beyond M re-read row M-1 (never
// stored).  Large grids walk their tiles in an order that keeps the blocks
// each of the chip's 8 dies runs together on shared operands.
//
// Split-K (KS > 1): block z of a tile accumulates k-tiles [z*nk/KS,
// (z+1)*nk/KS) and writes its partial tile to a workspace; a second, small
// kernel sums the KS partials of each tile in split order (so the result
// does not depend on scheduling) and runs the epilogue.  The partials are
// fp32, except those of the direct-to-LDS kernel with no epilogue (EpiNone,
// the output and down projections), which are bf16 and are summed by the
// fused residual reduction (resid_norm_kernel).  The kernel
// boundary makes the partials visible across the chip's separate L2 caches
// without device-wide cache flushes inside the GEMM.
//
// Epilogues consume the accumulators in registers:
//  * bias + SiLU (time-MLP), bias to fp32 (FiLM maps);
//  * QKV: queries and keys are rotated (half-split rotary pairs) and keys and
//    values are written straight into the layer's K / V^T arena at row
//    buffer_row0(len[b]) + token (the prefix length rounded up to 8), so
//    attention reads [prefix ; buffer] from one arena;
//  * gated residual h += gate[chunk] * acc;
//  * GeGLU gelu(g) * u and plain GELU.
// Element-type outputs of the QKV and GELU epilogues are transposed within
// each group of four lanes first, so a lane stores four consecutive columns
// of one row at once.
// Paired epilogues rely on the weight packing: columns [64p, 64p+32) and
// [64p+32, 64p+64) of a packed matrix hold the two partners of a pair, which
// then sit in the same lane and register of two adjacent 32-column tiles.
#include <type_traits>

#include "fv_internal.h"

namespace fv {

namespace {

// 32x32 MFMA per element type: bf16 32x32x16 (8 k per lane), fp32 32x32x2
// (1 k per lane).  Output layout (both): lane l, register r holds
// row 8*(r/4) + 4*(l/32) + r%4, column l%32 of the 32x32 tile.
template <typename T> struct Mf32;
template <> struct Mf32<bf16_t> {
  static constexpr int KG = 8, KM = 16;
  typedef bf16x8 frag;
  __device__ static __forceinline__ frag load(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(p));
  }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mf32<float> {
  static constexpr int KG = 1, KM = 2;
  typedef float frag;
  __device__ static __forceinline__ frag load(const float* p) { return *p; }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ int acc_row(int r, int lane) {
  return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}

// Registers 4q .. 4q+3 of a 32x32 accumulator hold four consecutive rows of
// the lane's column.  quad_rows transposes each such 4x4 block within its
// group of four lanes: lane l gets back row 8q + 4 (l / 32) + (l & 3) at the
// columns (l & 28) .. (l & 28) + 3 of the 32-column block, so a row's four
// outputs leave as one store instead of four 2-byte ones.  Every lane of the
// wave must be active.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ f32x4 quad_rows(float x0, float x1, float x2, float x3, int lane) {
  const bool b0 = lane & 1, b1 = lane & 2;
  // lanes l, l^1 trade: each then holds two adjacent columns of the rows
  // (l & 1) and 2 + (l & 1)
  const float r1 = dpp_mov<0xB1>(b0 ? x0 : x1);  // quad_perm [1,0,3,2]
  const float r2 = dpp_mov<0xB1>(b0 ? x2 : x3);
  const float z0 = b0 ? r1 : x0, z1 = b0 ? x1 : r1;
  const float z2 = b0 ? r2 : x2, z3 = b0 ? x3 : r2;
  // lanes l, l^2 trade column pairs
  const float t1 = dpp_mov<0x4E>(b1 ? z0 : z2);  // quad_perm [2,3,0,1]
  const float t2 = dpp_mov<0x4E>(b1 ? z1 : z3);
  return b1 ? f32x4{t1, t2, z2, z3} : f32x4{z0, z1, t1, t2};
}
// store of the four transposed values at p (4-element aligned when `vec`)
template <typename T>
__device__ __forceinline__ void store_quad(T* p, const f32x4& u, bool vec) {
  if (vec) {
    store4<T>(p, u[0], u[1], u[2], u[3]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] = from_f32<T>(u[e]);
  }
}

// Output tile of this block.  Block b of a launch runs on XCD b % 8 (the
// chip's 8 dies, each with its own L2).  When the grid is large enough, the
// (x, y) block index is remapped so that each die takes a contiguous range
// of tiles, walked in groups kTileGroup row panels tall, column by column:
// the tiles a die runs together then share A row panels and weight column
// blocks in its L2 instead of fetching them from memory once per die.
// Split-K grids (gridDim.z k slices dividing the 8 dies) give each die one
// k slice and a contiguous range of its column blocks, every row tile of
// them: a die then fetches its slice of A and its share of the weights, not
// the whole A of every slice.
constexpr int kTileGroup = 8;
__device__ __forceinline__ void tile_of(int& tm, int& tn, int& kz) {
  const int nN = gridDim.x, nM = gridDim.y, nK = gridDim.z, nb = nN * nM;
  kz = blockIdx.z;
  if (nK > 1 && 8 % nK == 0 && nN % (8 / nK) == 0) {
    const int dpk = 8 / nK;  // dies per k slice
    const int lin = (blockIdx.z * nM + blockIdx.y) * nN + blockIdx.x;
    const int x = lin & 7, s = lin >> 3;
    kz = x / dpk;
    tm = s % nM;
    tn = (x % dpk) * (nN / dpk) + s / nM;
    return;
  }
  if (nb < 64) {
    tm = blockIdx.y;
    tn = blockIdx.x;
    return;
  }
  const int b = blockIdx.y * nN + blockIdx.x;
  const int per = nb >> 3, rem = nb & 7;  // dies x < rem take per + 1 tiles
  const int x = b & 7, s = b >> 3;
  const int L = x * per + min(x, rem) + s;
  const int gsz = kTileGroup * nN;
  const int g = L / gsz, i = L - g * gsz;
  const int gm = min(kTileGroup, nM - g * kTileGroup);
  tm = g * kTileGroup + i % gm;
  tn = i / gm;
}

// Epilogues with a run-time skip flag (Epi::skipped()): the whole launch
// returns at once when it is set (every workgroup reads the same flag).
template <class Epi, class = void>
struct EpiSkip {
  __device__ static bool skip(const Epi&) { return false; }
};
template <class Epi>
struct EpiSkip<Epi, std::void_t<decltype(&Epi::skipped)>> {
  __device__ static bool skip(const Epi& e) { return e.skipped(); }
};

template <typename T, int BM, int BN, int NW, int WGM, int KG, class Epi>
__global__ __launch_bounds__(64 * NW * KG) void gemm_kernel(const T* __restrict__ A,
                                                            const T* __restrict__ Bt, int M,
                                                            int N, int K, int KS,
                                                            float* __restrict__ ws, Epi epi) {
  if (EpiSkip<Epi>::skip(epi)) return;
  using MF = Mf32<T>;
  constexpr int NT = 64 * NW * KG;
  constexpr int WGN = NW / WGM;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int EPV = 16 / (int)sizeof(T);  // elements per 16-byte vector
  constexpr int BK = 8 * EPV;               // 128 bytes of k per row and stage
  constexpr int LDR = BK + EPV;             // LDS row pitch (one vector of padding)
  constexpr int NA = BM * 8 / NT, NB = BN * 8 / NT, NP = NA + NB;  // 16-byte pieces per thread
  constexpr int NSTEP = BK / MF::KM;        // k-steps per stage
  constexpr int NSG = NSTEP / KG;           // k-steps of a stage per wave group
  static_assert(FM >= 1 && FN >= 1 && WGM * WGN == NW, "bad tile");
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0 && NSG % 2 == 0, "bad tile");
  static_assert(KG == 1 || NW * FM * FN * 4096 <= 2 * (BM + BN) * LDR * (int)sizeof(T),
                "k-group reduction does not fit the staging buffers");

  __shared__ __attribute__((aligned(16))) T sm[2 * (BM + BN) * LDR];  // [buf][A rows ; B rows]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = wave / NW, wv = wave - kg * NW;  // k-group; wave within the group
  const int wm = wv % WGM, wn = wv / WGM;
  int tm, tn, kz;
  tile_of(tm, tn, kz);
  const int m0 = tm * BM, n0 = tn * BN;
  const int arow = wm * WTM, brow = BM + wn * WTN;  // fragment rows in the stage
  const int nk_all = K / BK;
  const int kt0 = (kz * nk_all) / KS, kt1 = ((kz + 1) * nk_all) / KS;
  const int klast = (kt1 - 1) * BK;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};

  // Thread piece p: 16 bytes of row r, k-vector c of a stage (A rows first).
  const T* gp[NP];
  int lp[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const bool isa = p < NA;
    const int vi = tid + NT * (isa ? p : p - NA);
    const int r = vi >> 3, c = vi & 7;
    gp[p] = isa ? A + (size_t)min(m0 + r, M - 1) * K + c * EPV
                : Bt + (size_t)(n0 + r) * K + c * EPV;
    lp[p] = (isa ? r : BM + r) * LDR + c * EPV;
  }

  // Prologue: stage kt0 into LDS buffer 0, stage kt0+1 into registers.
  u32x4 rg[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) rg[p] = *reinterpret_cast<const u32x4*>(gp[p] + kt0 * BK);
#pragma unroll
  for (int p = 0; p < NP; ++p) *reinterpret_cast<u32x4*>(&sm[lp[p]]) = rg[p];
  {
    const int k1 = min((kt0 + 1) * BK, klast);
#pragma unroll
    for (int p = 0; p < NP; ++p) rg[p] = *reinterpret_cast<const u32x4*>(gp[p] + k1);
  }
  __syncthreads();

  // Fragments are double-buffered: those of k-step ks+1 are read while the
  // MFMAs of k-step ks run.  The next stage's register pieces go to the
  // other LDS buffer during a group's k-steps 0..NSG-2 (each freed register
  // then loads its piece of the stage after that); one barrier, placed
  // before the group's last k-step, publishes the new stage, whose first
  // fragments are read while the last k-step's MFMAs run.  With KG = 2 the
  // two wave groups take the first and second half of every stage's k-steps
  // on the same output tile (twice the waves per CU, and so twice the LDS
  // requests in flight, for the same LDS bytes) and their accumulators are
  // summed through LDS at the end.
  const int lr = lane & 31, lk = MF::KG * (lane >> 5);
  typename MF::frag af[2][FM], bfr[2][FN];
  auto read_frags = [&](int slot, int buf, int ks) __attribute__((always_inline)) {
    const T* base = sm + buf * (BM + BN) * LDR + ks * MF::KM + lk;
#pragma unroll
    for (int i = 0; i < FM; ++i) af[slot][i] = MF::load(base + (arow + 32 * i + lr) * LDR);
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[slot][j] = MF::load(base + (brow + 32 * j + lr) * LDR);
  };
  const int s0 = kg * NSG;
  read_frags(0, 0, s0);
  for (int kt = kt0; kt < kt1; ++kt) {
    const int cur = (kt - kt0) & 1;
    const int knext = min((kt + 2) * BK, klast);  // unconditional prefetch (clamped)
    T* const nxt = sm + (cur ^ 1) * (BM + BN) * LDR;
#pragma unroll
    for (int ks = 0; ks < NSG; ++ks) {
      const int cb = ks & 1;
      if (ks + 1 < NSG) {
        read_frags(cb ^ 1, cur, s0 + ks + 1);
      } else {
        __syncthreads();
        read_frags(cb ^ 1, cur ^ 1, s0);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = MF::mma(af[cb][i], bfr[cb][j], acc[i][j]);
      int nw = 0;
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        if (ks + 1 == NSG || (p * (NSG - 1)) / NP != ks) continue;
        *reinterpret_cast<u32x4*>(&nxt[lp[p]]) = rg[p];
        rg[p] = *reinterpret_cast<const u32x4*>(gp[p] + knext);
        ++nw;
      }
      // issue order: one fragment read after each MFMA, then one LDS store
      // and one global load per MFMA, then the remaining MFMAs
      constexpr int nrd = FM + FN < FM * FN ? FM + FN : FM * FN;
#pragma unroll
      for (int q = 0; q < nrd; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        if (q < nw && nrd + q < FM * FN) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
      }
#pragma unroll
      for (int q = 0; q < FM * FN; ++q)
        if (q >= nrd + nw) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  }
  if constexpr (KG > 1) {
    // group kg > 0 hands its sums to group 0 through the (now idle) staging
    // buffers: [wave][i][j][register quad][lane][4], 16 bytes per lane
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(sm);
    for (int g = 1; g < KG; ++g) {
      if (kg == g) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              red[(((wv * FM + i) * FN + j) * 4 + q) * 64 + lane] =
                  f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                        acc[i][j][4 * q + 3]};
      }
      __syncthreads();
      if (kg == 0) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const f32x4 v = red[(((wv * FM + i) * FN + j) * 4 + q) * 64 + lane];
#pragma unroll
              for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += v[e];
            }
      }
      if (g + 1 < KG) __syncthreads();
    }
    if (kg != 0) return;
  }
  const int ar = wm * WTM, bc = wn * WTN;

  if (KS > 1) {
    // Partial tile -> workspace, row-major [KS][M][N] fp32 (lanes of a row
    // write 32 consecutive columns); summed in split order afterwards.
    float* part = ws + (size_t)kz * M * N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + bc + 32 * j + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + ar + 32 * i + acc_row(r, lane);
          if (row < M) part[(size_t)row * N + col] = acc[i][j][r];
        }
      }
    return;
  }
  epi.template apply<FM, FN>(acc, m0 + ar, n0 + bc, lane, M);
}

// Epilogues with an LDS-staged form (Epi::kStaged) use it in the direct-to-LDS
// kernel, whose stage buffers are free after the main loop.
template <class Epi, class = void>
struct EpiStaged { static constexpr bool value = false; };
template <class Epi>
struct EpiStaged<Epi, std::void_t<decltype(Epi::kStaged)>> { static constexpr bool value = Epi::kStaged; };
template <class Epi>
constexpr bool epi_staged() { return EpiStaged<Epi>::value; }

// ------------------------------------------------- direct-to-LDS bf16 GEMM
// BM x BN output tile per block of NW waves (WGM along M).  The A and W
// k-tiles (64 k = 128 bytes per row) go from memory straight to LDS with the
// direct-to-LDS loads (no staging registers, no LDS store instructions) into
// a ring of NS stages; 16-byte piece c of stage row r sits at piece
// c ^ ((r / 2) % 8), which keeps the MFMA fragment reads conflict-free
// without padding.  One barrier per k-tile, after every wave's last fragment
// reads of the tile; the loads of tile k + NS are issued right after it into
// the stage just consumed, so NS - 1 tiles are in flight while one is
// multiplied.  Fragments of k-step s + LA are read during the MFMAs of
// k-step s (LA = 2 for the 32x64 wave tiles, 1 for 128x64), so the barrier
// comes LA - 1 k-steps before the end of a tile, once the wave has issued
// its last read of it.  Split-K (KS > 1) with EpiNone writes bf16 partials,
// four columns of a row per store (summed in fp32 by resid_norm_kernel);
// with any other epilogue it writes fp32 partials as gemm_kernel does.
//   * 256x256, 8 waves (128x64 wave tiles), 2 stages: large M (batch 64);
//   * 128x128, 8 waves and 64x128, 4 waves (32x64 wave tiles), 3 stages
//     (2 for 128x128 grids of several rounds): medium M (batch 1), where the
//     deeper ring hides the load latency.
__device__ __forceinline__ void lds_dma16(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {  // at most N vector memory ops outstanding
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}

template <int BM, int BN, int NW, int WGM, int NS>
constexpr int dma_lds_bytes() {
  return NS * (BM + BN) * 128;
}

struct EpiNone;  // partials only (split-K feeding the fused residual reduction)

template <int BM, int BN, int NW, int WGM, int NS, class Epi>
__global__ __launch_bounds__(64 * NW) void gemm_dma_kernel(const bf16_t* __restrict__ A,
                                                           const bf16_t* __restrict__ Bt, int M,
                                                           int N, int K, int KS,
                                                           float* __restrict__ ws, Epi epi) {
  if (EpiSkip<Epi>::skip(epi)) return;
  constexpr int WGN = NW / WGM, WTM = BM / WGM, WTN = BN / WGN, FM = WTM / 32, FN = WTN / 32;
  constexpr int BK = 64, NSTEP = 4;
  // k-steps whose fragments are read ahead: two for the 32x64 wave tiles,
  // whose two MFMAs per k-step are shorter than an LDS read (QKV at batch 1
  // 10.4 -> 10.2 us); one where a k-step has 8 MFMAs
  constexpr int LA = FM * FN >= 4 ? 1 : 2;
  constexpr int STAGE = (BM + BN) * 128;        // bytes
  constexpr int NI = (BM + BN) * 8 / (64 * NW);  // direct loads per wave per stage
  static_assert(NI * 64 * NW == (BM + BN) * 8 && FM >= 1 && FN >= 1 && NS >= 2, "bad tile");
  extern __shared__ __attribute__((aligned(16))) bf16_t dma_smem[];
  unsigned char* smem = reinterpret_cast<unsigned char*>(dma_smem);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WGM, wn = wave / WGM;
  int tm, tn;
  int kz;
  tile_of(tm, tn, kz);
  const int m0 = tm * BM, n0 = tn * BN;
  const int nk_all = K / BK;
  const int kt0 = (kz * nk_all) / KS, kt1 = ((kz + 1) * nk_all) / KS;

  // lane's piece of each of the wave's loads: 16-byte unit p of a stage
  const bf16_t* src[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int p = 64 * (NI * wave + i) + lane;
    const int r = p >> 3, c = (p & 7) ^ ((r >> 1) & 7);
    src[i] = r < BM ? A + (size_t)min(m0 + r, M - 1) * K + 8 * c
                    : Bt + (size_t)(n0 + r - BM) * K + 8 * c;
  }
  auto issue = [&](int kt, int stage) __attribute__((always_inline)) {
    unsigned char* st = smem + stage * STAGE + 1024 * NI * wave;
#pragma unroll
    for (int i = 0; i < NI; ++i) lds_dma16(src[i] + (size_t)kt * BK, st + 1024 * i);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};
  const int lr = lane & 31, lg = lane >> 5;
  const int swz = (lr >> 1) & 7;  // rows 32 i + lr of any fragment share it
  const int arow = wm * WTM, brow = BM + wn * WTN;
  // fragment slots: the k-step index within the tile when reading LA > 1
  // steps ahead, else alternate
  constexpr int NSL = LA == 1 ? 2 : NSTEP;
  u32x4 af[NSL][FM], bfr[NSL][FN];
  auto read_frags = [&](int slot, int stage, int ks) __attribute__((always_inline)) {
    const bf16_t* st = reinterpret_cast<const bf16_t*>(smem + stage * STAGE);
    const int co = 8 * ((2 * ks + lg) ^ swz);
#pragma unroll
    for (int i = 0; i < FM; ++i)
      af[slot][i] = *reinterpret_cast<const u32x4*>(st + (arow + 32 * i + lr) * 64 + co);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      bfr[slot][j] = *reinterpret_cast<const u32x4*>(st + (brow + 32 * j + lr) * 64 + co);
  };

#pragma unroll
  for (int p = 0; p < NS; ++p)
    if (kt0 + p < kt1) issue(kt0 + p, p);
  if (kt1 - kt0 >= NS)
    wait_vmcnt<(NS - 1) * NI>();  // tile kt0 landed, the next NS - 1 may be in flight
  else
    wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int p = 0; p < LA; ++p) read_frags(p % NSL, 0, p);
  int stage = 0;
  for (int kt = kt0; kt < kt1; ++kt) {
    const int nstage = stage + 1 == NS ? 0 : stage + 1;
#pragma unroll
    for (int ks = 0; ks < NSTEP; ++ks) {
      const int cb = ks % NSL;
      const int rs = ks + LA;  // k-step read now (rs >= NSTEP: of tile kt + 1)
      if (rs < NSTEP) {
        read_frags(rs % NSL, stage, rs);
      } else {
        if (rs == NSTEP) {
          // this wave's loads of tile kt + 1 landed (later ones may still
          // fly) and its reads of tile kt, all issued by now, completed; after
          // the barrier both hold for every wave, and this stage is free for
          // tile kt + NS
          if (kt + NS - 1 < kt1)
            wait_vmcnt<(NS - 2) * NI>();
          else
            wait_vmcnt<0>();
          wait_lgkmcnt0();
          __builtin_amdgcn_s_barrier();
          if (kt + NS < kt1) issue(kt + NS, stage);
        }
        if (kt + 1 < kt1) read_frags(rs % NSL, nstage, rs - NSTEP);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, af[cb][i]), __builtin_bit_cast(bf16x8, bfr[cb][j]),
              acc[i][j], 0, 0, 0);
      if (rs != NSTEP) {  // one fragment read after each MFMA
        constexpr int nrd = FM + FN < FM * FN ? FM + FN : FM * FN;
#pragma unroll
        for (int q = 0; q < nrd; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
#pragma unroll
        for (int q = nrd; q < FM * FN; ++q) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
    }
    stage = nstage;
  }
  const int ar = wm * WTM, bc = wn * WTN;
  if (KS > 1) {
    if constexpr (std::is_same<Epi, EpiNone>::value) {
      // partials for the fused residual reduction: bf16, four columns of a
      // row per store (the sum over splits and the residual stay fp32)
      bf16_t* part = reinterpret_cast<bf16_t*>(ws) + (size_t)kz * M * N;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = n0 + bc + 32 * j + (lane & 28);
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const f32x4 u = quad_rows(acc[i][j][4 * q4], acc[i][j][4 * q4 + 1],
                                      acc[i][j][4 * q4 + 2], acc[i][j][4 * q4 + 3], lane);
            const int row = m0 + ar + 32 * i + 8 * q4 + 4 * (lane >> 5) + (lane & 3);
            if (row < M) store4<bf16_t>(part + (size_t)row * N + col, u[0], u[1], u[2], u[3]);
          }
        }
    } else {
      float* part = ws + (size_t)kz * M * N;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = n0 + bc + 32 * j + lr;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = m0 + ar + 32 * i + acc_row(r, lane);
            if (row < M) part[(size_t)row * N + col] = acc[i][j][r];
          }
        }
    }
    return;
  }
  if constexpr (epi_staged<Epi>()) {
    __syncthreads();  // every wave is done with the k-tile stages
    epi.template apply_staged<FM, FN, NW, NS * STAGE>(acc, reinterpret_cast<float*>(smem), m0 + ar,
                                                      n0 + bc, lane, wave, M);
  } else {
    epi.template apply<FM, FN>(acc, m0 + ar, n0 + bc, lane, M);
  }
}

// Sum of the KS split partials of each tile, in split order, followed by the
// epilogue; same block shape and register layout as the GEMM that wrote them.
template <int BM, int BN, int NW, int WGM, class Epi>
__global__ __launch_bounds__(64 * NW) void gemm_reduce_kernel(const float* __restrict__ ws, int M,
                                                              int N, int KS, Epi epi) {
  if (EpiSkip<Epi>::skip(epi)) return;
  constexpr int WGN = NW / WGM;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave % WGM, wn = wave / WGM;
  const int row0 = blockIdx.y * BM + wm * WTM, col0 = blockIdx.x * BN + wn * WTN;
  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16{};
  for (int z = 0; z < KS; ++z) {  // split order; loads within a split are independent
    const float* part = ws + (size_t)z * M * N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = col0 + 32 * j + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = min(row0 + 32 * i + acc_row(r, lane), M - 1);
          acc[i][j][r] += part[(size_t)row * N + col];
        }
      }
  }
  epi.template apply<FM, FN>(acc, row0, col0, lane, M);
}

// ----------------------------------------------------------------- epilogues
// Raw split partials only (no epilogue, no reduction); the caller reduces them.
struct EpiNone {
  template <int FM, int FN>
  __device__ void apply(f32x16 (&)[FM][FN], int, int, int, int) const {}
};

// Element (i, j, r) of a wave's accumulators sits at
//   row = row0 + 32 i + acc_row(r, lane),   col = col0 + 32 j + lane % 32.

template <typename T>
struct EpiBiasSilu {
  T* out; const float* bias; int ldo;
  const int* skip;  // nullptr, or a flag that skips the launch when set
  __device__ bool skipped() const { return skip && *skip; }
  template <int FM, int FN>
  __device__ void apply(f32x16 (&acc)[FM][FN], int row0, int col0, int lane, int M) const {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = col0 + 32 * j + (lane & 31);
      const float b = bias[col];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + 32 * i + acc_row(r, lane);
          if (row < M) out[(size_t)row * ldo + col] = from_f32<T>(silu_f(acc[i][j][r] + b));
        }
    }
  }
};

struct EpiBiasF32 {
  float* out; const float* bias; int ldo;
  const int* skip;  // nullptr, or a flag that skips the launch when set
  __device__ bool skipped() const { return skip && *skip; }
  template <int FM, int FN>
  __device__ void apply(f32x16 (&acc)[FM][FN], int row0, int col0, int lane, int M) const {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = col0 + 32 * j + (lane & 31);
      const float b = bias[col];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + 32 * i + acc_row(r, lane);
          if (row < M) out[(size_t)row * ldo + col] = acc[i][j][r] + b;
        }
    }
  }
};

template <typename T>
struct EpiQkv {
  QkvArgs<T> a;
  template <int FM, int FN>
  __device__ void apply(f32x16 (&acc)[FM][FN], int row0, int col0, int lane, int M) const {
    static_assert(FN % 2 == 0, "QKV epilogue needs column pairs");
    const int dh = a.head_dim, half = dh / 2;
    const int qd = a.n_q_heads * dh, kd = a.n_kv_heads * dh;
    const float* __restrict__ rcos = a.rcos;
    const float* __restrict__ rsin = a.rsin;
    // (stream, arena row) of a token row: b = row / tokens,
    // buffer_row0(len[b]) + row - b tokens.  The wave's rows span at most two
    // streams when tokens >= 32 FM: their two lengths are read once (no
    // per-row lookup ahead of the rotary tables); otherwise every row looks
    // its stream up.
    const int ntok = a.tokens;
    const int b_lo = min(row0, M - 1) / ntok, b_hi = min(row0 + 32 * FM - 1, M - 1) / ntok;
    const bool two = b_hi - b_lo <= 1;
    const int len_lo = buffer_row0(a.len[b_lo]), len_hi = buffer_row0(a.len[b_hi]);
    const int gap_lo = len_lo - a.len[b_lo], gap_hi = len_hi - a.len[b_hi];
    const int row_hi = b_hi * ntok;
    // rotary position of a token = its arena row minus its stream's alignment gap
    auto gap_of = [&](int b) __attribute__((always_inline)) {
      if (two) return b == b_hi ? gap_hi : gap_lo;
      const int P = a.len[b];
      return buffer_row0(P) - P;
    };
    auto locate = [&](int row) __attribute__((always_inline)) {
      row = min(row, M - 1);
      if (two) {
        const bool hi = row >= row_hi;
        const int b = hi ? b_hi : b_lo;
        return int2{b, (hi ? len_hi : len_lo) + row - b * ntok};
      }
      const int b = row / ntok;
      return int2{b, buffer_row0(a.len[b]) + row - b * ntok};
    };
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      int2 rp[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) rp[r] = locate(row0 + 32 * i + acc_row(r, lane));
#pragma unroll
      for (int j = 0; j < FN; j += 2) {
        const int c0 = col0 + 32 * j;  // first packed column of the pair group
        if (c0 < qd + kd) {
          const bool isq = c0 < qd;
          const int cc = isq ? c0 : c0 - qd;
          const int head = cc / dh;
          const int dlo = 32 * ((cc - head * dh) >> 6) + (lane & 31);
          float cs[16], sn[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int pos = rp[r].y - gap_of(rp[r].x);
            cs[r] = rcos[(size_t)pos * half + dlo];
            sn[r] = rsin[(size_t)pos * half + dlo];
          }
          // rotated pair (d, d + dh/2) per register, then each group of
          // four rows transposed so a lane writes 4 features of one row
          const int d0 = dlo & ~3, k4 = lane & 3;
          // (stream, arena row) of the row each lane writes (K rows only)
          int2 pw[4];
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4)
            pw[q4] = isq ? int2{0, 0} : locate(row0 + 32 * i + 8 * q4 + 4 * (lane >> 5) + k4);
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            float y0[4], y1[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int r = 4 * q4 + e;
              const float x0 = acc[i][j][r], x1 = acc[i][j + 1][r];
              y0[e] = x0 * cs[r] - x1 * sn[r];
              y1[e] = x1 * cs[r] + x0 * sn[r];
            }
            const f32x4 u0 = quad_rows(y0[0], y0[1], y0[2], y0[3], lane);
            const f32x4 u1 = quad_rows(y1[0], y1[1], y1[2], y1[3], lane);
            const int row = row0 + 32 * i + 8 * q4 + 4 * (lane >> 5) + k4;
            if (row >= M) continue;
            T* dst = isq ? a.q + (size_t)row * qd + head * dh
                         : a.karena + (((size_t)pw[q4].x * a.n_kv_heads + head) * a.S + pw[q4].y) * dh;
            store4<T>(dst + d0, u0[0], u0[1], u0[2], u0[3]);
            store4<T>(dst + d0 + half, u1[0], u1[1], u1[2], u1[3]);
          }
        } else {
          // V^T rows: registers 4q..4q+3 of a lane are 4 consecutive tokens,
          // written as one 4-element run when they are valid rows of one stream
          const int cc = c0 - qd - kd;
          const int g = cc / dh, d = cc - g * dh + (lane & 31);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int rowq = row0 + 32 * i + acc_row(4 * q, lane);
            const bool run = rowq + 3 < M && rp[4 * q].x == rp[4 * q + 3].x &&
                             (rp[4 * q].y & 3) == 0;  // aligned 4-element run
            if (run) {
              T* base = a.vtarena + ((size_t)rp[4 * q].x * a.n_kv_heads + g) * dh * a.S + rp[4 * q].y;
              store4<T>(base + (size_t)d * a.S, acc[i][j][4 * q], acc[i][j][4 * q + 1],
                        acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
              store4<T>(base + (size_t)(d + 32) * a.S, acc[i][j + 1][4 * q],
                        acc[i][j + 1][4 * q + 1], acc[i][j + 1][4 * q + 2],
                        acc[i][j + 1][4 * q + 3]);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int r = 4 * q + e;
                if (rowq + e >= M) continue;
                T* base = a.vtarena + ((size_t)rp[r].x * a.n_kv_heads + g) * dh * a.S + rp[r].y;
                base[(size_t)d * a.S] = from_f32<T>(acc[i][j][r]);
                base[(size_t)(d + 32) * a.S] = from_f32<T>(acc[i][j + 1][r]);
              }
            }
          }
        }
      }
    }
  }
};

struct EpiGatedResid {
  static constexpr bool kStaged = true;
  float* h; const float* mod; int mod_ld, gate_off, chunk_len, ldh;
  const int* period;  // FiLM-row sharing flag (film_row), or nullptr
  // Direct-to-LDS kernels: the accumulators go through the (idle) LDS so that
  // h is read and written as whole-row 16-byte pieces, in passes of PI
  // 32-row slabs per wave; `smem` holds NW x PI x 32 x WTN floats.
  template <int FM, int FN, int NW, int LDS_BYTES>
  __device__ void apply_staged(f32x16 (&acc)[FM][FN], float* smem, int row0, int col0, int lane,
                               int wave, int M) const {
    constexpr int WTN = 32 * FN;
    constexpr int PI_MAX = LDS_BYTES / (NW * 32 * WTN * 4);
    constexpr int PI = PI_MAX >= FM ? FM : (PI_MAX >= 2 && FM % 2 == 0 ? 2 : 1);
    static_assert(PI >= 1 && FM % PI == 0, "staging does not fit");
    constexpr int C4 = WTN / 4;                // 16-byte pieces per row
    constexpr int PER = PI * 32 * C4 / 64;     // pieces per lane and pass
    const int per = film_period(period);
    float* cs = smem + wave * PI * 32 * WTN;
    float* __restrict__ hh = h;
    const float* __restrict__ mm = mod;
#pragma unroll
    for (int i0 = 0; i0 < FM; i0 += PI) {
      if (i0 > 0) __syncthreads();  // every wave done reading the last pass
#pragma unroll
      for (int ii = 0; ii < PI; ++ii)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            cs[(32 * ii + acc_row(r, lane)) * WTN + 32 * j + (lane & 31)] = acc[i0 + ii][j][r];
      __syncthreads();
#pragma unroll
      for (int q0 = 0; q0 < PER; q0 += 8) {
        f32x4 hv[8], gv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {  // independent loads first
          if (q0 + q >= PER) break;
          const int idx = (q0 + q) * 64 + lane, rr = idx / C4, c4 = idx - rr * C4;
          const int row = min(row0 + 32 * i0 + rr, M - 1);
          hv[q] = *reinterpret_cast<const f32x4*>(hh + (size_t)row * ldh + col0 + 4 * c4);
          const size_t mrow = (size_t)film_row(row / chunk_len, per) * mod_ld;
          gv[q] = *reinterpret_cast<const f32x4*>(mm + mrow + gate_off + col0 + 4 * c4);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (q0 + q >= PER) break;
          const int idx = (q0 + q) * 64 + lane, rr = idx / C4, c4 = idx - rr * C4;
          const int row = row0 + 32 * i0 + rr;
          const f32x4 a4 = *reinterpret_cast<const f32x4*>(cs + rr * WTN + 4 * c4);
          if (row < M)
            *reinterpret_cast<f32x4*>(hh + (size_t)row * ldh + col0 + 4 * c4) = hv[q] + gv[q] * a4;
        }
      }
    }
  }
  template <int FM, int FN>
  __device__ void apply(f32x16 (&acc)[FM][FN], int row0, int col0, int lane, int M) const {
    const int per = film_period(period);
    float* __restrict__ hh = h;
    const float* __restrict__ mm = mod;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = col0 + 32 * j + (lane & 31);
        float hv[16], gv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {  // independent loads first
          const int row = min(row0 + 32 * i + acc_row(r, lane), M - 1);
          hv[r] = hh[(size_t)row * ldh + col];
          gv[r] = mm[(size_t)film_row(row / chunk_len, per) * mod_ld + gate_off + col];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + 32 * i + acc_row(r, lane);
          if (row < M) hh[(size_t)row * ldh + col] = hv[r] + gv[r] * acc[i][j][r];
        }
      }
  }
};

template <typename T>
struct EpiGeglu {
  T* out; int ldo;
  template <int FM, int FN>
  __device__ void apply(f32x16 (&acc)[FM][FN], int row0, int col0, int lane, int M) const {
    static_assert(FN % 2 == 0, "GeGLU epilogue needs column pairs");
    const bool vec = (ldo & 3) == 0;
#pragma unroll
    for (int j = 0; j < FN; j += 2) {
      const int col = ((col0 + 32 * j) >> 1) + (lane & 28);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float y[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            y[e] = gelu_tanh_f(acc[i][j][4 * q4 + e]) * acc[i][j + 1][4 * q4 + e];
          const f32x4 u = quad_rows(y[0], y[1], y[2], y[3], lane);
          const int row = row0 + 32 * i + 8 * q4 + 4 * (lane >> 5) + (lane & 3);
          if (row < M) store_quad<T>(out + (size_t)row * ldo + col, u, vec);
        }
    }
  }
};

template <typename T>
struct EpiGelu {
  T* out; int ldo;
  template <int FM, int FN>
  __device__ void apply(f32x16 (&acc)[FM][FN], int row0, int col0, int lane, int M) const {
    const bool vec = (ldo & 3) == 0;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = col0 + 32 * j + (lane & 28);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float y[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) y[e] = gelu_tanh_f(acc[i][j][4 * q4 + e]);
          const f32x4 u = quad_rows(y[0], y[1], y[2], y[3], lane);
          const int row = row0 + 32 * i + 8 * q4 + 4 * (lane >> 5) + (lane & 3);
          if (row < M) store_quad<T>(out + (size_t)row * ldo + col, u, vec);
        }
    }
  }
};

// ------------------------------------------------------ few-row GEMM (GEMV)
// out[m][n] = silu(sum_k A[m][k] W[n][k] + bias[n]) for M <= kGemvRows rows
// (the time-MLP at small batch): one wave per output column n, lanes take
// 16-byte pieces of k (the weight row once, every input row at the same
// pieces), fp32 sums reduced across the wave.  One launch, no split-K pass.
constexpr int kGemvRows = 16;
template <typename T>
__global__ __launch_bounds__(256) void gemv_bias_silu_kernel(const T* __restrict__ A,
                                                             const T* __restrict__ Bt,
                                                             const float* __restrict__ bias,
                                                             T* __restrict__ out, int M, int N,
                                                             int K, const int* __restrict__ skip) {
  if (skip && *skip) return;
  constexpr int EPV = 16 / (int)sizeof(T);  // elements per 16-byte piece
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  float acc[kGemvRows];
#pragma unroll
  for (int m = 0; m < kGemvRows; ++m) acc[m] = 0.f;
  const T* wrow = Bt + (size_t)n * K;
  // rows m >= M re-read row M - 1 (in bounds, never stored), so every load
  // is unconditional, and the scheduling barrier keeps all of a k-piece's
  // loads ahead of its FMAs (left alone, the scheduler sinks each load next
  // to its use and the wave waits for them one by one)
#pragma unroll 1
  for (int k0 = EPV * lane; k0 < K; k0 += 64 * EPV) {
    const u32x4 wraw = *reinterpret_cast<const u32x4*>(wrow + k0);
    u32x4 araw[kGemvRows];
#pragma unroll
    for (int m = 0; m < kGemvRows; ++m)
      araw[m] = *reinterpret_cast<const u32x4*>(A + (size_t)min(m, M - 1) * K + k0);
    __builtin_amdgcn_sched_barrier(0);
    const T* we = reinterpret_cast<const T*>(&wraw);
#pragma unroll
    for (int m = 0; m < kGemvRows; ++m) {
      const T* e = reinterpret_cast<const T*>(&araw[m]);
#pragma unroll
      for (int i = 0; i < EPV; ++i) acc[m] = fmaf(to_f32(e[i]), to_f32(we[i]), acc[m]);
    }
  }
  const float b = bias[n];
#pragma unroll
  for (int m = 0; m < kGemvRows; ++m) {
    const float v = wave_sum(acc[m]);
    if (m < M && lane == 0) out[(size_t)m * N + n] = from_f32<T>(silu_f(v + b));
  }
}

// ------------------------------------------ few-row GEMM, weights streamed
// out[m][n] = sum_k A[m][k] W[n][k] + bias[n] in fp32, bf16 operands, for
// M <= 16 rows and a weight matrix far larger than the memory-side cache
// (the FiLM maps of every norm at small batch), so the kernel is a stream of
// the weights at HBM rate.  A wave owns 16 output columns at a time, whose
// weight rows are one contiguous range, and multiplies them with MFMA
// 16x16x32 tiles.  Lane (q, c) = (lane / 16, lane % 16) takes column c and,
// of every 128-element k batch, the 64 contiguous bytes at k = 32q: four
// 16-byte pieces, piece s holding k = 32q + 8s .. +8.  The MFMA's k order is
// permuted that way on both operands, so every lane's weight loads are
// contiguous; A, permuted once, stays in registers.  The weight pieces of
// the next three batches (across the end of a column group, the next
// group's first three) are in flight while one batch is multiplied.
constexpr int kStreamRows = 16;
template <int NB>
__global__ __launch_bounds__(256) void stream_bias_f32_kernel(const bf16_t* __restrict__ A,
                                                              const bf16_t* __restrict__ Bt,
                                                              const float* __restrict__ bias,
                                                              float* __restrict__ out, int M,
                                                              int N, const int* __restrict__ skip) {
  if (skip && *skip) return;
  constexpr int K = 128 * NB, R = 4, AHEAD = 3;  // ring slots; batches in flight
  static_assert(NB % R == 0 && AHEAD < R, "ring");
  const int lane = threadIdx.x & 63, q = lane >> 4, c = lane & 15;
  const int G = N / 16, stride = gridDim.x * 4;
  int g = blockIdx.x + gridDim.x * (threadIdx.x >> 6);
  if (g >= G) return;  // whole waves
  // rows m >= M repeat row M - 1: every load is in bounds and unconditional,
  // and those rows are never stored
  bf16x8 a[NB][4];
  const bf16_t* arow = A + (size_t)min(c, M - 1) * K + 32 * q;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int p = 0; p < 4; ++p)
      a[b][p] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(arow + 128 * b + 8 * p));
  auto wrow = [&](int gg) { return Bt + (size_t)(16 * gg + c) * K + 32 * q; };
  const bf16_t* cur = wrow(g);
  u16x8 w[R][4];
#pragma unroll
  for (int b = 0; b < AHEAD; ++b)
#pragma unroll
    for (int p = 0; p < 4; ++p) w[b][p] = *reinterpret_cast<const u16x8*>(cur + 128 * b + 8 * p);
  for (;;) {
    // the last group's look-ahead re-reads its own first batches (cache
    // hits) instead of another group's weights
    const bf16_t* nxt = g + stride < G ? wrow(g + stride) : cur;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int ib = b + AHEAD;
      const bf16_t* src = ib < NB ? cur + 128 * ib : nxt + 128 * (ib - NB);
#pragma unroll
      for (int p = 0; p < 4; ++p) w[ib % R][p] = *reinterpret_cast<const u16x8*>(src + 8 * p);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int p = 0; p < 4; ++p)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[b][p], __builtin_bit_cast(bf16x8, w[b % R][p]),
                                                      acc, 0, 0, 0);
    }
    const int n = 16 * g + c;
    const float bn = bias[n];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 4 * q + r;
      if (m < M) out[(size_t)m * N + n] = acc[r] + bn;
    }
    g += stride;
    if (g >= G) break;
    cur = nxt;
  }
}

template <int NB>
void launch_stream_bias_f32(const bf16_t* A, const bf16_t* Bt, const float* bias, float* out,
                            int M, int N, hipStream_t s, const int* skip) {
  // one workgroup of four waves per CU, every wave about G / 1024 column
  // groups (a cold read of the FiLM weights: 48.5 us against 50.4 with two
  // workgroups per CU, and 46.6 for a plain streaming read of the same bytes)
  const int G = N / 16, blocks = std::min(256, (G + 3) / 4);
  hipLaunchKernelGGL((stream_bias_f32_kernel<NB>), dim3(blocks), dim3(256), 0, s, A, Bt, bias, out,
                     M, N, skip);
}

// -------------------------------------------------------------- tile choice
// Tile shapes (BM x BN, waves); every wave owns a sub-tile at least 64
// columns wide, so paired epilogues find both partners of a 64-column pair
// group in one wave.
enum Tile { T256x128w8 = 0, T128x128w8 = 1, T64x128w4 = 2, T32x128w2 = 3, T256x256big = 4 };
constexpr int kTileBM[] = {256, 128, 64, 32, 256};
constexpr int kTileBN[] = {128, 128, 128, 128, 256};
// k-groups per tile (waves per block = NW x KG): the 2-wave 32-row tile
// (M <= 32: weight-streaming GEMMs) gets a second wave group, doubling the
// loads and LDS reads in flight; the larger tiles measured no gain.
constexpr int kTileKG[] = {1, 1, 1, 2};

template <typename T, int BM, int BN, int NW, int WGM, int KG, class Epi>
void launch_tile(const T* A, const T* Bt, int M, int N, int K, const GemmPlan& p,
                 const GemmWork& w, const Epi& epi, hipStream_t s) {
  dim3 grid(N / BN, (M + BM - 1) / BM, p.ks);
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, NW, WGM, KG, Epi>), grid, dim3(64 * NW * KG), 0, s,
                     A, Bt, M, N, K, p.ks, w.ws, epi);
  if (p.ks > 1 && !std::is_same<Epi, EpiNone>::value)
    hipLaunchKernelGGL((gemm_reduce_kernel<BM, BN, NW, WGM, Epi>), dim3(grid.x, grid.y),
                       dim3(64 * NW), 0, s, w.ws, M, N, p.ks, epi);
}

// Direct-to-LDS instances: (tile, waves, stages) of the bf16 tiles that use it.
#define FV_DMA_TILES(X) \
  X(256, 256, 8, 2, 2)  \
  X(128, 128, 8, 4, 3)  \
  X(128, 128, 8, 4, 2)  \
  X(64, 128, 4, 2, 3)

template <int BM, int BN, int NW, int WGM, int NS, class Epi>
hipError_t allow_dma_lds() {
  return hipFuncSetAttribute(
      reinterpret_cast<const void*>(&gemm_dma_kernel<BM, BN, NW, WGM, NS, Epi>),
      hipFuncAttributeMaxDynamicSharedMemorySize, dma_lds_bytes<BM, BN, NW, WGM, NS>());
}

template <int BM, int BN, int NW, int WGM, int NS, class Epi>
void launch_dma(const bf16_t* A, const bf16_t* Bt, int M, int N, int K, const GemmPlan& p,
                const GemmWork& w, const Epi& epi, hipStream_t s) {
  dim3 grid(N / BN, (M + BM - 1) / BM, p.ks);
  hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, NW, WGM, NS, Epi>), grid, dim3(64 * NW),
                     (dma_lds_bytes<BM, BN, NW, WGM, NS>()), s, A, Bt, M, N, K, p.ks, w.ws, epi);
  // the 256x256 tile never splits k (plan_gemm), so it has no reduction
  if constexpr (BM * BN < 256 * 256 && !std::is_same<Epi, EpiNone>::value)
    if (p.ks > 1)
      hipLaunchKernelGGL((gemm_reduce_kernel<BM, BN, NW, WGM, Epi>), dim3(grid.x, grid.y),
                         dim3(64 * NW), 0, s, w.ws, M, N, p.ks, epi);
}

// Launches tile p.tile with the direct-to-LDS kernel when it has one;
// returns false otherwise.  The 128x128 tile takes three stages when the
// grid fits the chip with one workgroup per CU (the deeper ring hides load
// latency, measured 1568 against 1864 us per batch-1 step with two), two
// stages otherwise (two workgroups then fit per CU and overlap each other).
template <class Epi>
bool try_dma(const bf16_t* A, const bf16_t* Bt, int M, int N, int K, const GemmPlan& p,
             const GemmWork& w, const Epi& epi, hipStream_t s) {
  const bool rounds = (long)p.tiles * p.ks > 256;
  switch (p.tile) {
    case T256x256big: launch_dma<256, 256, 8, 2, 2>(A, Bt, M, N, K, p, w, epi, s); return true;
    case T128x128w8:
      if (rounds)
        launch_dma<128, 128, 8, 4, 2>(A, Bt, M, N, K, p, w, epi, s);
      else
        launch_dma<128, 128, 8, 4, 3>(A, Bt, M, N, K, p, w, epi, s);
      return true;
    case T64x128w4:  // chosen only below about 400 tiles x splits: one round
      launch_dma<64, 128, 4, 2, 3>(A, Bt, M, N, K, p, w, epi, s);
      return true;
    default: return false;
  }
}

template <typename T, class Epi>
void run_gemm(const T* A, const T* Bt, int M, int N, int K, const GemmWork& w, const Epi& epi,
              hipStream_t s) {
  if (M <= 0) return;
  const GemmPlan p = plan_gemm(M, N, K, sizeof(T) == 2);
  if constexpr (sizeof(T) == 2) {
    if (try_dma(A, Bt, M, N, K, p, w, epi, s)) return;
  }
  switch (p.tile) {
    case T256x128w8: launch_tile<T, 256, 128, 8, 4, kTileKG[0]>(A, Bt, M, N, K, p, w, epi, s); break;
    case T128x128w8: launch_tile<T, 128, 128, 8, 4, kTileKG[1]>(A, Bt, M, N, K, p, w, epi, s); break;
    case T64x128w4: launch_tile<T, 64, 128, 4, 2, kTileKG[2]>(A, Bt, M, N, K, p, w, epi, s); break;
    case T32x128w2: launch_tile<T, 32, 128, 2, 1, kTileKG[3]>(A, Bt, M, N, K, p, w, epi, s); break;
    default: break;  // N % 128 != 0 is rejected at fv_create
  }
}

}  // namespace

// Tile by row count: large M takes 256x256 tiles (fewer re-reads of A and
// W) when that still gives about 200 blocks and no mostly idle second round,
// else 128x128 (bf16; two workgroups per CU); medium M takes 128x128 tiles when that still gives
// about 200 blocks (96 for an output or down projection), else 64x128;
// small M takes 64- or 32-row tiles.  When a
// grid has fewer than 128 tiles, k is split (KS a power of two, at least 4
// k-tiles per split, at most about 320 blocks) so that every CU streams its
// share of the weights; with `reduce_fused` (the output and down
// projections, whose split sum is fused into the next kernel at no extra
// launch) grids of up to 160 tiles are split too.
GemmPlan plan_gemm(int M, int N, int K, bool bf16, bool reduce_fused) {
  GemmPlan p;
  if (N % 128 || M <= 0) return p;
  const int bk = bf16 ? 64 : 32, nk = K / bk;
  auto ntiles = [&](int t) { return ((M + kTileBM[t] - 1) / kTileBM[t]) * (N / kTileBN[t]); };
  if (M >= 4096) {
    // 256x256 tiles run one workgroup per CU, 128x128 tiles two.  A grid of
    // two rounds of 256x256 tiles whose second round is mostly idle (under 72
    // of 256 tiles) takes 128x128 tiles instead: measured per step, batch 16
    // (QKV, 64 tiles in round two) 7.82 -> 7.67 ms, batch 36 (output and
    // down projections, 28) 17.67 -> 17.00, batch 40 (60) 19.03 -> 18.73;
    // slower at batch 44 (88) and 48 (120)
    const long n256 = ntiles(T256x256big);
    const bool big = n256 >= 200 && !(n256 > 256 && n256 <= 512 && n256 % 256 < 72);
    if (!bf16)
      p.tile = T256x128w8;
    else if (N % 256 == 0 && big)
      p.tile = T256x256big;
    else
      p.tile = N % 256 == 0 ? T128x128w8 : T256x128w8;
  } else if (M > 256) {
    // (an output or down projection takes 128x128 tiles from 96 of them on:
    // with k split in two they beat 64x128 tiles, batch 3 2790 -> 2722 us)
    if (reduce_fused && bf16 && ntiles(T128x128w8) >= 96)
      p.tile = T128x128w8;
    else
      p.tile = ntiles(T128x128w8) >= 200 ? T128x128w8 : T64x128w4;
  } else if (M > 32) {
    p.tile = T64x128w4;
  } else {
    p.tile = T32x128w2;
  }
  p.tiles = ntiles(p.tile);
  p.ks = 1;
  if ((p.tiles < 128 || (reduce_fused && p.tiles <= 160)) && p.tile != T256x256big)
    while ((long)p.tiles * p.ks * 2 <= 320 && nk / (p.ks * 2) >= 4 && p.ks < 8) p.ks *= 2;
  p.ws_floats = p.ks > 1 ? (size_t)p.ks * M * N : 0;
  return p;
}


// The direct-to-LDS tiles (every bf16 tile but 32x128) store bf16 partials.
bool gemm_partials_bf16(const GemmPlan& p, bool bf16) {
  return bf16 && p.ks > 1 &&
         (p.tile == T256x256big || p.tile == T128x128w8 || p.tile == T64x128w4);
}

template <typename T>
int gemm_partials(const T* A, const T* Bt, int M, int N, int K, const GemmWork& w,
                  hipStream_t s, bool* bf16_parts) {
  const GemmPlan p = plan_gemm(M, N, K, sizeof(T) == 2, true);
  *bf16_parts = false;
  if (p.ks <= 1) return 1;
  if constexpr (sizeof(T) == 2) {
    if (try_dma(A, Bt, M, N, K, p, w, EpiNone{}, s)) {
      *bf16_parts = true;
      return p.ks;
    }
  }
  switch (p.tile) {
    case T256x128w8: launch_tile<T, 256, 128, 8, 4, kTileKG[0]>(A, Bt, M, N, K, p, w, EpiNone{}, s); break;
    case T128x128w8: launch_tile<T, 128, 128, 8, 4, kTileKG[1]>(A, Bt, M, N, K, p, w, EpiNone{}, s); break;
    case T64x128w4: launch_tile<T, 64, 128, 4, 2, kTileKG[2]>(A, Bt, M, N, K, p, w, EpiNone{}, s); break;
    default: launch_tile<T, 32, 128, 2, 1, kTileKG[3]>(A, Bt, M, N, K, p, w, EpiNone{}, s);
  }
  return p.ks;
}

template <typename T>
void gemm_bias_silu(const T* A, const T* Bt, const float* bias, T* out, int M, int N, int K,
                    const GemmWork& w, hipStream_t s, const int* skip) {
  if (M <= kGemvRows && N % 4 == 0 && K % (16 / (int)sizeof(T)) == 0) {
    hipLaunchKernelGGL((gemv_bias_silu_kernel<T>), dim3(N / 4), dim3(256), 0, s, A, Bt, bias, out,
                       M, N, K, skip);
    return;
  }
  run_gemm(A, Bt, M, N, K, w, EpiBiasSilu<T>{out, bias, N, skip}, s);
}
template <typename T>
void gemm_bias_f32(const T* A, const T* Bt, const float* bias, float* out, int M, int N, int K,
                   const GemmWork& w, hipStream_t s, const int* skip) {
  if constexpr (sizeof(T) == 2) {
    if (M <= kStreamRows && N % 16 == 0) {
      switch (K) {
        case 512: launch_stream_bias_f32<4>(A, Bt, bias, out, M, N, s, skip); return;
        case 1024: launch_stream_bias_f32<8>(A, Bt, bias, out, M, N, s, skip); return;
        default: break;
      }
    }
  }
  run_gemm(A, Bt, M, N, K, w, EpiBiasF32{out, bias, N, skip}, s);
}
template <typename T>
void gemm_qkv(const T* A, const T* Bt, const QkvArgs<T>& qa, int M, int N, int K,
              const GemmWork& w, hipStream_t s) {
  run_gemm(A, Bt, M, N, K, w, EpiQkv<T>{qa}, s);
}
template <typename T>
void gemm_gated_resid(const T* A, const T* Bt, float* h, const float* mod, int mod_ld,
                      int gate_off, int chunk_len, int M, int N, int K, const GemmWork& w,
                      hipStream_t s, const int* period) {
  run_gemm(A, Bt, M, N, K, w, EpiGatedResid{h, mod, mod_ld, gate_off, chunk_len, N, period}, s);
}
template <typename T>
void gemm_geglu(const T* A, const T* Bt, T* out, int M, int N, int K, const GemmWork& w,
                hipStream_t s) {
  run_gemm(A, Bt, M, N, K, w, EpiGeglu<T>{out, N / 2}, s);
}
template <typename T>
void gemm_gelu(const T* A, const T* Bt, T* out, int M, int N, int K, const GemmWork& w,
               hipStream_t s) {
  run_gemm(A, Bt, M, N, K, w, EpiGelu<T>{out, N}, s);
}

// The direct-to-LDS kernels' dynamic LDS exceeds the default limit; every
// (tile, epilogue) instance is raised once per device before any launch.
template <class Epi>
hipError_t allow_dma_all() {
  hipError_t e = hipSuccess;
#define FV_ALLOW(BM, BN, NW, WGM, NS) \
  if (e == hipSuccess) e = allow_dma_lds<BM, BN, NW, WGM, NS, Epi>();
  FV_DMA_TILES(FV_ALLOW)
#undef FV_ALLOW
  return e;
}

hipError_t gemm_prepare() {
  const hipError_t e[] = {allow_dma_all<EpiBiasSilu<bf16_t>>(), allow_dma_all<EpiBiasF32>(),
                          allow_dma_all<EpiQkv<bf16_t>>(),      allow_dma_all<EpiGatedResid>(),
                          allow_dma_all<EpiGeglu<bf16_t>>(),    allow_dma_all<EpiGelu<bf16_t>>(),
                          allow_dma_all<EpiNone>()};
  for (hipError_t x : e)
    if (x != hipSuccess) return x;
  return hipSuccess;
}

#define FV_INSTANTIATE(T)                                                                        \
  template void gemm_bias_silu<T>(const T*, const T*, const float*, T*, int, int, int,           \
                                  const GemmWork&, hipStream_t, const int*);                     \
  template void gemm_bias_f32<T>(const T*, const T*, const float*, float*, int, int, int,        \
                                 const GemmWork&, hipStream_t, const int*);                      \
  template void gemm_qkv<T>(const T*, const T*, const QkvArgs<T>&, int, int, int,                \
                            const GemmWork&, hipStream_t);                                       \
  template void gemm_gated_resid<T>(const T*, const T*, float*, const float*, int, int, int,     \
                                    int, int, int, const GemmWork&, hipStream_t, const int*);    \
  template void gemm_geglu<T>(const T*, const T*, T*, int, int, int, const GemmWork&,            \
                              hipStream_t);                                                      \
  template void gemm_gelu<T>(const T*, const T*, T*, int, int, int, const GemmWork&, hipStream_t); \
  template int gemm_partials<T>(const T*, const T*, int, int, int, const GemmWork&, hipStream_t, \
                                bool*);
FV_INSTANTIATE(bf16_t)
FV_INSTANTIATE(float)
#undef FV_INSTANTIATE

}  // namespace fv
