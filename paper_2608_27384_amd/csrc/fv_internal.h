// Internal declarations of the gfx950 streaming action-decode library.
//
// Element types: "bf16" tensors hold raw bf16 bit patterns (uint16_t); every
// kernel is written once as a template over the storage type T (bf16_t or
// float) and uses the matching MFMA instruction (16x16x32 bf16 or 16x16x4
// fp32), so both precisions share one code path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <utility>
#include <vector>

#include "../../include/flashvla.h"

namespace fv {

typedef uint16_t bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // 16-byte moves (native vector)
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));  // 8-byte moves
typedef float f32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- conversions
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float((uint32_t)x << 16); }

// Round to nearest even (the gfx950 conversion instruction); NaN stays NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f32_to_bf16(x); }

// ------------------------------------------------------------ MFMA operands
// One 16x16 output tile: lane l holds rows 4*(l/16)+r (r = 0..3) of column
// l%16.  An A-operand (B-operand) fragment holds KG consecutive k of row
// (column) l%16 starting at k = KG*(l/16); one instruction covers KM = 4*KG k.
template <typename T> struct Mfma;
template <> struct Mfma<bf16_t> {
  static constexpr int KG = 8, KM = 32;
  typedef bf16x8 frag;
  __device__ static __forceinline__ frag load(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(p));
  }
  __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static constexpr int KG = 1, KM = 4;
  typedef float frag;
  __device__ static __forceinline__ frag load(const float* p) { return *p; }
  __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// Four consecutive elements as fp32 (16-byte fp32 or 8-byte bf16 load; p aligned to that).
__device__ __forceinline__ f32x4 load4_f32(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ f32x4 load4_f32(const bf16_t* p) {
  const u16x4 v = *reinterpret_cast<const u16x4*>(p);
  return f32x4{to_f32(v[0]), to_f32(v[1]), to_f32(v[2]), to_f32(v[3])};
}
// Four consecutive elements (16-byte fp32 or 8-byte bf16 store; p aligned to that).
template <typename T>
__device__ __forceinline__ void store4(T* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<f32x4*>(p) = f32x4{a, b, c, d};
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<u16x4*>(p) = u16x4{f32_to_bf16(a), f32_to_bf16(b), f32_to_bf16(c), f32_to_bf16(d)};
}

// Sum over the 64 lanes, the same value in every lane, without LDS
// permutes: the gfx950 lane swaps exchange across 32-lane halves and 16-lane
// rows; DPP row rotations by 8 and 4 and quad permutes (xor 2, xor 1) finish
// within a row.  Every lane adds the same pairs, so all lanes agree bit for
// bit.
template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  x = dpp_add<0x128>(x);  // row_ror:8
  x = dpp_add<0x124>(x);  // row_ror:4
  x = dpp_add<0x4E>(x);   // quad_perm [2,3,0,1]
  x = dpp_add<0xB1>(x);   // quad_perm [1,0,3,2]
  return x;
}

// Pulls part of [p, p + bytes) into the chip's memory-side cache ahead of
// the kernel that reads it next (the weights of the next GEMM, which would
// otherwise come cold from HBM): thread t of the grid (NT threads per
// block) loads the 16-byte pieces t, t + n, .. (NPF of them, n = the grid's
// threads) at its kernel's start and discards them at the end.  The loads
// are unconditional: a piece index past the buffer is clamped to its last
// piece, and with p == nullptr every load reads `fallback` (any readable
// 16-byte location, e.g. one of the kernel's own inputs).  A conditional
// load would make the compiler's memory-counter waits for the kernel's own
// loads (issued before these) also wait for the prefetch.
template <int NPF, int NT>
struct Prefetch {
  u32x4 v[NPF];
  __device__ __forceinline__ void issue(const void* p, size_t bytes, const void* fallback) {
    const size_t n = (size_t)gridDim.x * gridDim.y * gridDim.z * NT;
    const size_t t =
        (((size_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) * NT +
        threadIdx.x;
    const bool on = p != nullptr && bytes >= 16;
    const u32x4* q = static_cast<const u32x4*>(on ? p : fallback);
    const size_t last = on ? bytes / 16 - 1 : 0;
#pragma unroll
    for (int i = 0; i < NPF; ++i) {
      const size_t k = t + (size_t)i * n;
      v[i] = q[k < last ? k : last];
    }
  }
  __device__ __forceinline__ void retire() const {
#pragma unroll
    for (int i = 0; i < NPF; ++i) asm volatile("" ::"v"(v[i]));
  }
};

// Both activations are evaluated as x / (1 + 2^a) with the bare hardware
// exp2 and reciprocal instructions (1 ulp each; a few instructions instead
// of the library tanh, and instead of the range handling of exp2f and the
// IEEE division sequence); the tanh-form GELU uses
// 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)).  The limits hold: 2^a = inf gives
// 0, and 2^a below the normal range (flushed to 0) gives x.
__device__ __forceinline__ float silu_f(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}
__device__ __forceinline__ float gelu_tanh_f(float x) {
  const float c = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  return x * __builtin_amdgcn_rcpf(
                 1.0f + __builtin_amdgcn_exp2f(c * fmaf(0.044715f * x, x * x, x)));
}

// ------------------------------------------------------------ GEMM launches
// C[M][N] = A[M][K] * Bt[N][K]^T with fp32 accumulation, followed by a fused
// epilogue.  A is row-major with leading dimension K; Bt is the weight stored
// output-major ([out][in]).  Requirements: N % 128 == 0, K % 64 == 0 (bf16) or
// K % 32 == 0 (fp32), 16-byte aligned base pointers.
struct GemmPlan {
  int tile = -1, ks = 1, tiles = 0;  // tile shape id, split-K factor, output tiles
  size_t ws_floats = 0;              // split-K workspace this GEMM needs
};
// reduce_fused: the plan of an output or down projection (its split sum
// runs inside the next kernel, so splitting costs no launch).
GemmPlan plan_gemm(int M, int N, int K, bool bf16, bool reduce_fused = false);

// Split-K scratch shared by every GEMM of a handle (launches are stream
// ordered): partial tiles, fp32, or bf16 for the direct-to-LDS kernel with
// no epilogue (see gemm_partials).
struct GemmWork {
  float* ws = nullptr;
};

template <typename T>
struct QkvArgs {
  T* q;                 // [rows][Hq*dh] rotated queries
  T* karena;            // this layer's keys   [Bmax][Hkv][S][dh]
  T* vtarena;           // this layer's values [Bmax][Hkv][dh][S] (transposed)
  const float* rcos;    // [S][dh/2]
  const float* rsin;
  const int* len;       // [B] valid prefix rows: token row r of stream b = r / tokens
                        // goes to arena row buffer_row0(len[b]) + r - b * tokens
  int tokens, n_q_heads, n_kv_heads, head_dim, S;
};

// skip (optional): a device flag; when it holds a nonzero value at run time
// the launch computes nothing (its workgroups return at once).
template <typename T>
void gemm_bias_silu(const T* A, const T* Bt, const float* bias, T* out, int M, int N, int K,
                    const GemmWork& w, hipStream_t s, const int* skip = nullptr);
template <typename T>
void gemm_bias_f32(const T* A, const T* Bt, const float* bias, float* out, int M, int N, int K,
                   const GemmWork& w, hipStream_t s, const int* skip = nullptr);
template <typename T>
void gemm_qkv(const T* A, const T* Bt, const QkvArgs<T>& qa, int M, int N, int K,
              const GemmWork& w, hipStream_t s);
// h[row][col] += mod[film_row(row / chunk_len, *period)][gate_off + col] * acc
template <typename T>
void gemm_gated_resid(const T* A, const T* Bt, float* h, const float* mod, int mod_ld,
                      int gate_off, int chunk_len, int M, int N, int K, const GemmWork& w,
                      hipStream_t s, const int* period = nullptr);
// out[row][n] = gelu(acc_gate) * acc_up   (packed columns, N = 2F)
template <typename T>
void gemm_geglu(const T* A, const T* Bt, T* out, int M, int N, int K, const GemmWork& w,
                hipStream_t s);
template <typename T>
void gemm_gelu(const T* A, const T* Bt, T* out, int M, int N, int K, const GemmWork& w,
               hipStream_t s);
// Raises the dynamic LDS limit of the large-M GEMM kernels (call once per
// device before the first GEMM launch).
hipError_t gemm_prepare();
// Whether gemm_partials stores the partials of plan p as bf16.
bool gemm_partials_bf16(const GemmPlan& p, bool bf16);
// Split-K GEMM that only writes its partials [KS][M][N] to w.ws; returns KS,
// or 1 (nothing launched) when the plan does not split k.  *bf16_parts: the
// partials are bf16 (the direct-to-LDS tiles), else fp32.
template <typename T>
int gemm_partials(const T* A, const T* Bt, int M, int N, int K, const GemmWork& w,
                  hipStream_t s, bool* bf16_parts);

// ------------------------------------------------------------ other kernels
// FiLM maps shared across streams.  Chunk row cr (stream b, slot k, cr =
// b K + k) normally reads its own row of the FiLM maps.  When every stream's
// noise levels equal stream 0's bit for bit, identical rows are computed
// once: the step's period flag then holds K and chunk row cr reads row
// cr % K (stream 0's), else it holds 0.  Readers take the flag's address
// (`period`, nullptr: no sharing) and load it once.
__device__ __forceinline__ int film_period(const int* period) { return period ? *period : 0; }
__device__ __forceinline__ int film_row(int cr, int per) { return per ? cr % per : cr; }

// e[row] = timestep embedding of t[row]; with `period`, one workgroup also
// sets the period flag for rows of K slots per stream (K if every row's t
// equals, bit for bit, that of the same slot of stream 0, else 0).
template <typename T>
void launch_time_embed(const float* t, T* e, int rows, int width, hipStream_t s,
                       int* period = nullptr, int K = 0);
// xs (optional, only where head_fusable): a copy of x for the fused Euler
// update of launch_final_euler.  `period` (here and below): the FiLM-row
// sharing flag described above, or nullptr.
template <typename T>
void launch_embed_adarms(const float* x, const float* w_in, const float* b_in, float* h,
                         const float* mod, int mod_ld, int chunk_len, float eps, T* u, int rows,
                         int A, int W, hipStream_t s, float* xs = nullptr,
                         const int* period = nullptr);
// h += gate * sum_z part[z] (split order); then, if norm_off >= 0,
// u = rmsnorm(h) (1 + scale) + shift with the modulation at norm_off.
// part holds bf16 values when bf16_parts, else fp32.  [pf, pf + pf_bytes)
// (the next GEMM's weights, or nullptr) is pulled into the memory-side cache
// meanwhile.
template <typename T>
void launch_resid_norm(const void* part, bool bf16_parts, int ks, float* h, const float* mod,
                       int mod_ld, int gate_off, int norm_off, int chunk_len, float eps, T* u,
                       int rows, int W, const void* pf, size_t pf_bytes, hipStream_t s,
                       const int* period = nullptr);
template <typename T>
void launch_adarms(const float* h, const float* mod, int mod_ld, int scale_off, int chunk_len,
                   float eps, T* u, int rows, int W, hipStream_t s, const int* period = nullptr);
void launch_final(const float* h, const float* mod, int mod_ld, int scale_off, int chunk_len,
                  float eps, const float* w_out, const float* b_out, float* v, int rows, int W,
                  int A, hipStream_t s, const int* period = nullptr);
// Destination of the Euler update fused into the velocity head (Algorithm 1:
// x_k <- x_k - dt_k v_k, emit slot 0, shift, refill slot K-1): the caller's
// buffer, the copy xs of it taken by the embedding at the start of the step,
// t per slot, the emitted chunk, and the device noise / valid-slot state.
struct EulerDest {
  float* buf;
  const float* xs;
  const float* t;
  float* out;
  uint64_t* noise_state;
  uint32_t* ticket;
  int* n_valid;
  int K;
};
// Whether the few-row head (and the fused Euler update) applies.
bool head_fusable(int rows, int W, int A);
// The velocity head with the Euler update, emission, shift and refill of
// launch_euler_shift fused in (same rounding, same noise); v is not stored.
void launch_final_euler(const float* h, const float* mod, int mod_ld, int scale_off, int chunk_len,
                        float eps, const float* w_out, const float* b_out, int rows, int W, int A,
                        const EulerDest& eu, hipStream_t s, const int* period = nullptr);
void launch_euler_shift(float* buffer, const float* t, const float* v, float* out,
                        const uint64_t* noise_state, uint32_t* ticket, int* n_valid, int B, int K,
                        int CA, hipStream_t s);
void launch_seq_euler(float* x, const float* v, const float* tsched, int j, int n, hipStream_t s);
void launch_cold_start(float* buffer, uint64_t* noise_state, int* n_valid, int b0, int nb, int K,
                       int CA, hipStream_t s);
void launch_copy_f32(float* dst, const float* src, size_t n, hipStream_t s);
void launch_fill_t(float* t, const float* tsched, int j, int B, hipStream_t s);
template <typename T>
void launch_prefix_copy(const T* k, const T* v, int L, int B, int src_batch, int ld, int Hkv,
                        int dh, T* karena, T* vtarena, int Bmax, int S, const int* len,
                        hipStream_t s);

// Arena row of a stream's first buffer token: the prefix length rounded up
// to a multiple of 8, so the QKV epilogue's runs of four tokens of V^T (8
// bytes) start aligned for every prefix length.  Rows [P, buffer_row0(P))
// hold zeros or an earlier prefix's finite values and are never visible.
__host__ __device__ __forceinline__ int buffer_row0(int P) { return (P + 7) & ~7; }

struct AttnArgs {
  const void* q;        // [B*tokens][Hq][dh]
  const void* karena;   // layer base [Bmax][Hkv][S][dh]
  const void* vtarena;  // layer base [Bmax][Hkv][dh][S]
  const int* len;
  void* o;              // [B*tokens][Hq*dh]
  void* part_o;         // [n_split][B*tokens*Hq][dh] element type, normalised
  float* part_ml;       // [n_split][B*tokens*Hq][2]
  int B, tokens, chunk_len, n_q_heads, n_kv_heads, head_dim, S, n_split;
  const int* n_valid;   // [B] non-padding slots per stream (the last n_valid slots)
  int mask_mode;        // FV_MASK_*
  const void* pf;       // prefetched into the memory-side cache meanwhile (or nullptr)
  size_t pf_bytes;
  const int* bg_order;  // [B*Hkv] (stream, kv head) pairs in die order (die_order)
};

// The (stream, kv head) pairs in the order in which a large attention grid
// hands them to the 8 dies (die x takes the x-th eighth of the list): each
// die gets the same number of pairs and about the same total prefix length,
// the longest pairs first within a die.  Identity when B*Hkv is not a
// multiple of 8.
void die_order(const int* len, int B, int Hkv, int* order);

// Buffer chunks [lo, hi) visible to the queries of chunk kq (see the mask
// modes in the C header); slots before `first` are cold-start padding.
__host__ __device__ __forceinline__ void visible_chunks(int kq, int K, int first, int mode,
                                                        int& lo, int& hi) {
  if (kq < first || mode == FV_MASK_ISOLATED) {
    lo = kq;
    hi = kq + 1;
  } else if (mode == FV_MASK_CHUNK_CAUSAL) {
    lo = first;
    hi = kq + 1;
  } else {
    lo = first;
    hi = K;
  }
}
// parts: bit 0 launches the score/value kernel, bit 1 the split combine.
template <typename T>
void launch_attention(const AttnArgs& a, hipStream_t s, int parts = 3);
template <typename T>
int attention_row_tiles(int tokens, int n_q_heads, int n_kv_heads);
// Raises the dynamic LDS limit of the direct-load attention kernels (call
// once per device before the first launch).
hipError_t attention_prepare();

// ------------------------------------------------------------------- handle
struct GraphEntry {
  int kind = 0, batch = 0, n = 0, slot = 0;
  const void* p[4] = {nullptr, nullptr, nullptr, nullptr};
  hipGraphExec_t exec = nullptr;
  uint64_t last_use = 0;
};

struct Handle {
  fv_cfg cfg{};
  int device = 0;
  bool bf16 = true;
  int L = 0, W = 0, Hq = 0, Hkv = 0, dh = 0, F = 0, A = 0, C = 0, K = 0, T = 0;
  int Pmax = 0, Bmax = 0, S = 0;   // S: arena rows per (layer, stream, kv head)
  int Nqkv = 0, Nmod = 0, Ngu = 0;
  size_t esz = 2;                  // element size of T

  // packed weights (device)
  float* w_in = nullptr;  float* b_in = nullptr;   // fp32 [A][W], [W]
  void* w_t1 = nullptr;   float* b_t1 = nullptr;   // T [W][W] (out-major)
  void* w_t2 = nullptr;   float* b_t2 = nullptr;
  void* w_mod = nullptr;  float* b_mod = nullptr;  // T [Nmod][W], fp32 [Nmod]
  std::vector<void*> wqkv, wo, wgu, wd;            // T, out-major
  float* w_out = nullptr; float* b_out = nullptr;  // fp32 [W][A], [A]

  // prefix arena and lengths
  void* karena = nullptr;   // [L][Bmax][Hkv][S][dh]
  void* vtarena = nullptr;  // [L][Bmax][Hkv][dh][S]
  int* d_len = nullptr;
  std::vector<int32_t> len_host;   // followed on the device (d_len + Bmax) by die_order
  std::vector<int32_t> order_host;
  int batch = 0;
  bool prefix_set = false;

  // rotary tables [S][dh/2]
  float* rcos = nullptr; float* rsin = nullptr;

  // scratch
  void* e = nullptr; void* hid = nullptr; void* cond = nullptr;  // T [Bmax*K][W]
  float* mod = nullptr;                                           // [Bmax*K][Nmod]
  int* d_film_period = nullptr;   // FiLM-row sharing flag of the step (see film_row)
  const int* film_per = nullptr;  // the flag of h->mod's rows after the last velocity pass, or nullptr
  float* hres = nullptr;                                          // [Bmax*T][W]
  void* u = nullptr;                                              // T [Bmax*T][W]
  void* q = nullptr; void* o = nullptr;                           // T [Bmax*T][Hq*dh]
  void* m = nullptr;                                              // T [Bmax*T][F]
  float* v = nullptr;                                             // [Bmax][K][C][A]
  void* part_o = nullptr; float* part_ml = nullptr; int max_split = 1;
  float* seq_x = nullptr; float* seq_t = nullptr;
  std::vector<std::pair<int, float*>> tscheds;  // sequential-decode t_j tables by step count

  GemmWork gw;                    // split-K workspace and counters
  uint64_t* d_noise = nullptr;   // {seed, step}
  int* d_valid = nullptr;        // [Bmax] non-padding slots per stream (K: steady state)
  // Double-buffered observation prefix for the asynchronous pipeline: slot
  // cur_slot is the active arena (karena / vtarena / d_len point at it);
  // fv_set_prefix_async fills the other slot on the caller's copy stream.
  void* arena_k[2] = {nullptr, nullptr};
  void* arena_v[2] = {nullptr, nullptr};
  int* len_slot[2] = {nullptr, nullptr};
  std::vector<int> len_host_slot[2];
  int cur_slot = 0, staged_slot = -1, staged_batch = 0;
  bool async_ready = false;                    // second slot and events exist
  hipEvent_t ev_ready[2] = {nullptr, nullptr}; // staged prefix copied (copy stream)
  hipEvent_t ev_done[2] = {nullptr, nullptr};  // last pass that read the slot
  hipEvent_t ev_len[2] = {nullptr, nullptr};   // pinned length buffer consumed
  bool done_recorded[2] = {false, false}, len_recorded[2] = {false, false};
  int* pinned_len[2] = {nullptr, nullptr};
  int mask_mode = FV_MASK_CHUNK_CAUSAL;
  float* mod_cache = nullptr;    // [Bmax*K][Nmod] FiLM maps of a static schedule
  float* t_cache = nullptr;      // [Bmax*K] the schedule itself
  int* d_sched_period = nullptr;  // the schedule's FiLM-row sharing flag
  const int* sched_per = nullptr; // the flag its readers take, or nullptr
  int sched_batch = 0;           // batch the cached schedule was made for (0: none)
  uint32_t* d_ticket = nullptr;

  // graphs
  bool use_graphs = true;
  hipStream_t cap_stream = nullptr;
  std::vector<GraphEntry> graphs;
  uint64_t use_clock = 0;

  std::string last_error;
  std::vector<void*> allocations;
  size_t device_bytes = 0;
};

}  // namespace fv
