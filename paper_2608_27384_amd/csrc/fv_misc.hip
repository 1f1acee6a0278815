// Element-wise and row-wise kernels of the decode step.
#include <algorithm>

#include "fv_internal.h"

namespace fv {

namespace {

constexpr double kTwoPi = 6.283185307179586476925286766559;

// ------------------------------------------------------------------ helpers

// -------------------------------------------------------- time embedding
// e[row] = [sin(2 pi t / p_i) | cos(2 pi t / p_i)], p_i = 4e-3 * (4/4e-3)^(i/(W/2-1)),
// evaluated in fp64 (the timestep embedding that drives FiLM, Appendix
// "Model architecture").  With `period`, workgroup 0 also sets the FiLM-row
// sharing flag: K when every stream's K noise levels equal stream 0's bit
// for bit (equal t gives equal maps, so stream 0's rows serve all), else 0.
template <typename T>
__global__ void time_embed_kernel(const float* __restrict__ t, T* __restrict__ e, int rows,
                                  int width, int* __restrict__ period, int K) {
  if (period && blockIdx.x == 0) {
    int same = 1;
    for (int r = K + (int)threadIdx.x; r < rows; r += blockDim.x)
      same &= __float_as_uint(t[r]) == __float_as_uint(t[r % K]);
    same = __syncthreads_and(same);
    if (threadIdx.x == 0) *period = same ? K : 0;
  }
  const int half = width / 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * half) return;
  const int row = idx / half, i = idx - row * half;
  const double p_i = 4e-3 * pow(4.0 / 4e-3, (double)i / (double)(half - 1));
  const double ang = kTwoPi * (double)t[row] / p_i;
  double sv, cv;
  sincos(ang, &sv, &cv);
  e[(size_t)row * width + i] = from_f32<T>((float)sv);
  e[(size_t)row * width + half + i] = from_f32<T>((float)cv);
}

// ---------------------------------- action embedding + first FiLM RMSNorm
// h[row] = x[row] w_in + b_in (fp32), then u[row] = rmsnorm(h) (1 + scale) +
// shift with norm 0's modulation of the row's chunk.  A block takes
// kEmbRows rows; thread t owns 4 consecutive columns (per 1024-column chunk)
// of every row, reads w_in once for all rows in batches of independent
// loads and keeps the x rows in LDS.
constexpr int kEmbRows = 8;
// Row count from which the embedding and the velocity head switch to their
// weights-in-registers variants.
constexpr int kManyRows = 4096;

__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

template <typename T, int NC>
__global__ __launch_bounds__(256) void embed_adarms_kernel(
    const float* __restrict__ x, const float* __restrict__ w_in, const float* __restrict__ b_in,
    float* __restrict__ h, const float* __restrict__ mod, int mod_ld, int chunk_len, float eps,
    T* __restrict__ u, int rows, int A, int W, const int* __restrict__ period) {
  // thread t owns columns 4t + 1024 i (i < NC, W <= 1024 NC) of kEmbRows
  // rows; the modulation and the first weight batch are requested before
  // anything waits, and h stays in registers between the embedding and the
  // norm
  constexpr int AB = 16;  // weight rows per batch
  __shared__ float sx[64][kEmbRows];  // x transposed: one action entry of every row is contiguous
  __shared__ float sred[kEmbRows][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.x * kEmbRows;
  const int per = film_period(period);
  const f32x4 zero4 = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 sv[NC][kEmbRows], bv[NC][kEmbRows], acc[NC][kEmbRows];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = 4 * tid + 1024 * i;
    const bool ok = c < W;
    const f32x4 bias = ok ? *reinterpret_cast<const f32x4*>(b_in + c) : zero4;
#pragma unroll
    for (int r = 0; r < kEmbRows; ++r) {
      const int row = min(row0 + r, rows - 1);
      const float* sc = mod + (size_t)film_row(row / chunk_len, per) * mod_ld;
      sv[i][r] = ok ? *reinterpret_cast<const f32x4*>(sc + c) : zero4;
      bv[i][r] = ok ? *reinterpret_cast<const f32x4*>(sc + W + c) : zero4;
      acc[i][r] = bias;
    }
  }
  for (int idx = tid; idx < kEmbRows * A; idx += 256) {
    const int r = idx / A, a = idx - r * A;
    sx[a][r] = row0 + r < rows ? x[(size_t)(row0 + r) * A + a] : 0.f;
  }
  __syncthreads();
  for (int a0 = 0; a0 < A; a0 += AB) {
    f32x4 wv[NC][AB];
#pragma unroll
    for (int i = 0; i < NC; ++i)
#pragma unroll
      for (int j = 0; j < AB; ++j) {
        const int c = 4 * tid + 1024 * i;
        wv[i][j] = (c < W && a0 + j < A) ? *reinterpret_cast<const f32x4*>(w_in + (size_t)(a0 + j) * W + c)
                                         : zero4;
      }
#pragma unroll
    for (int j = 0; j < AB; ++j)
#pragma unroll
      for (int r = 0; r < kEmbRows; ++r) {
        const float xv = a0 + j < A ? sx[a0 + j][r] : 0.f;
#pragma unroll
        for (int i = 0; i < NC; ++i) acc[i][r] += xv * wv[i][j];
      }
  }
  float ss[kEmbRows];
#pragma unroll
  for (int r = 0; r < kEmbRows; ++r) {
    ss[r] = 0.f;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = 4 * tid + 1024 * i;
      if (c < W) {
        if (row0 + r < rows) *reinterpret_cast<f32x4*>(h + (size_t)(row0 + r) * W + c) = acc[i][r];
        ss[r] += acc[i][r][0] * acc[i][r][0] + acc[i][r][1] * acc[i][r][1] +
                 acc[i][r][2] * acc[i][r][2] + acc[i][r][3] * acc[i][r][3];
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kEmbRows; ++r) {
    const float v = wave_sum(ss[r]);
    if (lane == 0) sred[r][wave] = v;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kEmbRows; ++r) {
    const int row = row0 + r;
    if (row >= rows) break;
    const float tot = sred[r][0] + sred[r][1] + sred[r][2] + sred[r][3];
    const float rinv = 1.0f / sqrtf(tot / (float)W + eps);
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = 4 * tid + 1024 * i;
      if (c >= W) continue;
      const f32x4 hv = acc[i][r];
      store4<T>(u + (size_t)row * W + c, hv[0] * rinv * (1.0f + sv[i][r][0]) + bv[i][r][0],
                hv[1] * rinv * (1.0f + sv[i][r][1]) + bv[i][r][1],
                hv[2] * rinv * (1.0f + sv[i][r][2]) + bv[i][r][2],
                hv[3] * rinv * (1.0f + sv[i][r][3]) + bv[i][r][3]);
    }
  }
}

// Few rows, W <= 1024, A <= 32: kEmbSmallRows rows per block, so the grid
// spreads over the chip; every load of the kernel (the rows of x, all of
// w_in's rows at the thread's 4 columns, the modulation and the bias) is
// issued before any is used, unconditionally (indices clamped, the extra
// terms multiplied by zero), so the block waits for memory once.
constexpr int kEmbSmallRows = 2;
template <typename T>
__global__ __launch_bounds__(256) void embed_adarms_small_kernel(
    const float* __restrict__ x, const float* __restrict__ w_in, const float* __restrict__ b_in,
    float* __restrict__ h, const float* __restrict__ mod, int mod_ld, int chunk_len, float eps,
    T* __restrict__ u, int rows, int A, int W, float* __restrict__ xs,
    const int* __restrict__ period) {
  constexpr int R = kEmbSmallRows, AM = 32;
  __shared__ float sred[R][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.x * R;
  const int c = min(4 * tid, W - 4);
  const bool own = 4 * tid < W;
  const int per = film_period(period);
  float xv[R][AM];
  f32x4 wv[AM], sv[R], bv[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int row = min(row0 + r, rows - 1);
#pragma unroll
    for (int a = 0; a < AM; ++a) xv[r][a] = x[(size_t)row * A + min(a, A - 1)];
    const float* sc = mod + (size_t)film_row(row / chunk_len, per) * mod_ld;
    sv[r] = *reinterpret_cast<const f32x4*>(sc + c);
    bv[r] = *reinterpret_cast<const f32x4*>(sc + W + c);
  }
#pragma unroll
  for (int a = 0; a < AM; ++a) wv[a] = *reinterpret_cast<const f32x4*>(w_in + (size_t)min(a, A - 1) * W + c);
  const f32x4 bias = *reinterpret_cast<const f32x4*>(b_in + c);
  __builtin_amdgcn_sched_barrier(0);
  // a copy of the block's rows of x for the fused Euler update (xs != null),
  // after every other load is on its way
  if (xs && tid < R * A && row0 * A + tid < rows * A)
    xs[(size_t)row0 * A + tid] = x[(size_t)row0 * A + tid];
  f32x4 acc[R];
  float ss[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    acc[r] = bias;
#pragma unroll
    for (int a = 0; a < AM; ++a) acc[r] += (a < A ? xv[r][a] : 0.f) * wv[a];
    ss[r] = own ? acc[r][0] * acc[r][0] + acc[r][1] * acc[r][1] + acc[r][2] * acc[r][2] +
                      acc[r][3] * acc[r][3]
                : 0.f;
    if (own && row0 + r < rows) *reinterpret_cast<f32x4*>(h + (size_t)(row0 + r) * W + c) = acc[r];
    const float v = wave_sum(ss[r]);
    if (lane == 0) sred[r][wave] = v;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int row = row0 + r;
    if (row >= rows || !own) continue;
    const float tot = sred[r][0] + sred[r][1] + sred[r][2] + sred[r][3];
    const float rinv = 1.0f / sqrtf(tot / (float)W + eps);
    store4<T>(u + (size_t)row * W + c, acc[r][0] * rinv * (1.0f + sv[r][0]) + bv[r][0],
              acc[r][1] * rinv * (1.0f + sv[r][1]) + bv[r][1],
              acc[r][2] * rinv * (1.0f + sv[r][2]) + bv[r][2],
              acc[r][3] * rinv * (1.0f + sv[r][3]) + bv[r][3]);
  }
}

// Many rows (W <= 1024, A <= 32): thread t keeps its four columns of w_in in
// registers and the block runs batches of kEmbRows rows through them, so
// w_in is read once per block instead of once per batch.  The kernel holds
// more than 256 registers per lane, so one workgroup fits a CU, and the grid
// is sized to one round of them (launch_embed_adarms).  The next batch's x is requested at the
// start of a batch and its modulation rows right after its arithmetic, so
// their latency hides behind the arithmetic and the row-sum barrier.  Two barriers per batch: the one after the row sums
// also keeps the next batch's x out of sx until every wave has read it, and
// the one after sx is written keeps the next row sums out of sred until the
// current ones are read.
template <typename T>
__global__ __launch_bounds__(256) void embed_adarms_rows_kernel(
    const float* __restrict__ x, const float* __restrict__ w_in, const float* __restrict__ b_in,
    float* __restrict__ h, const float* __restrict__ mod, int mod_ld, int chunk_len, float eps,
    T* __restrict__ u, int rows, int A, int W, int rows_per_block, const int* __restrict__ period) {
  constexpr int R = kEmbRows;
  __shared__ __attribute__((aligned(16))) float sx[32][R];
  __shared__ float sred[R][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = 4 * tid;
  const bool ok = c < W;
  const int cc = min(c, W - 4);
  const f32x4 zero4 = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 wv[32];
#pragma unroll
  for (int a = 0; a < 32; ++a)
    wv[a] = ok && a < A ? *reinterpret_cast<const f32x4*>(w_in + (size_t)a * W + c) : zero4;
  const f32x4 bias = ok ? *reinterpret_cast<const f32x4*>(b_in + c) : zero4;
  const int per = film_period(period);
  const int rbeg = blockIdx.x * rows_per_block;
  const int rend = min(rows, rbeg + rows_per_block);
  // x of a batch: thread (r, a) = (tid / 32, tid % 32) holds entry a of row
  // r (entries a >= A are zero, and so are their weights)
  const int xr_r = tid >> 5, xr_a = tid & 31;
  auto load_x = [&](int row0) __attribute__((always_inline)) {
    return row0 + xr_r < rend && xr_a < A ? x[(size_t)(row0 + xr_r) * A + xr_a] : 0.f;
  };
  float xr = load_x(rbeg);
  for (int row0 = rbeg; row0 < rend; row0 += R) {
    sx[xr_a][xr_r] = xr;
    xr = load_x(row0 + R);
    __syncthreads();
    f32x4 acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = bias;
#pragma unroll
    for (int a = 0; a < 32; ++a) {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(&sx[a][0]);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(&sx[a][4]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        acc[r] += x0[r] * wv[a];
        acc[4 + r] += x1[r] * wv[a];
      }
      if ((a & 7) == 7) __builtin_amdgcn_sched_barrier(0);  // bounds the LDS reads in flight
    }
    // the modulation rows, in flight during the stores and the row-sum barrier
    f32x4 sv[R], bv[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int row = min(row0 + r, rend - 1);
      const float* sc = mod + (size_t)film_row(row / chunk_len, per) * mod_ld;
      sv[r] = *reinterpret_cast<const f32x4*>(sc + cc);
      bv[r] = *reinterpret_cast<const f32x4*>(sc + W + cc);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float ss = acc[r][0] * acc[r][0] + acc[r][1] * acc[r][1] + acc[r][2] * acc[r][2] +
                       acc[r][3] * acc[r][3];
      if (ok && row0 + r < rend) *reinterpret_cast<f32x4*>(h + (size_t)(row0 + r) * W + c) = acc[r];
      const float v = wave_sum(ok ? ss : 0.f);
      if (lane == 0) sred[r][wave] = v;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int row = row0 + r;
      if (row >= rend || !ok) break;
      const float tot = sred[r][0] + sred[r][1] + sred[r][2] + sred[r][3];
      const float rinv = 1.0f / sqrtf(tot / (float)W + eps);
      store4<T>(u + (size_t)row * W + c, acc[r][0] * rinv * (1.0f + sv[r][0]) + bv[r][0],
                acc[r][1] * rinv * (1.0f + sv[r][1]) + bv[r][1],
                acc[r][2] * rinv * (1.0f + sv[r][2]) + bv[r][2],
                acc[r][3] * rinv * (1.0f + sv[r][3]) + bv[r][3]);
    }
  }
}

// --------------------------------------- gated residual + next FiLM RMSNorm
// One block per row: h[row] += gate[chunk] * sum_z part[z][row] (split order,
// fp32 sums of the partials, which are stored as P), then (norm_off >= 0)
// u[row] = rmsnorm(h) (1 + scale) + shift.  Thread t owns columns
// 4t + 1024 q (q < NQ).  Every load of the block's row is issued before any
// is used, with no condition on the loads themselves: the split index is
// clamped to ks - 1 (the KSM slots past ks re-read split ks - 1 and are
// dropped from the sum) and the column to W - 4 (dropped likewise), so the
// compiler does not wait for each load on its own.  The prefetch of the next
// GEMM's weights is issued after them: the in-order memory counter then
// never makes this kernel's own loads wait behind it.
template <typename P> struct RawPart;
template <> struct RawPart<bf16_t> {
  typedef u32x2 type;  // four bf16
  __device__ static __forceinline__ type load(const bf16_t* p) {
    return *reinterpret_cast<const u32x2*>(p);
  }
  __device__ static __forceinline__ f32x4 unpack(type v) {
    return f32x4{__uint_as_float(v[0] << 16), __uint_as_float(v[0] & 0xffff0000u),
                 __uint_as_float(v[1] << 16), __uint_as_float(v[1] & 0xffff0000u)};
  }
};
template <> struct RawPart<float> {
  typedef f32x4 type;
  __device__ static __forceinline__ type load(const float* p) {
    return *reinterpret_cast<const f32x4*>(p);
  }
  __device__ static __forceinline__ f32x4 unpack(type v) { return v; }
};

template <typename T, typename P, int KSM, int NQ>
__global__ __launch_bounds__(256) void resid_norm_kernel(const P* __restrict__ part, int ks,
                                                         float* __restrict__ h,
                                                         const float* __restrict__ mod,
                                                         int mod_ld, int gate_off, int norm_off,
                                                         int chunk_len, float eps,
                                                         T* __restrict__ u, int rows, int W,
                                                         const void* pf, size_t pf_bytes,
                                                         const int* __restrict__ period) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const float* mrow = mod + (size_t)film_row(row / chunk_len, film_period(period)) * mod_ld;
  const int nrm = norm_off >= 0 ? norm_off : 0;
  typename RawPart<P>::type pr[NQ][KSM];
  f32x4 g[NQ], hv[NQ], svq[NQ], bvq[NQ];
  int col[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    col[q] = 4 * tid + 1024 * q;
    const int c = min(col[q], W - 4);
#pragma unroll
    for (int z = 0; z < KSM; ++z)
      pr[q][z] = RawPart<P>::load(part + ((size_t)min(z, ks - 1) * rows + row) * W + c);
    g[q] = *reinterpret_cast<const f32x4*>(mrow + gate_off + c);
    hv[q] = *reinterpret_cast<const f32x4*>(h + (size_t)row * W + c);
    svq[q] = *reinterpret_cast<const f32x4*>(mrow + nrm + c);
    bvq[q] = *reinterpret_cast<const f32x4*>(mrow + nrm + W + c);
  }
  Prefetch<8, 256> pre;
  pre.issue(pf, pf_bytes, h);
  float ss = 0.f;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    f32x4 acc = RawPart<P>::unpack(pr[q][0]);
#pragma unroll
    for (int z = 1; z < KSM; ++z)
      if (z < ks) acc += RawPart<P>::unpack(pr[q][z]);
    hv[q] += g[q] * acc;
    if (col[q] < W) {
      *reinterpret_cast<f32x4*>(h + (size_t)row * W + col[q]) = hv[q];
      ss += hv[q][0] * hv[q][0] + hv[q][1] * hv[q][1] + hv[q][2] * hv[q][2] +
            hv[q][3] * hv[q][3];
    }
  }
  if (norm_off < 0) {
    pre.retire();
    return;
  }
  const float rinv = 1.0f / sqrtf(block_sum_256(ss, red) / (float)W + eps);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (col[q] < W) {
      const f32x4 sv = svq[q], bv = bvq[q], x = hv[q];
      store4<T>(u + (size_t)row * W + col[q], x[0] * rinv * (1.0f + sv[0]) + bv[0],
                x[1] * rinv * (1.0f + sv[1]) + bv[1], x[2] * rinv * (1.0f + sv[2]) + bv[2],
                x[3] * rinv * (1.0f + sv[3]) + bv[3]);
    }
  }
  pre.retire();
}

// -------------------------------------------------- FiLM-conditioned RMSNorm
// u = h / sqrt(mean(h^2) + eps) * (1 + scale[chunk]) + shift[chunk]; one wave per row.
template <typename T>
__global__ __launch_bounds__(256) void adarms_kernel(const float* __restrict__ h,
                                                     const float* __restrict__ mod, int mod_ld,
                                                     int scale_off, int chunk_len, float eps,
                                                     T* __restrict__ u, int rows, int W,
                                                     const int* __restrict__ period) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  constexpr int NV = 2048 / 256;  // 4-float groups per lane for W <= 2048
  const float* hr = h + (size_t)row * W;
  const float* sc =
      mod + (size_t)film_row(row / chunk_len, film_period(period)) * mod_ld + scale_off;
  f32x4 x[NV], sv[NV], bv[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {  // all loads of the row first
    const int c = 4 * lane + 256 * i;
    const bool ok = c < W;
    x[i] = ok ? *reinterpret_cast<const f32x4*>(hr + c) : f32x4{0.f, 0.f, 0.f, 0.f};
    sv[i] = ok ? *reinterpret_cast<const f32x4*>(sc + c) : f32x4{0.f, 0.f, 0.f, 0.f};
    bv[i] = ok ? *reinterpret_cast<const f32x4*>(sc + W + c) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) ss += x[i][0] * x[i][0] + x[i][1] * x[i][1] + x[i][2] * x[i][2] + x[i][3] * x[i][3];
  ss = wave_sum(ss);
  const float rinv = 1.0f / sqrtf(ss / (float)W + eps);
  T* ur = u + (size_t)row * W;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = 4 * lane + 256 * i;
    if (c < W)
      store4<T>(ur + c, x[i][0] * rinv * (1.0f + sv[i][0]) + bv[i][0],
                x[i][1] * rinv * (1.0f + sv[i][1]) + bv[i][1],
                x[i][2] * rinv * (1.0f + sv[i][2]) + bv[i][2],
                x[i][3] * rinv * (1.0f + sv[i][3]) + bv[i][3]);
  }
}

// ------------------------------------- final FiLM RMSNorm + velocity head
// v[row] = (rmsnorm(h) (1 + scale) + shift) w_out + b_out, fp32.  A block
// handles kFinalRows rows: each wave normalises one row into LDS (every load
// of the row issued before use).  Then thread (part, a) sums output column a
// of all the block's rows over one contiguous slice of the width, reading
// w_out in batches of 32 independent loads that serve every row, and the
// slices are added in a fixed order.
constexpr int kFinalRows = 4;
constexpr int kMaxW = 2048;
__global__ __launch_bounds__(256) void final_kernel(const float* __restrict__ h,
                                                    const float* __restrict__ mod, int mod_ld,
                                                    int scale_off, int chunk_len, float eps,
                                                    const float* __restrict__ w_out,
                                                    const float* __restrict__ b_out,
                                                    float* __restrict__ v, int rows, int W,
                                                    int A, const int* __restrict__ period) {
  extern __shared__ float smem[];  // su [kFinalRows][W], sp [parts][kFinalRows][A]
  float* su = smem;
  float* sp = su + kFinalRows * W;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, tid = threadIdx.x;
  const int row0 = blockIdx.x * kFinalRows;
  {
    const int row = min(row0 + wave, rows - 1);
    const float* hr = h + (size_t)row * W;
    const float* sc =
        mod + (size_t)film_row(row / chunk_len, film_period(period)) * mod_ld + scale_off;
    constexpr int NPL = kMaxW / 64;
    float hv[NPL], sv[NPL], bv[NPL];
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      const int c = lane + 64 * i;
      hv[i] = c < W ? hr[c] : 0.f;
      sv[i] = c < W ? sc[c] : 0.f;
      bv[i] = c < W ? sc[W + c] : 0.f;
    }
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NPL; ++i) ss += hv[i] * hv[i];
    ss = wave_sum(ss);
    const float rinv = 1.0f / sqrtf(ss / (float)W + eps);
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      const int c = lane + 64 * i;
      if (c < W) su[wave * W + c] = hv[i] * rinv * (1.0f + sv[i]) + bv[i];
    }
  }
  __syncthreads();
  // thread (part, a): output column a of all kFinalRows rows over the
  // width slice `part`; weight loads go out 32 at a time, each used for
  // every row; the slices are then added in a fixed order
  constexpr int KB = 32;
  const int parts = 256 / A;
  const int part = tid / A, a = tid - part * A;
  const int kr = (W + parts - 1) / parts;
  const int k0 = part * kr, k1 = min(W, k0 + kr);
  float acc[kFinalRows] = {};
  if (part < parts) {
    for (int kb = k0; kb < k1; kb += KB) {
      float wv[KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) wv[j] = kb + j < k1 ? w_out[(size_t)(kb + j) * A + a] : 0.f;
#pragma unroll
      for (int j = 0; j < KB; ++j)
#pragma unroll
        for (int r = 0; r < kFinalRows; ++r)
          acc[r] = fmaf(kb + j < k1 ? su[r * W + kb + j] : 0.f, wv[j], acc[r]);
    }
#pragma unroll
    for (int r = 0; r < kFinalRows; ++r) sp[(part * kFinalRows + r) * A + a] = acc[r];
  }
  __syncthreads();
  if (tid < kFinalRows * A) {
    const int r = tid / A, aa = tid - r * A;
    if (row0 + r < rows) {
      float tot = b_out[aa];
      for (int p = 0; p < parts; ++p) tot += sp[(p * kFinalRows + r) * A + aa];
      v[(size_t)(row0 + r) * A + aa] = tot;
    }
  }
}

// ------------------------------------------------------------ Philox4x32-10
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    const uint32_t hi0 = __umulhi(M0, c[0]), lo0 = M0 * c[0];
    const uint32_t hi1 = __umulhi(M1, c[2]), lo1 = M1 * c[2];
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

__device__ __forceinline__ void box_muller(uint32_t r0, uint32_t r1, float* z0, float* z1) {
  const double u0 = ((double)r0 + 0.5) * 2.3283064365386962890625e-10;  // 2^-32
  const double u1 = ((double)r1 + 0.5) * 2.3283064365386962890625e-10;
  const double rad = sqrt(-2.0 * log(u0));
  double s, c;
  sincos(kTwoPi * u1, &s, &c);
  *z0 = (float)(rad * c);
  *z1 = (float)(rad * s);
}

// The Euler update, emission, shift and refill of one group of 4 elements
// (group j of its chunk), with the same rounding as euler_shift_kernel: x'
// = x - dt v, the product and the difference rounded separately.  x comes
// from a copy of the buffer taken at the start of the step, so writing the
// shifted slot k - 1 in place races with no reader.
__device__ __forceinline__ void euler_group(const EulerDest& eu, f32x4 v, f32x4 x, float dt, int b,
                                            int k, bool full, int j, size_t base, int CA,
                                            uint64_t seed, uint64_t step) {
#pragma clang fp contract(off)
  float xn[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float p = dt * v[e];
    xn[e] = x[e] - p;
  }
  if (k == 0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) eu.out[(size_t)b * CA + (base - (size_t)b * eu.K * CA) + e] = full ? xn[e] : 0.f;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) eu.buf[base - CA + e] = xn[e];
  }
  if (k == eu.K - 1) {
    uint32_t c[4] = {(uint32_t)j, (uint32_t)step, (uint32_t)(step >> 32), 0u};
    const uint64_t sb = seed + (uint64_t)b;
    philox4x32_10(c, (uint32_t)sb, (uint32_t)(sb >> 32));
    float z[4];
    box_muller(c[0], c[1], &z[0], &z[1]);
    box_muller(c[2], c[3], &z[2], &z[3]);
#pragma unroll
    for (int e = 0; e < 4; ++e) eu.buf[base + e] = z[e];
  }
}

// After every block has read the step counter and the valid-slot counts,
// the last block to finish advances them.
__device__ __forceinline__ void euler_finish(const EulerDest& eu, int B, uint64_t step) {
  __shared__ int s_last;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t done =
        __hip_atomic_fetch_add(eu.ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = done == gridDim.x - 1;
    if (s_last) {
      eu.noise_state[1] = step + 1;
      __hip_atomic_store(eu.ticket, 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (s_last)
    for (int bb = threadIdx.x; bb < B; bb += blockDim.x) eu.n_valid[bb] = min(eu.n_valid[bb] + 1, eu.K);
}

// Few rows, W <= 1024, A <= 32 (A % 4 == 0): the same head with one wait
// for memory.  Every load is issued first, unconditionally: wave w's row
// (h, scale, shift; 16 per lane) and thread (part, q)'s 32 rows of w_out at
// outputs 4q..4q+3, part = tid / 8 taking rows 32 part .. +32.  After the
// normalised rows are in LDS, each thread forms its partial sums for the
// block's rows; the 8 parts of a wave are added across lanes (lane bits 5,
// 4, 3) and the 4 waves in a fixed order.
__device__ __forceinline__ float sum_lane_bits_543(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  return dpp_add<0x128>(x);  // row_ror:8
}
constexpr int kFinalSmallRows = 4;
template <bool EU>
__global__ __launch_bounds__(256) void final_small_kernel(const float* __restrict__ h,
                                                          const float* __restrict__ mod, int mod_ld,
                                                          int scale_off, int chunk_len, float eps,
                                                          const float* __restrict__ w_out,
                                                          const float* __restrict__ b_out,
                                                          float* __restrict__ v, int rows, int W,
                                                          int A, EulerDest eu,
                                                          const int* __restrict__ period) {
  constexpr int R = kFinalSmallRows, NPL = 16, KR = 32;
  __shared__ __attribute__((aligned(16))) float su[R][1024];
  __shared__ f32x4 sp[4][R][8];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int row0 = blockIdx.x * R;
  const int q = tid & 7, part = tid >> 3;
  const int qa = min(4 * q, A - 4);
  const int k0 = part * KR;
  // output thread (r, q) = (tid / 8, tid % 8) of the block's rows: its bias
  // and, with the Euler update, its slot's inputs, loaded up front
  const int orow = min(row0 + (tid >> 3 & (R - 1)), rows - 1);
  const f32x4 bo = *reinterpret_cast<const f32x4*>(b_out + qa);
  int ek = 0, eb = 0, nvalid = 0;
  float dt = 0.f;
  f32x4 x4 = {0.f, 0.f, 0.f, 0.f};
  uint64_t seed = 0, step = 0;
  if constexpr (EU) {
    const int T = eu.K * chunk_len;
    eb = orow / T;
    ek = (orow - eb * T) / chunk_len;
    const float tk = eu.t[(size_t)eb * eu.K + ek];
    const float tp = eu.t[(size_t)eb * eu.K + max(ek - 1, 0)];
    dt = tk - (ek > 0 ? tp : 0.f);
    x4 = *reinterpret_cast<const f32x4*>(eu.xs + (size_t)orow * A + qa);
    nvalid = eu.n_valid[eb];
    seed = eu.noise_state[0];
    step = eu.noise_state[1];
  }
  // loads: the head weights of this thread's slice, then wave's row
  f32x4 wv[KR];
#pragma unroll
  for (int j = 0; j < KR; ++j)
    wv[j] = *reinterpret_cast<const f32x4*>(w_out + (size_t)min(k0 + j, W - 1) * A + qa);
  const int row = min(row0 + wave, rows - 1);
  const float* hr = h + (size_t)row * W;
  const float* sc =
      mod + (size_t)film_row(row / chunk_len, film_period(period)) * mod_ld + scale_off;
  float hv[NPL], sv[NPL], bv[NPL];
#pragma unroll
  for (int i = 0; i < NPL; ++i) {
    const int cc = min(lane + 64 * i, W - 1);
    hv[i] = hr[cc];
    sv[i] = sc[cc];
    bv[i] = sc[W + cc];
  }
  __builtin_amdgcn_sched_barrier(0);
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NPL; ++i) ss += lane + 64 * i < W ? hv[i] * hv[i] : 0.f;
  ss = wave_sum(ss);
  const float rinv = 1.0f / sqrtf(ss / (float)W + eps);
#pragma unroll
  for (int i = 0; i < NPL; ++i)
    su[wave][lane + 64 * i] = lane + 64 * i < W ? hv[i] * rinv * (1.0f + sv[i]) + bv[i] : 0.f;
  __syncthreads();
  // columns past W read zeros from LDS (written above), so their weights
  // (clamped to row W - 1) contribute nothing
#pragma unroll
  for (int r = 0; r < R; ++r) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KR; j += 4) {
      const f32x4 x4 = *reinterpret_cast<const f32x4*>(&su[r][k0 + j]);
      acc += x4[0] * wv[j];
      acc += x4[1] * wv[j + 1];
      acc += x4[2] * wv[j + 2];
      acc += x4[3] * wv[j + 3];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = sum_lane_bits_543(acc[e]);
    if (lane < 8) sp[wave][r][lane] = acc;
  }
  __syncthreads();
  if (tid < R * 8) {
    const int r = tid >> 3;
    if (row0 + r < rows && 4 * q < A) {
      const f32x4 vv = sp[0][r][q] + sp[1][r][q] + sp[2][r][q] + sp[3][r][q] + bo;
      if constexpr (!EU) {
        *reinterpret_cast<f32x4*>(v + (size_t)(row0 + r) * A + 4 * q) = vv;
      } else {
        euler_group(eu, vv, x4, dt, eb, ek, nvalid >= eu.K, (row0 + r) % chunk_len * (A / 4) + q,
                    (size_t)(row0 + r) * A + 4 * q, chunk_len * A, seed, step);
      }
    }
  }
  if constexpr (EU) euler_finish(eu, rows / (eu.K * chunk_len), step);
}

// Many rows (W <= 1024, A <= 32, A % 4 == 0): 512 threads; thread (part, q)
// keeps rows 16 part .. 16 part + 15 of w_out at outputs 4q .. 4q + 3 in
// registers and the block runs batches of 8 rows (one per wave) through
// them: w_out is read once per block, and every normalised value read from
// LDS feeds four outputs.  The 8 parts of a wave are added across lanes
// (lane bits 5, 4, 3) and the 8 waves in a fixed order.  One workgroup per
// CU and a grid of one round (launch_final); each wave requests its next row
// (h, scale, shift) as soon as the current one is in LDS, so the load latency
// hides behind the head's arithmetic.  Two barriers per batch: the one after
// the partial sums also keeps the next rows out of su until every wave has
// read it, and the one after su is written keeps the next partial sums out
// of sp until the current ones are added.
constexpr int kFinalRowsBig = 8;
__global__ __launch_bounds__(512) void final_rows_kernel(const float* __restrict__ h,
                                                         const float* __restrict__ mod, int mod_ld,
                                                         int scale_off, int chunk_len, float eps,
                                                         const float* __restrict__ w_out,
                                                         const float* __restrict__ b_out,
                                                         float* __restrict__ v, int rows, int W,
                                                         int A, int rows_per_block,
                                                         const int* __restrict__ period) {
  constexpr int R = kFinalRowsBig, KS = 16, NPL = 1024 / 64;
  __shared__ __attribute__((aligned(16))) float su[R][1024];  // zero past W
  __shared__ f32x4 sp[8][R][8];                                 // [wave][row][quad]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, tid = threadIdx.x;
  const int q = tid & 7, part = tid >> 3;
  const int qa = min(4 * q, A - 4);
  const int k0 = KS * part;
  f32x4 wr[KS];
#pragma unroll
  for (int j = 0; j < KS; ++j)
    wr[j] = k0 + j < W && 4 * q < A ? *reinterpret_cast<const f32x4*>(w_out + (size_t)(k0 + j) * A + qa)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
  const f32x4 bo = *reinterpret_cast<const f32x4*>(b_out + qa);
  const int per = film_period(period);
  const int rbeg = blockIdx.x * rows_per_block;
  const int rend = min(rows, rbeg + rows_per_block);
  float hv[NPL], sv[NPL], bv[NPL];
  auto load_row = [&](int row0) __attribute__((always_inline)) {  // this wave's row of a batch
    const int row = min(row0 + wave, rend - 1);
    const float* hr = h + (size_t)row * W;
    const float* sc = mod + (size_t)film_row(row / chunk_len, per) * mod_ld + scale_off;
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      const int cc = min(lane + 64 * i, W - 1);
      hv[i] = hr[cc];
      sv[i] = sc[cc];
      bv[i] = sc[W + cc];
    }
  };
  if (rbeg < rend) load_row(rbeg);
  for (int row0 = rbeg; row0 < rend; row0 += R) {
    {
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < NPL; ++i) ss += lane + 64 * i < W ? hv[i] * hv[i] : 0.f;
      ss = wave_sum(ss);
      const float rinv = 1.0f / sqrtf(ss / (float)W + eps);
#pragma unroll
      for (int i = 0; i < NPL; ++i) {
        const int cc = lane + 64 * i;
        su[wave][cc] = cc < W ? hv[i] * rinv * (1.0f + sv[i]) + bv[i] : 0.f;
      }
    }
    if (row0 + R < rend) load_row(row0 + R);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < KS; j += 4) {
        const f32x4 x4 = *reinterpret_cast<const f32x4*>(&su[r][k0 + j]);
        acc += x4[0] * wr[j];
        acc += x4[1] * wr[j + 1];
        acc += x4[2] * wr[j + 2];
        acc += x4[3] * wr[j + 3];
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = sum_lane_bits_543(acc[e]);
      if (lane < 8) sp[wave][r][lane] = acc;
    }
    __syncthreads();
    if (tid < R * 8) {
      const int r = tid >> 3;
      if (row0 + r < rend && 4 * q < A) {
        f32x4 vv = bo;
#pragma unroll
        for (int w = 0; w < 8; ++w) vv += sp[w][r][q];
        *reinterpret_cast<f32x4*>(v + (size_t)(row0 + r) * A + 4 * q) = vv;
      }
    }
  }
}

// ------------------------------------------- Euler + emit + shift + refill
// Thread (j, k) owns group j of 4 consecutive elements of the [C][A] chunk in
// slot k of stream b; all K slots of a group live in one block.  A block
// holds gpb = 256 / K consecutive groups; thread t takes slot t / gpb and
// group t % gpb, so neighbouring lanes touch neighbouring groups (whole
// 16-byte runs of a slot) and the fp64 refill of slot K-1 runs in one wave.
// Every thread loads its slot and applies x'_k = x_k - dt_k v_k (rounded
// product, rounded difference); after a barrier slot 0 writes the emitted
// chunk, slot k >= 1 writes buffer[k-1], and slot K-1 also writes fresh noise
// into buffer[K-1].  All loads precede the barrier and all stores follow it,
// so the in-place shift has no race.  The last block to finish advances the
// step counter.
__global__ __launch_bounds__(256) void euler_shift_kernel(float* __restrict__ buf,
                                                          const float* __restrict__ t,
                                                          const float* __restrict__ v,
                                                          float* __restrict__ out,
                                                          uint64_t* __restrict__ noise_state,
                                                          uint32_t* __restrict__ ticket,
                                                          int* __restrict__ n_valid, int B,
                                                          int K, int CA) {
  // The update must round the product and the difference separately.
#pragma clang fp contract(off)
  const int groups = (CA + 3) >> 2;
  const int gpb = 256 / K;                      // element groups per block
  const int k = threadIdx.x / gpb, jl = threadIdx.x % gpb;
  const int gid = blockIdx.x * gpb + jl;        // global group index over (b, j)
  const uint64_t seed = noise_state[0], step = noise_state[1];
  const bool active = k < K && gid < B * groups;
  float xn[4] = {0.f, 0.f, 0.f, 0.f};
  int b = 0, j = 0, e0 = 0, ne = 0;
  bool full = true;  // the popped slot holds a real chunk (not cold-start padding)
  if (active) {
    b = gid / groups;
    j = gid - b * groups;
    e0 = 4 * j;
    ne = min(4, CA - e0);
    full = n_valid[b] >= K;
    const float tk = t[(size_t)b * K + k];
    const float tp = k > 0 ? t[(size_t)b * K + k - 1] : 0.f;
    const float dt = tk - tp;
    const size_t base = ((size_t)b * K + k) * CA + e0;
    for (int i = 0; i < ne; ++i) {
      const float p = dt * v[base + i];
      xn[i] = buf[base + i] - p;
    }
  }
  __syncthreads();
  if (active) {
    const size_t base = ((size_t)b * K + k) * CA + e0;
    if (k == 0) {
      for (int i = 0; i < ne; ++i) out[(size_t)b * CA + e0 + i] = full ? xn[i] : 0.f;
    } else {
      for (int i = 0; i < ne; ++i) buf[base - CA + i] = xn[i];
    }
    if (k == K - 1) {
      uint32_t c[4] = {(uint32_t)j, (uint32_t)step, (uint32_t)(step >> 32), 0u};
      const uint64_t sb = seed + (uint64_t)b;
      philox4x32_10(c, (uint32_t)sb, (uint32_t)(sb >> 32));
      float z[4];
      box_muller(c[0], c[1], &z[0], &z[1]);
      box_muller(c[2], c[3], &z[2], &z[3]);
      for (int i = 0; i < ne; ++i) buf[base + i] = z[i];
    }
  }
  // step counter and valid-slot counts: advanced by the last block, once
  // every block has read them
  __shared__ int s_last;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t done =
        __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = done == gridDim.x - 1;
    if (s_last) {
      noise_state[1] = step + 1;
      __hip_atomic_store(ticket, 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (s_last)
    for (int bb = threadIdx.x; bb < B; bb += blockDim.x) n_valid[bb] = min(n_valid[bb] + 1, K);
}

// Cold start of streams [b0, b0 + nb): slots 0..K-2 become zero padding, slot
// K-1 a fresh Gaussian chunk drawn as euler_shift_kernel draws its tail (at
// the current step); then the step counter advances and those streams hold
// one valid slot.  One block.
__global__ __launch_bounds__(256) void cold_start_kernel(float* __restrict__ buf,
                                                         uint64_t* __restrict__ noise_state,
                                                         int* __restrict__ n_valid, int b0,
                                                         int nb, int K, int CA) {
  const uint64_t seed = noise_state[0], step = noise_state[1];
  const int groups = (CA + 3) >> 2;
  for (int idx = threadIdx.x; idx < nb * K * groups; idx += blockDim.x) {
    const int bl = idx / (K * groups), rem = idx - bl * (K * groups);
    const int k = rem / groups, j = rem - k * groups;
    const int b = b0 + bl, e0 = 4 * j, ne = min(4, CA - e0);
    float* dst = buf + ((size_t)b * K + k) * CA + e0;
    if (k < K - 1) {
      for (int i = 0; i < ne; ++i) dst[i] = 0.f;
    } else {
      uint32_t c[4] = {(uint32_t)j, (uint32_t)step, (uint32_t)(step >> 32), 0u};
      const uint64_t sb = seed + (uint64_t)b;
      philox4x32_10(c, (uint32_t)sb, (uint32_t)(sb >> 32));
      float z[4];
      box_muller(c[0], c[1], &z[0], &z[1]);
      box_muller(c[2], c[3], &z[2], &z[3]);
      for (int i = 0; i < ne; ++i) dst[i] = z[i];
    }
  }
  __syncthreads();  // every thread has read the step counter
  if (threadIdx.x == 0) noise_state[1] = step + 1;
  for (int bl = threadIdx.x; bl < nb; bl += blockDim.x) n_valid[b0 + bl] = 1;
}

// x <- x - (t_j - t_{j+1}) v   (sequential decode; product then difference rounded)
__global__ void seq_euler_kernel(float* __restrict__ x, const float* __restrict__ v,
                                 const float* __restrict__ tsched, int j, int n) {
#pragma clang fp contract(off)
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n) return;
  const float dt = tsched[j] - tsched[j + 1];
  const float p = dt * v[idx];
  x[idx] = x[idx] - p;
}

__global__ void copy_f32_kernel(float* __restrict__ d, const float* __restrict__ s, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) d[i] = s[i];
}

__global__ void fill_t_kernel(float* __restrict__ t, const float* __restrict__ tsched, int j,
                              int B) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < B) t[i] = tsched[j];
}

// ---------------------------------------------------------- prefix install
// k: [L][B][ld][Hkv][dh] -> karena [L][Bmax][Hkv][S][dh], rows p < len[b];
// v: same source layout -> vtarena [L][Bmax][Hkv][dh][S] through a 64x64 LDS
// transpose (p-major reads and d-major writes are both coalesced).
template <typename T>
__global__ __launch_bounds__(256) void prefix_copy_kernel(const T* __restrict__ k,
                                                          const T* __restrict__ v, int B,
                                                          int src_batch, int ld, int Hkv, int dh,
                                                          T* __restrict__ karena,
                                                          T* __restrict__ vtarena, int Bmax,
                                                          int S, const int* __restrict__ len) {
  __shared__ T tile[64][65];
  const int pt = blockIdx.x, dt = blockIdx.y;
  const int lbg = blockIdx.z;  // (l, b, g)
  const int g = lbg % Hkv, lb = lbg / Hkv, b = lb % B, l = lb / B;
  const int n = len[b];
  const int p0 = pt * 64, d0 = dt * 64;
  if (p0 >= n) return;
  // src_batch == 1: one observation shared by every stream
  const size_t src_base = (((size_t)l * src_batch + (src_batch == 1 ? 0 : b)) * ld) * Hkv * dh;
  const size_t kdst = (((size_t)l * Bmax + b) * Hkv + g) * (size_t)S * dh;
  const size_t vdst = (((size_t)l * Bmax + b) * Hkv + g) * (size_t)dh * S;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int pp = ty; pp < 64; pp += 4) {
    const int p = p0 + pp, d = d0 + tx;
    if (p < n && d < dh) {
      const size_t si = src_base + ((size_t)p * Hkv + g) * dh + d;
      karena[kdst + (size_t)p * dh + d] = k[si];
      tile[pp][tx] = v[si];
    }
  }
  __syncthreads();
  for (int dd = ty; dd < 64; dd += 4) {
    const int d = d0 + dd, p = p0 + tx;
    if (p < n && d < dh) vtarena[vdst + (size_t)d * S + p] = tile[tx][dd];
  }
}

}  // namespace

template <typename T>
void launch_time_embed(const float* t, T* e, int rows, int width, hipStream_t s, int* period,
                       int K) {
  const int n = rows * (width / 2);
  hipLaunchKernelGGL((time_embed_kernel<T>), dim3((n + 255) / 256), dim3(256), 0, s, t, e, rows,
                     width, period, K);
}

bool head_fusable(int rows, int W, int A) {
  return rows < kManyRows && W <= 1024 && W % 4 == 0 && A <= 32 && A % 4 == 0;
}

template <typename T>
void launch_embed_adarms(const float* x, const float* w_in, const float* b_in, float* h,
                         const float* mod, int mod_ld, int chunk_len, float eps, T* u, int rows,
                         int A, int W, hipStream_t s, float* xs, const int* period) {
  if (rows >= kManyRows && W <= 1024 && A <= 32) {
    // one round of one workgroup per CU
    const int rpb = kEmbRows * ((rows + kEmbRows * 256 - 1) / (kEmbRows * 256));
    hipLaunchKernelGGL((embed_adarms_rows_kernel<T>), dim3((rows + rpb - 1) / rpb), dim3(256), 0, s,
                       x, w_in, b_in, h, mod, mod_ld, chunk_len, eps, u, rows, A, W, rpb, period);
    return;
  }
  if (W <= 1024 && W % 4 == 0 && A <= 32) {
    hipLaunchKernelGGL((embed_adarms_small_kernel<T>), dim3((rows + kEmbSmallRows - 1) / kEmbSmallRows),
                       dim3(256), 0, s, x, w_in, b_in, h, mod, mod_ld, chunk_len, eps, u, rows, A, W,
                       xs, period);
    return;
  }
  const dim3 grid((rows + kEmbRows - 1) / kEmbRows);
  if (W <= 1024)
    hipLaunchKernelGGL((embed_adarms_kernel<T, 1>), grid, dim3(256), 0, s, x, w_in, b_in, h, mod,
                       mod_ld, chunk_len, eps, u, rows, A, W, period);
  else
    hipLaunchKernelGGL((embed_adarms_kernel<T, 2>), grid, dim3(256), 0, s, x, w_in, b_in, h, mod,
                       mod_ld, chunk_len, eps, u, rows, A, W, period);
}

template <typename T>
void launch_resid_norm(const void* part, bool bf16_parts, int ks, float* h, const float* mod,
                       int mod_ld, int gate_off, int norm_off, int chunk_len, float eps, T* u,
                       int rows, int W, const void* pf, size_t pf_bytes, hipStream_t s,
                       const int* period) {
  // split slots (power of two >= ks, at most 8) and column groups per thread
  const int ksm = ks <= 2 ? 2 : ks <= 4 ? 4 : 8;
  const int nq = W <= 1024 ? 1 : 2;
  auto go = [&](auto kern, const auto* pp) {
    hipLaunchKernelGGL(kern, dim3(rows), dim3(256), 0, s, pp, ks, h, mod, mod_ld, gate_off,
                       norm_off, chunk_len, eps, u, rows, W, pf, pf_bytes, period);
  };
#define FV_RN(P, KSM, NQ) go(resid_norm_kernel<T, P, KSM, NQ>, static_cast<const P*>(part))
#define FV_RN_Q(P, KSM) (nq == 1 ? FV_RN(P, KSM, 1) : FV_RN(P, KSM, 2))
#define FV_RN_K(P) (ksm == 2 ? FV_RN_Q(P, 2) : ksm == 4 ? FV_RN_Q(P, 4) : FV_RN_Q(P, 8))
  if (bf16_parts)
    FV_RN_K(bf16_t);
  else
    FV_RN_K(float);
#undef FV_RN_K
#undef FV_RN_Q
#undef FV_RN
}

template <typename T>
void launch_adarms(const float* h, const float* mod, int mod_ld, int scale_off, int chunk_len,
                   float eps, T* u, int rows, int W, hipStream_t s, const int* period) {
  hipLaunchKernelGGL((adarms_kernel<T>), dim3((rows + 3) / 4), dim3(256), 0, s, h, mod, mod_ld,
                     scale_off, chunk_len, eps, u, rows, W, period);
}

void launch_final(const float* h, const float* mod, int mod_ld, int scale_off, int chunk_len,
                  float eps, const float* w_out, const float* b_out, float* v, int rows, int W,
                  int A, hipStream_t s, const int* period) {
  const size_t lds = (size_t)(kFinalRows * W + 256 * kFinalRows) * sizeof(float);
  if (rows >= kManyRows && W <= 1024 && W % 4 == 0 && A <= 32 && A % 4 == 0) {
    // one round of one workgroup per CU
    const int rpb = kFinalRowsBig * ((rows + kFinalRowsBig * 256 - 1) / (kFinalRowsBig * 256));
    hipLaunchKernelGGL(final_rows_kernel, dim3((rows + rpb - 1) / rpb), dim3(512), 0, s, h, mod,
                       mod_ld, scale_off, chunk_len, eps, w_out, b_out, v, rows, W, A, rpb, period);
    return;
  }
  if (W <= 1024 && A <= 32 && A % 4 == 0) {
    hipLaunchKernelGGL(final_small_kernel<false>, dim3((rows + kFinalSmallRows - 1) / kFinalSmallRows),
                       dim3(256), 0, s, h, mod, mod_ld, scale_off, chunk_len, eps, w_out, b_out, v,
                       rows, W, A, EulerDest{}, period);
    return;
  }
  hipLaunchKernelGGL(final_kernel, dim3((rows + kFinalRows - 1) / kFinalRows), dim3(256), lds, s, h, mod, mod_ld,
                     scale_off, chunk_len, eps, w_out, b_out, v, rows, W, A, period);
}

void launch_final_euler(const float* h, const float* mod, int mod_ld, int scale_off, int chunk_len,
                        float eps, const float* w_out, const float* b_out, int rows, int W, int A,
                        const EulerDest& eu, hipStream_t s, const int* period) {
  hipLaunchKernelGGL(final_small_kernel<true>, dim3((rows + kFinalSmallRows - 1) / kFinalSmallRows),
                     dim3(256), 0, s, h, mod, mod_ld, scale_off, chunk_len, eps, w_out, b_out,
                     nullptr, rows, W, A, eu, period);
}

void launch_euler_shift(float* buffer, const float* t, const float* v, float* out,
                        const uint64_t* noise_state, uint32_t* ticket, int* n_valid, int B, int K,
                        int CA, hipStream_t s) {
  const int groups = (CA + 3) / 4;
  const int gpb = 256 / K;
  const int n = B * groups;
  hipLaunchKernelGGL(euler_shift_kernel, dim3((n + gpb - 1) / gpb), dim3(256), 0, s, buffer, t, v,
                     out, const_cast<uint64_t*>(noise_state), ticket, n_valid, B, K, CA);
}

void launch_cold_start(float* buffer, uint64_t* noise_state, int* n_valid, int b0, int nb, int K,
                       int CA, hipStream_t s) {
  hipLaunchKernelGGL(cold_start_kernel, dim3(1), dim3(256), 0, s, buffer, noise_state, n_valid, b0,
                     nb, K, CA);
}

void launch_seq_euler(float* x, const float* v, const float* tsched, int j, int n,
                      hipStream_t s) {
  hipLaunchKernelGGL(seq_euler_kernel, dim3((n + 255) / 256), dim3(256), 0, s, x, v, tsched, j,
                     n);
}

void launch_copy_f32(float* dst, const float* src, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(copy_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dst,
                     src, n);
}

void launch_fill_t(float* t, const float* tsched, int j, int B, hipStream_t s) {
  hipLaunchKernelGGL(fill_t_kernel, dim3((B + 255) / 256), dim3(256), 0, s, t, tsched, j, B);
}

template <typename T>
void launch_prefix_copy(const T* k, const T* v, int L, int B, int src_batch, int ld, int Hkv,
                        int dh, T* karena, T* vtarena, int Bmax, int S, const int* len,
                        hipStream_t s) {
  dim3 grid((ld + 63) / 64, (dh + 63) / 64, L * B * Hkv);
  hipLaunchKernelGGL((prefix_copy_kernel<T>), grid, dim3(256), 0, s, k, v, B, src_batch, ld, Hkv,
                     dh, karena, vtarena, Bmax, S, len);
}

template void launch_time_embed<bf16_t>(const float*, bf16_t*, int, int, hipStream_t, int*, int);
template void launch_time_embed<float>(const float*, float*, int, int, hipStream_t, int*, int);
template void launch_embed_adarms<bf16_t>(const float*, const float*, const float*, float*,
                                          const float*, int, int, float, bf16_t*, int, int, int,
                                          hipStream_t, float*, const int*);
template void launch_embed_adarms<float>(const float*, const float*, const float*, float*,
                                         const float*, int, int, float, float*, int, int, int,
                                         hipStream_t, float*, const int*);
template void launch_resid_norm<bf16_t>(const void*, bool, int, float*, const float*, int, int,
                                        int, int, float, bf16_t*, int, int, const void*, size_t,
                                        hipStream_t, const int*);
template void launch_resid_norm<float>(const void*, bool, int, float*, const float*, int, int,
                                       int, int, float, float*, int, int, const void*, size_t,
                                       hipStream_t, const int*);
template void launch_adarms<bf16_t>(const float*, const float*, int, int, int, float, bf16_t*,
                                    int, int, hipStream_t, const int*);
template void launch_adarms<float>(const float*, const float*, int, int, int, float, float*, int,
                                   int, hipStream_t, const int*);
template void launch_prefix_copy<bf16_t>(const bf16_t*, const bf16_t*, int, int, int, int, int,
                                         int, bf16_t*, bf16_t*, int, int, const int*, hipStream_t);
template void launch_prefix_copy<float>(const float*, const float*, int, int, int, int, int, int,
                                        float*, float*, int, int, const int*, hipStream_t);

}  // namespace fv
