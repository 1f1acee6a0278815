// Runtime behind the C ABI: validation, weight packing, device arenas,
// step orchestration and HIP-graph capture/replay.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <exception>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "fv_internal.h"

struct fv_handle_s : public fv::Handle {};

// Scratch of fv_decode_step_noalloc: the attention key-split partials and
// the split-K partial tiles of one step, in a fixed array that every GPU the
// library runs on holds until the process ends (each GPU its own copy, at
// its own address).  Host code never uses this name as an address: the
// per-device address comes from hipGetSymbolAddress (see static_scratch).
constexpr size_t kStaticScratchBytes = FV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace fv {
namespace {

struct FvError {
  fv_status st;
  std::string msg;
};

[[noreturn]] void fail(fv_status st, const std::string& m) { throw FvError{st, m}; }

#define FV_HIP(x)                                                                       \
  do {                                                                                  \
    hipError_t e_ = (x);                                                                \
    if (e_ != hipSuccess) fail(FV_ERR_HIP, std::string(#x) + ": " + hipGetErrorString(e_)); \
  } while (0)

// Restores the caller's current device on scope exit.
struct DeviceScope {
  int prev = -1;
  explicit DeviceScope(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) FV_HIP(hipSetDevice(dev));
  }
  ~DeviceScope() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

template <typename Fn>
fv_status guarded(Handle* h, Fn&& fn) {
  try {
    fn();
    if (h) h->last_error.clear();
    return FV_OK;
  } catch (const FvError& e) {
    if (h) h->last_error = e.msg;
    return e.st;
  } catch (const std::bad_alloc&) {
    if (h) h->last_error = "host allocation failed";
    return FV_ERR_OOM;
  } catch (const std::exception& e) {
    if (h) h->last_error = e.what();
    return FV_ERR_INTERNAL;
  } catch (...) {
    if (h) h->last_error = "unknown internal error";
    return FV_ERR_INTERNAL;
  }
}

uint16_t host_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

void* dalloc(Handle* h, size_t bytes) {
  void* p = nullptr;
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    fail(FV_ERR_OOM, "hipMalloc of " + std::to_string(bytes) + " bytes failed: " +
                         hipGetErrorString(e));
  }
  h->allocations.push_back(p);
  h->device_bytes += bytes;
  return p;
}

// Uploads host fp32 values as the handle's storage type (bf16 RNE or fp32).
void* upload_T(Handle* h, const std::vector<float>& v) {
  void* d = dalloc(h, v.size() * h->esz);
  if (h->bf16) {
    std::vector<uint16_t> b(v.size());
    for (size_t i = 0; i < v.size(); ++i) b[i] = host_bf16(v[i]);
    FV_HIP(hipMemcpy(d, b.data(), b.size() * 2, hipMemcpyHostToDevice));
  } else {
    FV_HIP(hipMemcpy(d, v.data(), v.size() * 4, hipMemcpyHostToDevice));
  }
  return d;
}

// fp32 upload; in bf16 mode values are first rounded to bf16 (stored as fp32).
float* upload_f32(Handle* h, const float* src, size_t n, bool round) {
  std::vector<float> v(src, src + n);
  if (round && h->bf16)
    for (float& x : v) {
      uint32_t u = (uint32_t)host_bf16(x) << 16;
      std::memcpy(&x, &u, 4);
    }
  float* d = static_cast<float*>(dalloc(h, n * 4));
  FV_HIP(hipMemcpy(d, v.data(), n * 4, hipMemcpyHostToDevice));
  return d;
}

void need(const void* p, const char* what) {
  if (!p) fail(FV_ERR_INVALID_ARG, std::string("NULL pointer: ") + what);
}

// Appends rows of Bt [out][in] for output columns [c0, c0+cnt) of W [in][out].
void append_out_major(std::vector<float>& dst, const float* W, int in, int out, int col) {
  for (int k = 0; k < in; ++k) dst.push_back(W[(size_t)k * out + col]);
}

void validate_cfg(const fv_cfg& c) {
  auto bad = [](const std::string& m) { fail(FV_ERR_INVALID_ARG, "invalid config: " + m); };
  if (c.n_layers < 1 || c.width < 1 || c.n_q_heads < 1 || c.n_kv_heads < 1 || c.head_dim < 1 ||
      c.mlp_dim < 1 || c.action_dim < 1 || c.chunk_len < 1 || c.n_chunks < 1 ||
      c.max_prefix < 0 || c.max_batch < 1)
    bad("sizes must be >= 1 (max_prefix >= 0)");
  if (c.dtype != FV_BF16 && c.dtype != FV_FP32) bad("dtype must be FV_BF16 or FV_FP32");
  if (c.mlp_gated != 0 && c.mlp_gated != 1) bad("mlp_gated must be 0 or 1");
  if (c.n_q_heads % c.n_kv_heads) bad("n_q_heads must be a multiple of n_kv_heads");
  if (c.width % 128) bad("width must be a multiple of 128");
  if (c.head_dim % 64 || c.head_dim > 256) bad("head_dim must be 64, 128, 192 or 256");
  if (c.mlp_dim % 64) bad("mlp_dim must be a multiple of 64");
  if (!c.mlp_gated && c.mlp_dim % 128) bad("mlp_dim must be a multiple of 128 for a plain MLP");
  if (((c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim) % 128)
    bad("(n_q_heads + 2 n_kv_heads) * head_dim must be a multiple of 128");
  if (c.action_dim > 64) bad("action_dim must be at most 64");
  if ((long)c.n_chunks * c.chunk_len > 4096) bad("n_chunks * chunk_len must be at most 4096");
  if (c.n_chunks > 256) bad("n_chunks must be at most 256");  // one queue-update block per group
  if ((long)c.max_prefix + (long)c.n_chunks * c.chunk_len > 32768)
    bad("max_prefix + n_chunks * chunk_len must be at most 32768");
  if (c.max_batch > 4096) bad("max_batch must be at most 4096");
  if (c.width > 2048) bad("width must be at most 2048");
  if ((long)c.max_batch * c.n_chunks * c.chunk_len > 262144)
    bad("max_batch * n_chunks * chunk_len must be at most 262144");
  if ((long)c.n_layers * c.max_batch * c.n_kv_heads > 65535)
    bad("n_layers * max_batch * n_kv_heads must be at most 65535");
  if (!(c.rms_eps >= 0.f) || !std::isfinite(c.rms_eps)) bad("rms_eps must be finite and >= 0");
  if (!(c.rope_theta > 0.f) || !std::isfinite(c.rope_theta)) bad("rope_theta must be > 0");
}

// Key splits per attention row tile: enough blocks for two per CU (about 512),
// at most 8 splits.
int attn_split(const Handle* h, int B) {
  const int tiles = h->bf16 ? attention_row_tiles<bf16_t>(h->T, h->Hq, h->Hkv)
                            : attention_row_tiles<float>(h->T, h->Hq, h->Hkv);
  const int base = tiles * B * h->Hkv;
  int s = (512 + base - 1) / base;
  return s < 1 ? 1 : (s > 8 ? 8 : s);
}

// ------------------------------------------------------------------ forward
// Output projection / down projection with the gated residual, fused with
// the FiLM RMSNorm that feeds the next GEMM (norm_off < 0: none).
// Kernels ahead of a GEMM pull its weights into the memory-side cache.

// per: the FiLM-row sharing flag the maps' readers take (film_row), or nullptr.
template <typename T>
void resid_block(Handle* h, const float* mod, const int* per, const T* A, const T* Bt, int K,
                 int gate_off, int norm_off, int rowsT, hipStream_t s,
                 const void* next_w = nullptr, size_t next_bytes = 0) {
  const int W = h->W;
  bool bf16_parts = false;
  const int ks = gemm_partials<T>(A, Bt, rowsT, W, K, h->gw, s, &bf16_parts);
  if (ks <= 1)
    gemm_gated_resid<T>(A, Bt, h->hres, mod, h->Nmod, gate_off, h->C, rowsT, W, K, h->gw, s, per);
  if (ks > 1) {
    launch_resid_norm<T>(h->gw.ws, bf16_parts, ks, h->hres, mod, h->Nmod, gate_off, norm_off,
                         h->C, h->cfg.rms_eps, (T*)h->u, rowsT, W,
                         next_w, next_bytes, s, per);
  } else {
    if (norm_off >= 0)
      launch_adarms<T>(h->hres, mod, h->Nmod, norm_off, h->C, h->cfg.rms_eps, (T*)h->u, rowsT,
                       W, s, per);
  }
}

// Time-MLP and FiLM-map GEMM of rows [r0, r0 + n) of the time embedding
// (skip: a flag that makes every launch return at once when set, or nullptr).
template <typename T>
void film_rows(Handle* h, int r0, int n, float* mod, hipStream_t s, const int* skip) {
  const int W = h->W;
  const size_t o = (size_t)r0 * W;
  gemm_bias_silu<T>((T*)h->e + o, (T*)h->w_t1, h->b_t1, (T*)h->hid + o, n, W, W, h->gw, s, skip);
  gemm_bias_silu<T>((T*)h->hid + o, (T*)h->w_t2, h->b_t2, (T*)h->cond + o, n, W, W, h->gw, s,
                    skip);
  gemm_bias_f32<T>((T*)h->cond + o, (T*)h->w_mod, h->b_mod, mod + (size_t)r0 * h->Nmod, n,
                   h->Nmod, W, h->gw, s, skip);
}

// FiLM maps of every norm for noise levels t [B*K]: timestep embedding,
// time-MLP, one GEMM for all (2L+1) [scale | shift | gate] maps -> mod.
// With a sharing flag and several streams, the K rows of stream 0 are
// computed and the rest only when some stream's noise levels differ from
// stream 0's (the time embedding sets the flag; otherwise those launches
// return at once, and the readers take stream 0's rows).  Returns the flag
// for the readers, or nullptr when every row was computed.
template <typename T>
const int* enqueue_film_maps(Handle* h, const float* t, int B, float* mod, hipStream_t s,
                             int* flag) {
  const int K = h->K, rowsK = B * K;
  if (B <= 1) flag = nullptr;
  launch_time_embed<T>(t, (T*)h->e, rowsK, h->W, s, flag, K);
  film_rows<T>(h, 0, flag ? K : rowsK, mod, s, nullptr);
  if (!flag) return nullptr;
  film_rows<T>(h, K, rowsK - K, mod, s, flag);
  return flag;
}

// pf: the weights the next kernels read, pulled into the memory-side cache by
// the attention (nullptr: none)
AttnArgs attn_args(const Handle* h, const void* kar, const void* var, int B, int n_split,
                   const void* pf = nullptr, size_t pf_bytes = 0) {
  return AttnArgs{h->q,  kar,      var,  h->d_len, h->o,          h->part_o,
                  h->part_ml, B,   h->T, h->C,     h->Hq,         h->Hkv,
                  h->dh, h->S,     n_split, h->d_valid, h->mask_mode, pf,
                  pf_bytes, h->d_len + h->Bmax};
}

// Velocity pass.  `mod_cached` (FiLM maps of a static schedule) replaces the
// time conditioning of t when given.  With `eu` (a decode step) and a head
// that takes it, the Euler update, emission, shift and refill run inside the
// velocity head (the embedding keeps a copy of the buffer in h->v, which the
// fused head reads instead of v); returns whether it did.
// `share_film`: streams whose noise levels equal stream 0's take stream 0's
// FiLM rows (enqueue_film_maps); off where every row of h->mod must be filled.
// The static-schedule maps were made the same way (their own flag).
template <typename T>
bool enqueue_forward(Handle* h, const float* buffer, const float* t, int B, float* v_out,
                     int n_layers_run, hipStream_t s, const float* mod_cached,
                     const EulerDest* eu, bool share_film) {
  const int W = h->W, rowsT = B * h->T;
  const int Nmod = h->Nmod;
  const size_t layer_elems = (size_t)h->Bmax * h->Hkv * h->S * h->dh;
  const bool fuse = eu && n_layers_run == h->L && head_fusable(rowsT, W, h->A);
  const float* mod = mod_cached;
  const int* per = mod_cached ? h->sched_per : nullptr;
  if (!mod) {
    per = enqueue_film_maps<T>(h, t, B, h->mod, s, share_film ? h->d_film_period : nullptr);
    mod = h->mod;
  }
  h->film_per = mod_cached ? nullptr : per;  // the flag that goes with h->mod (debug stages)
  launch_embed_adarms<T>(buffer, h->w_in, h->b_in, h->hres, mod, Nmod, h->C, h->cfg.rms_eps,
                         (T*)h->u, rowsT, h->A, W, s, fuse ? h->v : nullptr, per);
  const int n_split = attn_split(h, B);
  for (int l = 0; l < n_layers_run; ++l) {
    T* kar = (T*)h->karena + l * layer_elems;
    T* var = (T*)h->vtarena + l * layer_elems;
    const int n_attn = 2 * l, n_mlp = 2 * l + 1;
    QkvArgs<T> qa{(T*)h->q, kar, var, h->rcos, h->rsin, h->d_len, h->T, h->Hq, h->Hkv, h->dh,
                  h->S};
    gemm_qkv<T>((T*)h->u, (const T*)h->wqkv[l], qa, rowsT, h->Nqkv, W, h->gw, s);
    // each kernel ahead of a GEMM pulls that GEMM's weights into the
    // memory-side cache while it runs
    const AttnArgs aa = attn_args(h, kar, var, B, n_split, h->wo[l],
                                  (size_t)W * h->Hq * h->dh * h->esz);
    launch_attention<T>(aa, s);
    // (no prefetch of the gate/up weights here: the reduction would wait
    // for 16.8 MB of loads, batch-1 step 1433 -> 1415 us without it)
    resid_block<T>(h, mod, per, (const T*)h->o, (const T*)h->wo[l], h->Hq * h->dh,
                   n_attn * 3 * W + 2 * W, n_mlp * 3 * W, rowsT, s);
    if (h->cfg.mlp_gated)
      gemm_geglu<T>((T*)h->u, (const T*)h->wgu[l], (T*)h->m, rowsT, h->Ngu, W, h->gw, s);
    else
      gemm_gelu<T>((T*)h->u, (const T*)h->wgu[l], (T*)h->m, rowsT, h->Ngu, W, h->gw, s);
    const int next_norm = l + 1 < h->L ? 2 * (l + 1) * 3 * W : -1;
    resid_block<T>(h, mod, per, (const T*)h->m, (const T*)h->wd[l], h->F,
                   n_mlp * 3 * W + 2 * W, next_norm, rowsT, s,
                   l + 1 < h->L ? h->wqkv[l + 1] : nullptr, (size_t)h->Nqkv * W * h->esz);
  }
  if (fuse) {
    EulerDest d = *eu;
    d.xs = h->v;
    launch_final_euler(h->hres, mod, Nmod, 6 * h->L * W, h->C, h->cfg.rms_eps, h->w_out,
                       h->b_out, rowsT, W, h->A, d, s, per);
    return true;
  }
  if (v_out)
    launch_final(h->hres, mod, Nmod, 6 * h->L * W, h->C, h->cfg.rms_eps, h->w_out, h->b_out,
                 v_out, rowsT, W, h->A, s, per);
  return false;
}

// One projection GEMM with the gated residual, alone: the split-K partials
// (when k is split) or the GEMM with the residual in its epilogue.
template <typename T>
void proj_gemm_only(Handle* h, const T* A, const T* Bt, int K, int gate_off, int rowsT,
                    hipStream_t s) {
  bool bf16_parts = false;
  if (gemm_partials<T>(A, Bt, rowsT, h->W, K, h->gw, s, &bf16_parts) <= 1)
    gemm_gated_resid<T>(A, Bt, h->hres, h->mod, h->Nmod, gate_off, h->C, rowsT, h->W, K, h->gw,
                        s, h->film_per);
}

// The FiLM norm that follows a projection, alone: the split-K reduction with
// the gated residual and the norm (when k is split), or the plain norm.
// As in a step, the reduction pulls the next GEMM's weights [pf, pf + bytes)
// into the memory-side cache meanwhile.
template <typename T>
void proj_norm_only(Handle* h, int K, int gate_off, int norm_off, int rowsT, hipStream_t s,
                    const void* pf, size_t pf_bytes) {
  const GemmPlan p = plan_gemm(rowsT, h->W, K, h->bf16, true);
  if (p.ks > 1)
    launch_resid_norm<T>(h->gw.ws, gemm_partials_bf16(p, h->bf16), p.ks, h->hres, h->mod, h->Nmod,
                         gate_off, norm_off, h->C, h->cfg.rms_eps, (T*)h->u, rowsT, h->W,
                         pf, pf_bytes, s, h->film_per);
  else if (norm_off >= 0)
    launch_adarms<T>(h->hres, h->mod, h->Nmod, norm_off, h->C, h->cfg.rms_eps, (T*)h->u, rowsT,
                     h->W, s, h->film_per);
}

template <typename T>
void run_stage(Handle* h, int stage, int l, hipStream_t s) {
  const int B = h->batch, W = h->W, rowsK = B * h->K, rowsT = B * h->T;
  const size_t layer_elems = (size_t)h->Bmax * h->Hkv * h->S * h->dh;
  T* kar = (T*)h->karena + l * layer_elems;
  T* var = (T*)h->vtarena + l * layer_elems;
  const int n_attn = 2 * l, n_mlp = 2 * l + 1;
  switch (stage) {
    case 8:
      proj_gemm_only<T>(h, (const T*)h->o, (const T*)h->wo[l], h->Hq * h->dh,
                        n_attn * 3 * W + 2 * W, rowsT, s);
      return;
    case 9:
      proj_gemm_only<T>(h, (const T*)h->m, (const T*)h->wd[l], h->F, n_mlp * 3 * W + 2 * W,
                        rowsT, s);
      return;
    case 10:
      proj_norm_only<T>(h, h->Hq * h->dh, n_attn * 3 * W + 2 * W, n_mlp * 3 * W, rowsT, s,
                        nullptr, 0);
      return;
    case 11:
      proj_norm_only<T>(h, h->F, n_mlp * 3 * W + 2 * W,
                        l + 1 < h->L ? 2 * (l + 1) * 3 * W : -1, rowsT, s,
                        l + 1 < h->L ? h->wqkv[l + 1] : nullptr, (size_t)h->Nqkv * W * h->esz);
      return;
    default:
      break;
  }
  switch (stage) {
    case 0:  // the FiLM-map GEMM as the last velocity pass ran it
      if (h->film_per) {
        gemm_bias_f32<T>((T*)h->cond, (T*)h->w_mod, h->b_mod, h->mod, h->K, h->Nmod, W, h->gw, s);
        const size_t o = (size_t)h->K * W;
        gemm_bias_f32<T>((T*)h->cond + o, (T*)h->w_mod, h->b_mod, h->mod + (size_t)h->K * h->Nmod,
                         rowsK - h->K, h->Nmod, W, h->gw, s, h->film_per);
      } else {
        gemm_bias_f32<T>((T*)h->cond, (T*)h->w_mod, h->b_mod, h->mod, rowsK, h->Nmod, W, h->gw, s);
      }
      break;
    case 1: {
      QkvArgs<T> qa{(T*)h->q, kar, var, h->rcos, h->rsin, h->d_len, h->T, h->Hq, h->Hkv,
                    h->dh, h->S};
      gemm_qkv<T>((T*)h->u, (const T*)h->wqkv[l], qa, rowsT, h->Nqkv, W, h->gw, s);
      break;
    }
    case 2:
    case 4:
    case 5: {
      launch_attention<T>(attn_args(h, kar, var, B, attn_split(h, B), h->wo[l],
                                    (size_t)W * h->Hq * h->dh * h->esz),
                          s, stage == 2 ? 3 : stage == 4 ? 1 : 2);
      break;
    }
    case 6: {
      resid_block<T>(h, h->mod, h->film_per, (const T*)h->o, (const T*)h->wo[l], h->Hq * h->dh,
                     n_attn * 3 * W + 2 * W, n_mlp * 3 * W, rowsT, s);
      break;
    }
    case 7: {
      const int next_norm = l + 1 < h->L ? 2 * (l + 1) * 3 * W : -1;
      resid_block<T>(h, h->mod, h->film_per, (const T*)h->m, (const T*)h->wd[l], h->F,
                     n_mlp * 3 * W + 2 * W, next_norm, rowsT, s);
      break;
    }
    default:
      if (h->cfg.mlp_gated)
        gemm_geglu<T>((T*)h->u, (const T*)h->wgu[l], (T*)h->m, rowsT, h->Ngu, W, h->gw, s);
      else
        gemm_gelu<T>((T*)h->u, (const T*)h->wgu[l], (T*)h->m, rowsT, h->Ngu, W, h->gw, s);
  }
}

bool forward(Handle* h, const float* buffer, const float* t, int B, float* v_out, int n_layers,
             hipStream_t s, const float* mod_cached = nullptr, const EulerDest* eu = nullptr,
             bool share_film = true) {
  if (h->bf16)
    return enqueue_forward<bf16_t>(h, buffer, t, B, v_out, n_layers, s, mod_cached, eu,
                                   share_film);
  return enqueue_forward<float>(h, buffer, t, B, v_out, n_layers, s, mod_cached, eu, share_film);
}

// One decode step (Algorithm 1): the velocity pass, then the Euler update,
// emission, shift and refill, fused into the velocity head where it can be.
void decode(Handle* h, float* buffer, const float* t, int B, float* out_chunk, hipStream_t s,
            const float* mod_cached) {
  const EulerDest eu{buffer, nullptr, t, out_chunk, h->d_noise, h->d_ticket, h->d_valid, h->K};
  if (!forward(h, buffer, t, B, h->v, h->L, s, mod_cached, &eu))
    launch_euler_shift(buffer, t, h->v, out_chunk, h->d_noise, h->d_ticket, h->d_valid, B, h->K,
                       h->C * h->A, s);
}

// FiLM maps of a static schedule, rows shared across streams as in a step
// (flag: the schedule's own sharing flag); returns the flag its readers take.
const int* film_maps(Handle* h, const float* t, int B, float* mod, hipStream_t s, int* flag) {
  if (h->bf16) return enqueue_film_maps<bf16_t>(h, t, B, mod, s, flag);
  return enqueue_film_maps<float>(h, t, B, mod, s, flag);
}

void check_launch() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) fail(FV_ERR_HIP, std::string("kernel launch failed: ") + hipGetErrorString(e));
}

// Runs `enq` directly, or through a cached HIP graph keyed by (kind, batch,
// pointers, n).  Capture happens on the handle's own stream; the instantiated
// graph is launched on the caller's stream.
template <typename Enq>
void run_step(Handle* h, int kind, const void* p0, const void* p1, const void* p2,
              const void* p3, int n, hipStream_t stream, Enq&& enq) {
  (void)hipGetLastError();
  if (!h->use_graphs) {
    enq(stream);
    check_launch();
    return;
  }
  GraphEntry* ent = nullptr;
  for (GraphEntry& g : h->graphs)
    if (g.kind == kind && g.batch == h->batch && g.n == n && g.slot == h->cur_slot &&
        g.p[0] == p0 && g.p[1] == p1 && g.p[2] == p2 && g.p[3] == p3)
      ent = &g;
  if (!ent) {
    if (h->graphs.size() >= 8) {
      size_t lru = 0;
      for (size_t i = 1; i < h->graphs.size(); ++i)
        if (h->graphs[i].last_use < h->graphs[lru].last_use) lru = i;
      (void)hipGraphExecDestroy(h->graphs[lru].exec);
      h->graphs.erase(h->graphs.begin() + lru);
    }
    FV_HIP(hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal));
    hipGraph_t graph = nullptr;
    try {
      enq(h->cap_stream);
    } catch (...) {
      (void)hipStreamEndCapture(h->cap_stream, &graph);
      if (graph) (void)hipGraphDestroy(graph);
      throw;
    }
    hipError_t le = hipGetLastError();
    hipError_t ee = hipStreamEndCapture(h->cap_stream, &graph);
    if (le != hipSuccess || ee != hipSuccess) {
      if (graph) (void)hipGraphDestroy(graph);
      fail(FV_ERR_HIP, std::string("graph capture failed: ") +
                           hipGetErrorString(le != hipSuccess ? le : ee));
    }
    hipGraphExec_t exec = nullptr;
    hipError_t ie = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ie != hipSuccess) fail(FV_ERR_HIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(ie));
    GraphEntry g;
    g.kind = kind;
    g.batch = h->batch;
    g.n = n;
    g.slot = h->cur_slot;
    g.p[0] = p0; g.p[1] = p1; g.p[2] = p2; g.p[3] = p3;
    g.exec = exec;
    h->graphs.push_back(g);
    ent = &h->graphs.back();
  }
  ent->last_use = ++h->use_clock;
  FV_HIP(hipGraphLaunch(ent->exec, stream));
}

void check_ptr(const void* p, const char* what) {
  need(p, what);
  if (reinterpret_cast<uintptr_t>(p) % 16)
    fail(FV_ERR_INVALID_ARG, std::string(what) + " must be 16-byte aligned");
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  return x < y + nb && y < x + na;
}

// Device address of `scratch` per device ordinal, looked up once per device
// (with that device current) when the first handle on it is created.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
hipError_t g_scratch_err[kMaxDevices] = {};
bool g_scratch_done[kMaxDevices] = {};

void lookup_static_scratch(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_done[dev]) return;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  g_scratch_err[dev] = e;
  g_scratch_ptr[dev] = e == hipSuccess ? p : nullptr;
  if (e != hipSuccess) (void)hipGetLastError();
  g_scratch_done[dev] = true;
}

void* static_scratch(int dev) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (dev < 0 || dev >= kMaxDevices || !g_scratch_done[dev] || !g_scratch_ptr[dev])
    fail(FV_ERR_HIP, std::string("no static scratch address on this device: ") +
                         (dev >= 0 && dev < kMaxDevices && g_scratch_done[dev]
                              ? hipGetErrorString(g_scratch_err[dev])
                              : "device not set up"));
  return g_scratch_ptr[dev];
}

size_t round256(size_t n) { return (n + 255) & ~size_t(255); }

// Scratch one step at `batch` streams needs: attention split partials
// (element type) and their (max, sum) pairs, and the largest split-K
// workspace of the step's GEMMs.
struct StepScratch {
  size_t part_o = 0, part_ml = 0, ws = 0;
  size_t total() const { return part_o + part_ml + ws; }
};
StepScratch step_scratch(const Handle* h, int B) {
  StepScratch r;
  const int s = attn_split(h, B);
  if (s > 1) {
    const size_t rows = (size_t)s * B * h->T * h->Hq;
    r.part_o = round256(rows * h->dh * h->esz);
    r.part_ml = round256(rows * 2 * 4);
  }
  const int W = h->W, rk = B * h->K, rt = B * h->T, qd = h->Hq * h->dh;
  const GemmPlan ps[] = {plan_gemm(rk, W, W, h->bf16), plan_gemm(rk, h->Nmod, W, h->bf16),
                         plan_gemm(rt, h->Nqkv, W, h->bf16), plan_gemm(rt, W, qd, h->bf16, true),
                         plan_gemm(rt, h->Ngu, W, h->bf16), plan_gemm(rt, W, h->F, h->bf16, true)};
  for (const GemmPlan& p : ps) r.ws = std::max(r.ws, round256(p.ws_floats * 4));
  return r;
}

// Points the handle's split partials and split-K workspace at caller-given
// memory for the duration of an eager (uncaptured) pass, then restores them.
struct ScratchSwap {
  Handle* h;
  float* ws;
  void* part_o;
  float* part_ml;
  ScratchSwap(Handle* hh, unsigned char* base, const StepScratch& sz)
      : h(hh), ws(hh->gw.ws), part_o(hh->part_o), part_ml(hh->part_ml) {
    h->part_o = base;
    h->part_ml = reinterpret_cast<float*>(base + sz.part_o);
    h->gw.ws = reinterpret_cast<float*>(base + sz.part_o + sz.part_ml);
  }
  ~ScratchSwap() {
    h->gw.ws = ws;
    h->part_o = part_o;
    h->part_ml = part_ml;
  }
};

void need_prefix(const Handle* h) {
  if (!h->prefix_set && h->staged_slot < 0)
    fail(FV_ERR_STATE, "no observation prefix: call fv_set_prefix first");
}

enum Kind { KIND_STEP = 1, KIND_VELOCITY = 2, KIND_SEQ = 3, KIND_STEP_CACHED = 4,
            KIND_VELOCITY_CACHED = 5, KIND_STAGE = 6 };

// Batch of the next pass: a staged observation's once the pass switches to it.
int pending_batch(const Handle* h) { return h->staged_slot >= 0 ? h->staged_batch : h->batch; }

// The noise levels a pass over `batch` streams uses: the caller's t, or the
// installed schedule.  Checked before anything changes.
const float* schedule_or(const Handle* h, const float* t, int batch) {
  if (t) return t;
  if (h->sched_batch != batch)
    fail(FV_ERR_STATE, "t is NULL but no schedule is installed for the active batch "
                       "(call fv_set_schedule)");
  return h->t_cache;
}

// Drops the captured graphs (their kernel arguments are out of date).
void clear_graphs(Handle* h) {
  if (h->graphs.empty()) return;
  (void)hipDeviceSynchronize();
  for (GraphEntry& g : h->graphs)
    if (g.exec) (void)hipGraphExecDestroy(g.exec);
  h->graphs.clear();
}

void destroy_handle(Handle* h) {
  if (h->allocations.empty() && !h->cap_stream && h->graphs.empty()) return;
  (void)hipDeviceSynchronize();
  for (GraphEntry& g : h->graphs)
    if (g.exec) (void)hipGraphExecDestroy(g.exec);
  h->graphs.clear();
  for (void* p : h->allocations) (void)hipFree(p);
  h->allocations.clear();
  for (int i = 0; i < 2; ++i) {
    if (h->pinned_len[i]) (void)hipHostFree(h->pinned_len[i]);
    if (h->ev_ready[i]) (void)hipEventDestroy(h->ev_ready[i]);
    if (h->ev_done[i]) (void)hipEventDestroy(h->ev_done[i]);
    if (h->ev_len[i]) (void)hipEventDestroy(h->ev_len[i]);
    h->pinned_len[i] = nullptr;
    h->ev_ready[i] = h->ev_done[i] = h->ev_len[i] = nullptr;
  }
  if (h->cap_stream) (void)hipStreamDestroy(h->cap_stream);
  h->cap_stream = nullptr;
}

// A pass about to read the prefix on `stream`: switch to a staged
// observation (the stream waits for its copy) ...
void activate_staged(Handle* h, hipStream_t stream) {
  if (h->staged_slot < 0) return;
  const int sl = h->staged_slot;
  FV_HIP(hipStreamWaitEvent(stream, h->ev_ready[sl], 0));
  h->cur_slot = sl;
  h->karena = h->arena_k[sl];
  h->vtarena = h->arena_v[sl];
  h->d_len = h->len_slot[sl];
  h->len_host = h->len_host_slot[sl];
  h->batch = h->staged_batch;
  h->staged_slot = -1;
  h->prefix_set = true;
}

// ... and after it: the slot is free for restaging once `stream` passes here.
void mark_used(Handle* h, hipStream_t stream) {
  if (!h->async_ready) return;
  FV_HIP(hipEventRecord(h->ev_done[h->cur_slot], stream));
  h->done_recorded[h->cur_slot] = true;
}

}  // namespace
}  // namespace fv

using namespace fv;

extern "C" {

int32_t fv_abi_version(void) { return FV_ABI_VERSION; }

const char* fv_status_string(fv_status s) {
  switch (s) {
    case FV_OK: return "ok";
    case FV_ERR_INVALID_ARG: return "invalid argument";
    case FV_ERR_STATE: return "invalid state";
    case FV_ERR_OOM: return "out of device memory";
    case FV_ERR_HIP: return "HIP runtime error";
    case FV_ERR_INTERNAL: return "internal error";
  }
  return "unknown status";
}

const char* fv_last_error(fv_handle h) { return h ? h->last_error.c_str() : ""; }

fv_status fv_create(const fv_weights* w, const fv_cfg* cfg, fv_handle* out) {
  if (!out) return FV_ERR_INVALID_ARG;
  *out = nullptr;
  if (!w || !cfg) return FV_ERR_INVALID_ARG;
  fv_handle_s* h = nullptr;
  try {
    h = new fv_handle_s();
  } catch (...) {
    return FV_ERR_OOM;
  }
  fv_status st = guarded(h, [&] {
    validate_cfg(*cfg);
    Handle& H = *h;
    H.cfg = *cfg;
    H.bf16 = cfg->dtype == FV_BF16;
    H.esz = H.bf16 ? 2 : 4;
    H.L = cfg->n_layers; H.W = cfg->width; H.Hq = cfg->n_q_heads; H.Hkv = cfg->n_kv_heads;
    H.dh = cfg->head_dim; H.F = cfg->mlp_dim; H.A = cfg->action_dim; H.C = cfg->chunk_len;
    H.K = cfg->n_chunks; H.T = H.K * H.C; H.Pmax = cfg->max_prefix; H.Bmax = cfg->max_batch;
    H.S = ((buffer_row0(H.Pmax) + H.T + 63) / 64) * 64;
    H.Nqkv = (H.Hq + 2 * H.Hkv) * H.dh;
    H.Nmod = (6 * H.L + 2) * H.W;
    H.Ngu = cfg->mlp_gated ? 2 * H.F : H.F;
    const int W = H.W, L = H.L, F = H.F, dh = H.dh;

    need(w->w_in, "w_in"); need(w->b_in, "b_in"); need(w->w_t1, "w_t1"); need(w->b_t1, "b_t1");
    need(w->w_t2, "w_t2"); need(w->b_t2, "b_t2"); need(w->w_out, "w_out"); need(w->b_out, "b_out");
    need(w->w_mod, "w_mod"); need(w->b_mod, "b_mod"); need(w->wq, "wq"); need(w->wk, "wk");
    need(w->wv, "wv"); need(w->wo, "wo"); need(w->wu, "wu"); need(w->wd, "wd");
    if (cfg->mlp_gated) need(w->wg, "wg");
    for (int n = 0; n <= 2 * L; ++n) { need(w->w_mod[n], "w_mod[n]"); need(w->b_mod[n], "b_mod[n]"); }
    for (int l = 0; l < L; ++l) {
      need(w->wq[l], "wq[l]"); need(w->wk[l], "wk[l]"); need(w->wv[l], "wv[l]");
      need(w->wo[l], "wo[l]"); need(w->wu[l], "wu[l]"); need(w->wd[l], "wd[l]");
      if (cfg->mlp_gated) need(w->wg[l], "wg[l]");
    }

    FV_HIP(hipGetDevice(&H.device));
    lookup_static_scratch(H.device);
    if (H.bf16) {
      FV_HIP(gemm_prepare());
      FV_HIP(attention_prepare());
    }
    FV_HIP(hipStreamCreateWithFlags(&H.cap_stream, hipStreamNonBlocking));

    // ---- weights
    H.w_in = upload_f32(h, w->w_in, (size_t)H.A * W, true);
    H.b_in = upload_f32(h, w->b_in, W, true);
    H.b_t1 = upload_f32(h, w->b_t1, W, true);
    H.b_t2 = upload_f32(h, w->b_t2, W, true);
    H.w_out = upload_f32(h, w->w_out, (size_t)W * H.A, true);
    H.b_out = upload_f32(h, w->b_out, H.A, true);
    {
      std::vector<float> v;
      v.reserve((size_t)W * W);
      for (int c = 0; c < W; ++c) append_out_major(v, w->w_t1, W, W, c);
      H.w_t1 = upload_T(h, v);
      v.clear();
      for (int c = 0; c < W; ++c) append_out_major(v, w->w_t2, W, W, c);
      H.w_t2 = upload_T(h, v);
    }
    {
      std::vector<float> v, bias;
      v.reserve((size_t)H.Nmod * W);
      for (int n = 0; n <= 2 * L; ++n) {
        const int cols = n < 2 * L ? 3 * W : 2 * W;  // the final norm's gate is never used
        for (int c = 0; c < cols; ++c) {
          append_out_major(v, w->w_mod[n], W, 3 * W, c);
          bias.push_back(w->b_mod[n][c]);
        }
      }
      H.w_mod = upload_T(h, v);
      H.b_mod = upload_f32(h, bias.data(), bias.size(), true);
    }
    const int qd = H.Hq * dh, kd = H.Hkv * dh;
    for (int l = 0; l < L; ++l) {
      std::vector<float> v;
      v.reserve((size_t)H.Nqkv * W);
      // queries and keys: per head, rotary partners (d, d + dh/2) packed into
      // columns 64p + i and 64p + 32 + i, d = 32p + i
      auto rot_head = [&](const float* Wm, int out, int head) {
        for (int pc = 0; pc < dh; ++pc) {
          const int p = pc >> 6, i = pc & 63;
          const int d = i < 32 ? 32 * p + i : dh / 2 + 32 * p + (i - 32);
          append_out_major(v, Wm, W, out, head * dh + d);
        }
      };
      for (int hq = 0; hq < H.Hq; ++hq) rot_head(w->wq[l], qd, hq);
      for (int g = 0; g < H.Hkv; ++g) rot_head(w->wk[l], kd, g);
      for (int c = 0; c < kd; ++c) append_out_major(v, w->wv[l], W, kd, c);
      H.wqkv.push_back(upload_T(h, v));
      v.clear();
      for (int c = 0; c < W; ++c) append_out_major(v, w->wo[l], qd, W, c);
      H.wo.push_back(upload_T(h, v));
      v.clear();
      if (cfg->mlp_gated) {
        // gate/up partners packed into columns 64p + i and 64p + 32 + i, f = 32p + i
        for (int pc = 0; pc < 2 * F; ++pc) {
          const int p = pc >> 6, i = pc & 63;
          if (i < 32) append_out_major(v, w->wg[l], W, F, 32 * p + i);
          else append_out_major(v, w->wu[l], W, F, 32 * p + i - 32);
        }
      } else {
        for (int c = 0; c < F; ++c) append_out_major(v, w->wu[l], W, F, c);
      }
      H.wgu.push_back(upload_T(h, v));
      v.clear();
      for (int c = 0; c < W; ++c) append_out_major(v, w->wd[l], F, W, c);
      H.wd.push_back(upload_T(h, v));
    }

    // ---- rotary tables, built in fp64 and rounded to fp32
    {
      const int half = dh / 2;
      std::vector<float> cs((size_t)H.S * half), sn((size_t)H.S * half);
      for (int pos = 0; pos < H.S; ++pos)
        for (int i = 0; i < half; ++i) {
          const double inv = std::pow((double)cfg->rope_theta, -(double)i * 2.0 / (double)dh);
          const double ang = (double)pos * inv;
          cs[(size_t)pos * half + i] = (float)std::cos(ang);
          sn[(size_t)pos * half + i] = (float)std::sin(ang);
        }
      H.rcos = upload_f32(h, cs.data(), cs.size(), false);
      H.rsin = upload_f32(h, sn.data(), sn.size(), false);
    }

    // ---- arenas and scratch
    const size_t arena = (size_t)L * H.Bmax * H.Hkv * H.S * dh * H.esz;
    H.karena = dalloc(h, arena);
    H.vtarena = dalloc(h, arena);
    FV_HIP(hipMemset(H.karena, 0, arena));
    FV_HIP(hipMemset(H.vtarena, 0, arena));
    // [len | die_order]: Bmax lengths, then the Bmax*Hkv (stream, kv head) order
    H.d_len = static_cast<int*>(dalloc(h, (size_t)H.Bmax * (1 + H.Hkv) * 4));
    FV_HIP(hipMemset(H.d_len, 0, (size_t)H.Bmax * (1 + H.Hkv) * 4));
    H.arena_k[0] = H.karena;
    H.arena_v[0] = H.vtarena;
    H.len_slot[0] = H.d_len;
    {
      const std::vector<int> full(H.Bmax, H.K);  // every stream starts in steady state
      H.d_valid = static_cast<int*>(dalloc(h, (size_t)H.Bmax * 4));
      FV_HIP(hipMemcpy(H.d_valid, full.data(), (size_t)H.Bmax * 4, hipMemcpyHostToDevice));
    }
    const size_t rowsK = (size_t)H.Bmax * H.K, rowsT = (size_t)H.Bmax * H.T;
    H.e = dalloc(h, rowsK * W * H.esz);
    H.hid = dalloc(h, rowsK * W * H.esz);
    H.cond = dalloc(h, rowsK * W * H.esz);
    H.mod = static_cast<float*>(dalloc(h, rowsK * H.Nmod * 4));
    H.hres = static_cast<float*>(dalloc(h, rowsT * W * 4));
    H.u = dalloc(h, rowsT * W * H.esz);
    H.q = dalloc(h, rowsT * qd * H.esz);
    H.o = dalloc(h, rowsT * qd * H.esz);
    H.m = dalloc(h, rowsT * F * H.esz);
    H.v = static_cast<float*>(dalloc(h, rowsT * H.A * 4));
    size_t part_rows = 0;
    for (int B = 1; B <= H.Bmax; ++B) {
      const int s = attn_split(h, B);
      if (s > 1) part_rows = std::max(part_rows, (size_t)s * B * H.T * H.Hq);
    }
    H.part_o = dalloc(h, part_rows * dh * H.esz);
    H.part_ml = static_cast<float*>(dalloc(h, part_rows * 2 * 4));
    {
      size_t ws = 0;
      const bool b16 = H.bf16;
      for (int B = 1; B <= H.Bmax; ++B) {
        const int rk = B * H.K, rt = B * H.T;
        const GemmPlan ps[] = {plan_gemm(rk, W, W, b16), plan_gemm(rk, H.Nmod, W, b16),
                               plan_gemm(rt, H.Nqkv, W, b16), plan_gemm(rt, W, qd, b16, true),
                               plan_gemm(rt, H.Ngu, W, b16), plan_gemm(rt, W, F, b16, true)};
        for (const GemmPlan& p : ps) ws = std::max(ws, p.ws_floats);
      }
      H.gw.ws = static_cast<float*>(dalloc(h, ws * 4));
    }
    H.seq_x = static_cast<float*>(dalloc(h, (size_t)H.Bmax * H.T * H.A * 4));
    H.seq_t = static_cast<float*>(dalloc(h, (size_t)H.Bmax * 4));
    H.d_noise = static_cast<uint64_t*>(dalloc(h, 16));
    H.d_ticket = static_cast<uint32_t*>(dalloc(h, 4));
    H.d_film_period = static_cast<int*>(dalloc(h, 4));
    const uint64_t ns[2] = {cfg->noise_seed, 0};
    FV_HIP(hipMemcpy(H.d_noise, ns, 16, hipMemcpyHostToDevice));
    FV_HIP(hipMemset(H.d_ticket, 0, 4));
    FV_HIP(hipMemset(H.d_film_period, 0, 4));
    FV_HIP(hipDeviceSynchronize());
  });
  if (st != FV_OK) {
    destroy_handle(h);
    delete h;
    return st;
  }
  *out = h;
  return FV_OK;
}

fv_status fv_set_prefix(fv_handle h, const void* k, const void* v, const int32_t* len_host,
                        int32_t batch, int32_t ld, void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need(k, "k");
    need(v, "v");
    need(len_host, "len_host");
    if (batch < 1 || batch > h->Bmax)
      fail(FV_ERR_INVALID_ARG, "batch must be in [1, max_batch=" + std::to_string(h->Bmax) + "]");
    int maxlen = 0;
    for (int b = 0; b < batch; ++b) {
      if (len_host[b] < 0 || len_host[b] > h->Pmax)
        fail(FV_ERR_INVALID_ARG, "len[" + std::to_string(b) + "]=" + std::to_string(len_host[b]) +
                                     " outside [0, max_prefix=" + std::to_string(h->Pmax) + "]");
      maxlen = std::max(maxlen, (int)len_host[b]);
    }
    if (ld < maxlen || ld < 0) fail(FV_ERR_INVALID_ARG, "ld must be >= max(len)");
    DeviceScope ds(h->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    h->staged_slot = -1;  // a pending asynchronous observation is superseded
    h->len_host.assign(len_host, len_host + batch);
    h->order_host.resize((size_t)batch * h->Hkv);
    die_order(h->len_host.data(), batch, h->Hkv, h->order_host.data());
    FV_HIP(hipMemcpyAsync(h->d_len, h->len_host.data(), (size_t)batch * 4, hipMemcpyHostToDevice, s));
    FV_HIP(hipMemcpyAsync(h->d_len + h->Bmax, h->order_host.data(), h->order_host.size() * 4,
                          hipMemcpyHostToDevice, s));
    if (ld > 0 && maxlen > 0) {
      if (h->bf16)
        launch_prefix_copy<bf16_t>((const bf16_t*)k, (const bf16_t*)v, h->L, batch, batch, ld,
                                   h->Hkv, h->dh, (bf16_t*)h->karena, (bf16_t*)h->vtarena,
                                   h->Bmax, h->S, h->d_len, s);
      else
        launch_prefix_copy<float>((const float*)k, (const float*)v, h->L, batch, batch, ld, h->Hkv,
                                  h->dh, (float*)h->karena, (float*)h->vtarena, h->Bmax, h->S,
                                  h->d_len, s);
      check_launch();
    }
    // The host copy of len must stay valid until the async copy has read it.
    FV_HIP(hipStreamSynchronize(s));
    h->batch = batch;
    h->prefix_set = true;
  });
}

fv_status fv_set_prefix_async(fv_handle h, const void* k, const void* v, const int32_t* len_host,
                              int32_t batch, int32_t ld, void* copy_stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need(k, "k");
    need(v, "v");
    need(len_host, "len_host");
    if (batch < 1 || batch > h->Bmax)
      fail(FV_ERR_INVALID_ARG, "batch must be in [1, max_batch=" + std::to_string(h->Bmax) + "]");
    int maxlen = 0;
    for (int b = 0; b < batch; ++b) {
      if (len_host[b] < 0 || len_host[b] > h->Pmax)
        fail(FV_ERR_INVALID_ARG, "len[" + std::to_string(b) + "] outside [0, max_prefix]");
      maxlen = std::max(maxlen, (int)len_host[b]);
    }
    if (ld < maxlen || ld < 0) fail(FV_ERR_INVALID_ARG, "ld must be >= max(len)");
    DeviceScope ds(h->device);
    if (!h->async_ready) {  // second arena slot and the ordering events, once
      const size_t arena = (size_t)h->L * h->Bmax * h->Hkv * h->S * h->dh * h->esz;
      h->arena_k[1] = dalloc(h, arena);
      h->arena_v[1] = dalloc(h, arena);
      h->len_slot[1] = static_cast<int*>(dalloc(h, (size_t)h->Bmax * (1 + h->Hkv) * 4));
      FV_HIP(hipMemset(h->arena_k[1], 0, arena));
      FV_HIP(hipMemset(h->arena_v[1], 0, arena));
      for (int i = 0; i < 2; ++i) {
        FV_HIP(hipEventCreateWithFlags(&h->ev_ready[i], hipEventDisableTiming));
        FV_HIP(hipEventCreateWithFlags(&h->ev_done[i], hipEventDisableTiming));
        FV_HIP(hipEventCreateWithFlags(&h->ev_len[i], hipEventDisableTiming));
        FV_HIP(hipHostMalloc(reinterpret_cast<void**>(&h->pinned_len[i]),
                             (size_t)h->Bmax * (1 + h->Hkv) * 4, hipHostMallocDefault));
      }
      h->async_ready = true;
    }
    hipStream_t cs = static_cast<hipStream_t>(copy_stream);
    const int sl = h->staged_slot >= 0 ? h->staged_slot : 1 - h->cur_slot;
    // the slot's previous readers and the previous copy from its length
    // buffer must be done before it is overwritten
    if (h->done_recorded[sl]) FV_HIP(hipStreamWaitEvent(cs, h->ev_done[sl], 0));
    if (h->staged_slot >= 0) FV_HIP(hipStreamWaitEvent(cs, h->ev_ready[sl], 0));
    if (h->len_recorded[sl]) FV_HIP(hipEventSynchronize(h->ev_len[sl]));
    std::memcpy(h->pinned_len[sl], len_host, (size_t)batch * 4);
    die_order(h->pinned_len[sl], batch, h->Hkv, h->pinned_len[sl] + h->Bmax);
    (void)hipGetLastError();
    FV_HIP(hipMemcpyAsync(h->len_slot[sl], h->pinned_len[sl], (size_t)batch * 4,
                          hipMemcpyHostToDevice, cs));
    FV_HIP(hipMemcpyAsync(h->len_slot[sl] + h->Bmax, h->pinned_len[sl] + h->Bmax,
                          (size_t)batch * h->Hkv * 4, hipMemcpyHostToDevice, cs));
    FV_HIP(hipEventRecord(h->ev_len[sl], cs));
    h->len_recorded[sl] = true;
    if (ld > 0 && maxlen > 0) {
      if (h->bf16)
        launch_prefix_copy<bf16_t>((const bf16_t*)k, (const bf16_t*)v, h->L, batch, batch, ld,
                                   h->Hkv, h->dh, (bf16_t*)h->arena_k[sl],
                                   (bf16_t*)h->arena_v[sl], h->Bmax, h->S, h->len_slot[sl], cs);
      else
        launch_prefix_copy<float>((const float*)k, (const float*)v, h->L, batch, batch, ld, h->Hkv,
                                  h->dh, (float*)h->arena_k[sl], (float*)h->arena_v[sl], h->Bmax,
                                  h->S, h->len_slot[sl], cs);
      check_launch();
    }
    FV_HIP(hipEventRecord(h->ev_ready[sl], cs));
    h->len_host_slot[sl].assign(len_host, len_host + batch);
    h->staged_slot = sl;
    h->staged_batch = batch;
  });
}

fv_status fv_decode_step(fv_handle h, float* buffer, const float* t, float* out_chunk,
                         void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    // every check precedes the first side effect (switching to a staged
    // observation enqueues a wait on the caller's stream)
    need_prefix(h);
    check_ptr(buffer, "buffer");
    if (t) check_ptr(t, "t_per_chunk");
    check_ptr(out_chunk, "out_chunk");
    const int B = pending_batch(h);
    const size_t nbuf = (size_t)B * h->T * h->A * 4, nout = (size_t)B * h->C * h->A * 4;
    if (overlap(buffer, nbuf, out_chunk, nout)) fail(FV_ERR_INVALID_ARG, "buffer and out_chunk overlap");
    const float* tt = schedule_or(h, t, B);
    const float* mod = t ? nullptr : h->mod_cache;
    DeviceScope ds(h->device);
    hipStream_t st = static_cast<hipStream_t>(stream);
    activate_staged(h, st);
    run_step(h, t ? KIND_STEP : KIND_STEP_CACHED, buffer, tt, out_chunk, nullptr, 0, st,
             [&](hipStream_t s) { decode(h, buffer, tt, B, out_chunk, s, mod); });
    mark_used(h, st);
  });
}

fv_status fv_decode_step_noalloc(fv_handle h, float* buffer, const float* t, float* out_chunk,
                                 void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    check_ptr(buffer, "buffer");
    if (t) check_ptr(t, "t_per_chunk");
    check_ptr(out_chunk, "out_chunk");
    const int B = pending_batch(h);
    const size_t nbuf = (size_t)B * h->T * h->A * 4, nout = (size_t)B * h->C * h->A * 4;
    if (overlap(buffer, nbuf, out_chunk, nout)) fail(FV_ERR_INVALID_ARG, "buffer and out_chunk overlap");
    const float* tt = schedule_or(h, t, B);
    const float* mod = t ? nullptr : h->mod_cache;
    const StepScratch need = step_scratch(h, B);
    if (need.total() > kStaticScratchBytes)
      fail(FV_ERR_INVALID_ARG, "a step at batch " + std::to_string(B) + " needs " +
                                   std::to_string(need.total()) +
                                   " bytes of scratch; the static scratch holds " +
                                   std::to_string(kStaticScratchBytes) +
                                   " (use fv_decode_step)");
    DeviceScope ds(h->device);
    unsigned char* base = static_cast<unsigned char*>(static_scratch(h->device));
    hipStream_t st = static_cast<hipStream_t>(stream);
    activate_staged(h, st);
    {
      ScratchSwap sw(h, base, need);
      (void)hipGetLastError();
      decode(h, buffer, tt, B, out_chunk, st, mod);
      check_launch();
    }
    mark_used(h, st);
  });
}

fv_status fv_velocity(fv_handle h, const float* buffer, const float* t, float* v_out,
                      void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    check_ptr(buffer, "buffer");
    if (t) check_ptr(t, "t");
    check_ptr(v_out, "v_out");
    const int B = pending_batch(h);
    const size_t nbuf = (size_t)B * h->T * h->A * 4;
    if (overlap(buffer, nbuf, v_out, nbuf)) fail(FV_ERR_INVALID_ARG, "buffer and v_out overlap");
    const float* tt = schedule_or(h, t, B);
    const float* mod = t ? nullptr : h->mod_cache;
    DeviceScope ds(h->device);
    hipStream_t st = static_cast<hipStream_t>(stream);
    activate_staged(h, st);
    run_step(h, t ? KIND_VELOCITY : KIND_VELOCITY_CACHED, buffer, tt, v_out, nullptr, 0, st,
             [&](hipStream_t s) { forward(h, buffer, tt, B, v_out, h->L, s, mod); });
    mark_used(h, st);
  });
}

fv_status fv_euler_shift(fv_handle h, float* buffer, const float* t, const float* v,
                         float* out_chunk, void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    check_ptr(buffer, "buffer");
    check_ptr(t, "t");
    check_ptr(v, "v");
    check_ptr(out_chunk, "out_chunk");
    const int B = h->batch > 0 ? h->batch : 1;
    const size_t nbuf = (size_t)B * h->T * h->A * 4, nout = (size_t)B * h->C * h->A * 4;
    if (overlap(buffer, nbuf, out_chunk, nout)) fail(FV_ERR_INVALID_ARG, "buffer and out_chunk overlap");
    DeviceScope ds(h->device);
    (void)hipGetLastError();
    launch_euler_shift(buffer, t, v, out_chunk, h->d_noise, h->d_ticket, h->d_valid, B, h->K,
                       h->C * h->A, static_cast<hipStream_t>(stream));
    check_launch();
  });
}

fv_status fv_sequential_decode(fv_handle h, const float* noise, int32_t n_steps,
                               float* out_chunk, void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    if (h->K != 1) fail(FV_ERR_STATE, "fv_sequential_decode needs a handle with n_chunks == 1");
    check_ptr(noise, "noise");
    check_ptr(out_chunk, "out_chunk");
    if (n_steps < 1 || n_steps > 4096) fail(FV_ERR_INVALID_ARG, "n_steps must be in [1, 4096]");
    DeviceScope ds(h->device);
    float* ts = nullptr;
    for (auto& e : h->tscheds)
      if (e.first == n_steps) ts = e.second;
    if (!ts) {
      std::vector<float> tv(n_steps + 1);
      for (int j = 0; j <= n_steps; ++j) tv[j] = (float)((double)(n_steps - j) / (double)n_steps);
      ts = upload_f32(h, tv.data(), tv.size(), false);
      h->tscheds.emplace_back(n_steps, ts);
    }
    activate_staged(h, static_cast<hipStream_t>(stream));
    const int B = h->batch;
    const size_t n = (size_t)B * h->C * h->A;
    run_step(h, KIND_SEQ, noise, out_chunk, nullptr, nullptr, n_steps,
             static_cast<hipStream_t>(stream), [&](hipStream_t s) {
               launch_copy_f32(h->seq_x, noise, n, s);
               for (int j = 0; j < n_steps; ++j) {
                 launch_fill_t(h->seq_t, ts, j, B, s);
                 forward(h, h->seq_x, h->seq_t, B, h->v, h->L, s);
                 launch_seq_euler(h->seq_x, h->v, ts, j, (int)n, s);
               }
               launch_copy_f32(out_chunk, h->seq_x, n, s);
             });
    mark_used(h, static_cast<hipStream_t>(stream));
  });
}

fv_status fv_set_valid_slots(fv_handle h, const int32_t* n_valid, int32_t count) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need(n_valid, "n_valid");
    if (count < 1 || count > h->Bmax) fail(FV_ERR_INVALID_ARG, "count outside 1..max_batch");
    for (int b = 0; b < count; ++b)
      if (n_valid[b] < 1 || n_valid[b] > h->K)
        fail(FV_ERR_INVALID_ARG, "valid slot count outside 1..n_chunks");
    DeviceScope ds(h->device);
    FV_HIP(hipDeviceSynchronize());
    FV_HIP(hipMemcpy(h->d_valid, n_valid, (size_t)count * 4, hipMemcpyHostToDevice));
  });
}

fv_status fv_multibuffer_velocity(fv_handle h, const void* k, const void* v, int32_t prefix_len,
                                  int32_t ld, const float* buffers, const float* t, float* v_out,
                                  void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need(k, "k");
    need(v, "v");
    check_ptr(buffers, "buffers");
    check_ptr(t, "t");
    check_ptr(v_out, "v_out");
    const int N = h->K;
    if (h->Bmax < N) fail(FV_ERR_INVALID_ARG, "max_batch must be >= n_chunks");
    if (prefix_len < 0 || prefix_len > h->Pmax) fail(FV_ERR_INVALID_ARG, "prefix_len out of range");
    if (ld < prefix_len) fail(FV_ERR_INVALID_ARG, "ld must be >= prefix_len");
    DeviceScope ds(h->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    // one observation for all N configurations; configuration j (stream j-1)
    // holds j real chunks after N - j padding slots
    h->staged_slot = -1;  // a pending asynchronous observation is superseded
    h->len_host.assign(N, prefix_len);
    h->order_host.resize((size_t)N * h->Hkv);
    die_order(h->len_host.data(), N, h->Hkv, h->order_host.data());
    std::vector<int> valid(N);
    for (int j = 0; j < N; ++j) valid[j] = j + 1;
    FV_HIP(hipMemcpyAsync(h->d_len, h->len_host.data(), (size_t)N * 4, hipMemcpyHostToDevice, s));
    FV_HIP(hipMemcpyAsync(h->d_len + h->Bmax, h->order_host.data(), h->order_host.size() * 4,
                          hipMemcpyHostToDevice, s));
    FV_HIP(hipMemcpyAsync(h->d_valid, valid.data(), (size_t)N * 4, hipMemcpyHostToDevice, s));
    if (ld > 0 && prefix_len > 0) {
      if (h->bf16)
        launch_prefix_copy<bf16_t>((const bf16_t*)k, (const bf16_t*)v, h->L, N, 1, ld, h->Hkv,
                                   h->dh, (bf16_t*)h->karena, (bf16_t*)h->vtarena, h->Bmax, h->S,
                                   h->d_len, s);
      else
        launch_prefix_copy<float>((const float*)k, (const float*)v, h->L, N, 1, ld, h->Hkv, h->dh,
                                  (float*)h->karena, (float*)h->vtarena, h->Bmax, h->S, h->d_len,
                                  s);
      check_launch();
    }
    FV_HIP(hipStreamSynchronize(s));  // the host copies above must stay valid until read
    h->batch = N;
    h->prefix_set = true;
    run_step(h, KIND_VELOCITY, buffers, t, v_out, nullptr, 0, s,
             [&](hipStream_t st) { forward(h, buffers, t, N, v_out, h->L, st); });
    mark_used(h, s);
  });
}

fv_status fv_set_mask_mode(fv_handle h, int32_t mode) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    if (mode != FV_MASK_CHUNK_CAUSAL && mode != FV_MASK_ISOLATED && mode != FV_MASK_BIDIRECTIONAL)
      fail(FV_ERR_INVALID_ARG, "unknown mask mode");
    if (mode == h->mask_mode) return;
    DeviceScope ds(h->device);
    clear_graphs(h);
    h->mask_mode = mode;
  });
}

fv_status fv_set_schedule(fv_handle h, const float* t, void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    check_ptr(t, "t");
    DeviceScope ds(h->device);
    if (!h->mod_cache) {
      h->mod_cache = static_cast<float*>(dalloc(h, (size_t)h->Bmax * h->K * h->Nmod * 4));
      h->t_cache = static_cast<float*>(dalloc(h, (size_t)h->Bmax * h->K * 4));
      h->d_sched_period = static_cast<int*>(dalloc(h, 4));
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    const int B = h->batch;
    launch_copy_f32(h->t_cache, t, (size_t)B * h->K, s);
    h->sched_per = film_maps(h, h->t_cache, B, h->mod_cache, s, h->d_sched_period);
    check_launch();
    h->sched_batch = B;
  });
}

fv_status fv_cold_start(fv_handle h, float* buffer, int32_t first_stream, int32_t n_streams,
                        void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    check_ptr(buffer, "buffer");
    if (first_stream < 0 || n_streams < 1 || first_stream + n_streams > h->batch)
      fail(FV_ERR_INVALID_ARG, "stream range outside the active batch");
    DeviceScope ds(h->device);
    (void)hipGetLastError();
    launch_cold_start(buffer, h->d_noise, h->d_valid, first_stream, n_streams, h->K, h->C * h->A,
                      static_cast<hipStream_t>(stream));
    check_launch();
  });
}

fv_status fv_get_valid_slots(fv_handle h, int32_t* out, int32_t count) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need(out, "out");
    if (count < 1 || count > h->Bmax) fail(FV_ERR_INVALID_ARG, "count outside 1..max_batch");
    DeviceScope ds(h->device);
    FV_HIP(hipDeviceSynchronize());
    FV_HIP(hipMemcpy(out, h->d_valid, (size_t)count * 4, hipMemcpyDeviceToHost));
  });
}

fv_status fv_get_noise_state(fv_handle h, uint64_t* seed, uint64_t* step) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need(seed, "seed");
    need(step, "step");
    DeviceScope ds(h->device);
    FV_HIP(hipDeviceSynchronize());
    uint64_t ns[2];
    FV_HIP(hipMemcpy(ns, h->d_noise, 16, hipMemcpyDeviceToHost));
    *seed = ns[0];
    *step = ns[1];
  });
}

fv_status fv_set_noise_state(fv_handle h, uint64_t seed, uint64_t step) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    DeviceScope ds(h->device);
    FV_HIP(hipDeviceSynchronize());
    const uint64_t ns[2] = {seed, step};
    FV_HIP(hipMemcpy(h->d_noise, ns, 16, hipMemcpyHostToDevice));
  });
}

fv_status fv_set_graph_mode(fv_handle h, int32_t enabled) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    if (enabled != 0 && enabled != 1) fail(FV_ERR_INVALID_ARG, "enabled must be 0 or 1");
    h->use_graphs = enabled == 1;
  });
}

fv_status fv_query(fv_handle h, int32_t what, int32_t batch, int64_t* value) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    check_ptr(value, "value");
    switch (what) {
      case FV_QUERY_ATTN_SPLITS:
        if (batch < 1 || batch > h->Bmax) fail(FV_ERR_INVALID_ARG, "batch outside 1..max_batch");
        *value = attn_split(h, batch);
        break;
      case FV_QUERY_DEVICE_BYTES:
        *value = (int64_t)h->device_bytes;
        break;
      case FV_QUERY_OUT_PROJ_SPLITS:
        if (batch < 1 || batch > h->Bmax) fail(FV_ERR_INVALID_ARG, "batch outside 1..max_batch");
        *value = plan_gemm(batch * h->T, h->W, h->Hq * h->dh, h->bf16, true).ks;
        break;
      case FV_QUERY_NOALLOC_SCRATCH_BYTES:
        if (batch < 1 || batch > h->Bmax) fail(FV_ERR_INVALID_ARG, "batch outside 1..max_batch");
        *value = (int64_t)step_scratch(h, batch).total();
        break;
      default:
        fail(FV_ERR_INVALID_ARG, "unknown query");
    }
  });
}

fv_status fv_debug_forward(fv_handle h, const float* buffer, const float* t, int32_t n_layers_run,
                           float* h_out, float* mod_out, void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    check_ptr(buffer, "buffer");
    check_ptr(t, "t");
    check_ptr(h_out, "h_out");
    if (n_layers_run < 0 || n_layers_run > h->L) fail(FV_ERR_INVALID_ARG, "n_layers_run out of range");
    DeviceScope ds(h->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    activate_staged(h, s);
    (void)hipGetLastError();
    const int B = h->batch;
    forward(h, buffer, t, B, nullptr, n_layers_run, s, nullptr, nullptr, false);  // every FiLM row
    launch_copy_f32(h_out, h->hres, (size_t)B * h->T * h->W, s);
    if (mod_out) launch_copy_f32(mod_out, h->mod, (size_t)B * h->K * h->Nmod, s);
    check_launch();
    mark_used(h, s);
  });
}

fv_status fv_debug_stage(fv_handle h, int32_t stage, int32_t layer, int32_t reps, void* stream) {
  if (!h) return FV_ERR_INVALID_ARG;
  return guarded(h, [&] {
    need_prefix(h);
    if (stage < 0 || stage > 11) fail(FV_ERR_INVALID_ARG, "stage must be 0..11");
    if (layer < -1 || layer >= h->L) fail(FV_ERR_INVALID_ARG, "layer out of range");
    if (reps < 1 || reps > 100000) fail(FV_ERR_INVALID_ARG, "reps must be 1..100000");
    if (h->staged_slot >= 0) fail(FV_ERR_STATE, "a staged observation is pending");
    DeviceScope ds(h->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // layer -1: repetition r runs layer r mod L, as the step walks the layers
    run_step(h, KIND_STAGE, nullptr, nullptr, nullptr, nullptr,
             (stage + 16 * (layer + 1)) + 4096 * reps, s, [&](hipStream_t st) {
               for (int r = 0; r < reps; ++r) {
                 const int l = layer >= 0 ? layer : r % h->L;
                 if (h->bf16)
                   run_stage<bf16_t>(h, stage, l, st);
                 else
                   run_stage<float>(h, stage, l, st);
               }
             });
    mark_used(h, s);
  });
}

fv_status fv_destroy(fv_handle h) {
  if (!h) return FV_ERR_INVALID_ARG;
  {
    int prev = -1;
    (void)hipGetDevice(&prev);
    (void)hipSetDevice(h->device);
    destroy_handle(h);
    if (prev >= 0) (void)hipSetDevice(prev);
  }
  delete h;
  return FV_OK;
}

}  // extern "C"
