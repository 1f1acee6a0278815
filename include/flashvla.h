/*
 * flashvla.h -- C ABI of the MI355X (gfx950) streaming action-decode library.
 *
 * One call of fv_decode_step() is one steady-streaming step of FlashVLA
 * (Li, Tang, Liu, "FlashVLA: Streaming Action Decoding for Fast and
 * Asynchronous VLA Inference"): a single forward pass of the flow-matching
 * action expert over a buffer of K action chunks held at staggered noise
 * levels (Sec. 3.1, Eq. 2), under the chunk-wise causal mask with a cached
 * observation prefix (Sec. 3.1), followed by one Euler step of every chunk
 * (Eq. 1: x <- x - dt * v, tau = 1 is noise), emission of the cleanest chunk,
 * a shift of the others, and fresh Gaussian noise in the last slot (Sec. 3.2,
 * Algorithm 1, steady streaming).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - Every call returns an fv_status and never aborts; C++ exceptions are
 *    caught at this boundary and reported as FV_ERR_INTERNAL.
 *  - Arguments are validated synchronously before anything is enqueued, so
 *    a call that returns an error has had no side effect on caller memory.
 *  - "dev" pointers are device memory of the GPU the handle was created on,
 *    owned by the caller and borrowed only for the stream-ordered duration of
 *    the call.  "host" pointers are read before the call returns.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *    on it and the call returns without waiting; completion is observed on
 *    that stream.
 *  - A handle is not thread-safe; separate handles are independent.
 *  - All sizes are int32 element counts; tensors are dense, row-major, in the
 *    index order written next to them.
 */
#ifndef FLASHVLA_H
#define FLASHVLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FV_ABI_VERSION 2

typedef struct fv_handle_s *fv_handle;

typedef enum {
  FV_OK = 0,
  FV_ERR_INVALID_ARG = 1, /* bad size, pointer, alignment or config */
  FV_ERR_STATE = 2,       /* call not valid in the handle's state */
  FV_ERR_OOM = 3,         /* device allocation failed */
  FV_ERR_HIP = 4,         /* a HIP runtime call or launch failed */
  FV_ERR_INTERNAL = 5     /* unexpected internal error */
} fv_status;

enum { FV_BF16 = 0, FV_FP32 = 1 };

/*
 * Attention masks over the buffer (every action query also sees every valid
 * prefix token; slots holding cold-start padding are never keys of a valid
 * chunk, and a padding chunk's own queries see only itself):
 *  FV_MASK_CHUNK_CAUSAL   chunk k sees chunks <= k (Sec. 3.1; the default);
 *  FV_MASK_ISOLATED       chunk k sees only itself -- the no-causal ablation
 *                         of Appendix "Ablations", where chunks of the buffer
 *                         do not attend to each other;
 *  FV_MASK_BIDIRECTIONAL  chunk k sees every valid chunk.
 */
enum { FV_MASK_CHUNK_CAUSAL = 0, FV_MASK_ISOLATED = 1, FV_MASK_BIDIRECTIONAL = 2 };

/*
 * Shape and numerics of the action expert (Appendix "Model architecture":
 * a pi0.5-style expert whose norms are FiLM-conditioned on each chunk's
 * noise level).
 *
 *  n_layers L, width W, n_q_heads Hq, n_kv_heads Hkv (Hq % Hkv == 0),
 *  head_dim dh, mlp_dim F, action_dim A, chunk_len C, n_chunks K (the
 *  buffer length N of Sec. 3.1), max_prefix (largest observation prefix),
 *  max_batch (largest number of independent streams).
 *  dtype: FV_BF16 -- weights, prefix K/V and GEMM operands in bf16 with fp32
 *         accumulation, fp32 residual stream and fp32 buffer;
 *         FV_FP32 -- fp32 throughout.
 *  mlp_gated: 1 = GeGLU MLP (tanh GELU), 0 = plain tanh-GELU MLP.
 *  rms_eps: RMSNorm epsilon; rope_theta: rotary base for action tokens.
 *  noise_seed: stream b draws its fresh noise with seed noise_seed + b.
 *
 * Requirements (else FV_ERR_INVALID_ARG): every size >= 1 (max_prefix >= 0);
 * W % 128 == 0 and W <= 2048; dh in {64, 128, 192, 256}; F % 64 == 0 (F % 128
 * == 0 for the plain MLP); ((Hq + 2 Hkv) * dh) % 128 == 0; A <= 64;
 * K * C <= 4096; K <= 256; max_prefix + K * C <= 32768; max_batch <= 4096;
 * max_batch * K * C <= 262144; L * max_batch * Hkv <= 65535.
 */
typedef struct {
  int32_t n_layers, width, n_q_heads, n_kv_heads, head_dim, mlp_dim, action_dim;
  int32_t chunk_len, n_chunks, max_prefix, max_batch;
  int32_t dtype, mlp_gated;
  float rms_eps, rope_theta;
  uint64_t noise_seed;
} fv_cfg;

/*
 * Host fp32 expert weights in the y = x W layout (W is [in][out], row-major).
 *  w_in [A][W], b_in [W]             action-token embedding
 *  w_t1 [W][W], b_t1 [W],
 *  w_t2 [W][W], b_t2 [W]             time-MLP: cond = silu(silu(e w_t1 + b_t1) w_t2 + b_t2)
 *  w_mod[n] [W][3W], b_mod[n] [3W]   FiLM map of norm n = 0..2L: columns are
 *                                    [scale | shift | gate]; norm 2l precedes
 *                                    attention of layer l, 2l+1 its MLP, 2L is the
 *                                    final norm (its gate columns are not read)
 *  wq[l] [W][Hq*dh], wk[l], wv[l] [W][Hkv*dh], wo[l] [Hq*dh][W]   (no biases)
 *  wg[l], wu[l] [W][F], wd[l] [F][W] (no biases; wg is NULL when mlp_gated == 0)
 *  w_out [W][A], b_out [A]           velocity head
 * Query/key head h occupies columns [h*dh, (h+1)*dh).
 */
typedef struct {
  const float *w_in, *b_in, *w_t1, *b_t1, *w_t2, *b_t2;
  const float *const *w_mod, *const *b_mod;
  const float *const *wq, *const *wk, *const *wv, *const *wo;
  const float *const *wg, *const *wu, *const *wd;
  const float *w_out, *b_out;
} fv_weights;

/*
 * fv_create -- validate cfg, copy and pack the weights, allocate the handle.
 * The host weights are copied (in FV_BF16 mode each value is rounded to the
 * nearest bf16, ties to even) and may be freed when the call returns.  The
 * handle owns the packed device weights, the observation-prefix arena, the
 * rotary tables, all scratch memory, the captured step graphs and the noise
 * state (seed cfg->noise_seed, step counter 0).  Synchronises the device.
 * Errors: FV_ERR_INVALID_ARG (cfg or a weight pointer), FV_ERR_OOM, FV_ERR_HIP.
 */
fv_status fv_create(const fv_weights *weights, const fv_cfg *cfg, fv_handle *out);

/*
 * fv_set_prefix -- install the cached observation context that every action
 * token attends to (Sec. 3.1: all passes condition on the same observation
 * o_t; the encoder's K/V are computed once per observation).
 *  k, v     dev [L][batch][ld][Hkv][dh], in the cfg dtype (bf16 bit patterns
 *           for FV_BF16, fp32 for FV_FP32); keys already position-encoded.
 *           Rows >= len_host[b] are never read.
 *  len_host host int32 [batch]: valid prefix length of stream b, 0..max_prefix.
 *  batch    number of streams for the following steps, 1..max_batch.
 *  ld       leading row count of k/v, >= max(len_host).
 * The data are copied into the handle's arena on `stream`, and the call
 * waits for that copy to finish before it returns (host-synchronous), so k,
 * v and len_host may be reused as soon as it returns; fv_set_prefix_async is
 * the asynchronous form.  Sets the active batch and cancels a pending
 * fv_set_prefix_async observation.
 * Errors: FV_ERR_INVALID_ARG (NULL pointer, batch, ld or a length out of range),
 * FV_ERR_HIP; after FV_ERR_INVALID_ARG the handle is unchanged.
 */
fv_status fv_set_prefix(fv_handle h, const void *k, const void *v, const int32_t *len_host,
                        int32_t batch, int32_t ld, void *stream);

/*
 * fv_set_prefix_async -- asynchronous observation pipeline: install the
 * prefix of the next observation while the current one is still being
 * decoded (Sec. 4.2: the next inference starts before the current chunk has
 * finished executing).  Same arguments as fv_set_prefix, enqueued on
 * `copy_stream`.  The data go to a second arena slot (allocated by the first
 * call: as much device memory as the first arena), so passes still running
 * on the active observation are unaffected; the next fv_decode_step /
 * fv_velocity / fv_sequential_decode / fv_debug_forward makes its stream
 * wait for this copy and switches to the new observation (and its batch).
 * No host synchronisation except on a slot's third reuse before its previous
 * length copy finished.  A later fv_set_prefix_async before that switch
 * replaces the pending observation; fv_set_prefix cancels it.
 * Errors: FV_ERR_INVALID_ARG (as fv_set_prefix), FV_ERR_OOM, FV_ERR_HIP.
 */
fv_status fv_set_prefix_async(fv_handle h, const void *k, const void *v, const int32_t *len_host,
                              int32_t batch, int32_t ld, void *copy_stream);

/*
 * fv_decode_step -- one streaming step (Algorithm 1).
 *  buffer       dev fp32 [batch][K][C][A], in/out.  Slot 0 is the cleanest chunk.
 *  t_per_chunk  dev fp32 [batch][K]: noise level of each slot (0 < t_0 < ... ),
 *               or NULL to use the schedule installed by fv_set_schedule.
 *  out_chunk    dev fp32 [batch][C][A]: the emitted (executable) chunk.
 * Computes v = v_theta(buffer, t | prefix) for every chunk, then per slot
 * x'_k = x_k - dt_k v_k with dt_k = t_k - t_{k-1} (t_{-1} = 0) in fp32 (product
 * rounded, then difference rounded; no fused multiply-add); writes
 * out_chunk = x'_0, buffer[k] = x'_{k+1} for k < K-1, and buffer[K-1] = fresh
 * N(0, I) noise: Philox4x32-10 keyed by seed_b = seed + b, counter
 * (j, lo32(step), hi32(step), 0) for the j-th group of 4 values of the
 * row-major [C][A] chunk, u = (r + 0.5) 2^-32, Box-Muller in fp64, rounded to
 * fp32.  Then the step counter advances by one.  With t_{K-1} = 1 and
 * t_k - dt_k = t_{k-1}, the shifted buffer sits again at t_per_chunk.
 * A stream in cold start (fewer than K valid slots, see fv_cold_start) pops
 * a padding slot: its out_chunk is all zeros (the caller executes its safe
 * default action) and it gains one valid slot.
 * buffer and out_chunk must not overlap (FV_ERR_INVALID_ARG).  A staged
 * fv_set_prefix_async observation is switched to only after every check has
 * passed.  The first call with a new set of
 * pointers captures a HIP graph (host-synchronous); later calls replay it.
 * Errors: FV_ERR_STATE (no prefix set; t_per_chunk NULL without a schedule
 * for the active batch), FV_ERR_INVALID_ARG (NULL or misaligned pointer:
 * 16-byte alignment required), FV_ERR_HIP.
 */
fv_status fv_decode_step(fv_handle h, float *buffer, const float *t_per_chunk, float *out_chunk,
                         void *stream);

/*
 * fv_decode_step_noalloc -- fv_decode_step for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops and
 * harnesses that forbid hipMalloc.  Same arguments, checks, semantics and
 * results (bit-identical) as fv_decode_step, but nothing is allocated or
 * freed: the kernels are launched one by one on `stream` (no graph is
 * captured or instantiated), and the step's scratch -- the attention
 * key-split partials and the split-K partial tiles -- lives in a static
 * device array of FV_NOALLOC_SCRATCH_BYTES (24 MiB) that each GPU the library
 * runs on holds until the process ends, instead of the handle's own scratch.
 * A step that needs more (fv_query FV_QUERY_NOALLOC_SCRATCH_BYTES; the
 * pi0.5-shaped expert needs about 21 MB at batch 1 and more at batch 2 to 8)
 * returns FV_ERR_INVALID_ARG.  Every call on a GPU shares that GPU's array
 * and nothing in it needs to start at zero; calls that overlap on one GPU
 * (from any handle or stream) race.
 * Errors: as fv_decode_step, plus FV_ERR_INVALID_ARG (scratch too small for
 * the active batch) and FV_ERR_HIP (the array's address is unavailable).
 */
#define FV_NOALLOC_SCRATCH_BYTES (24u << 20)
fv_status fv_decode_step_noalloc(fv_handle h, float *buffer, const float *t_per_chunk,
                                 float *out_chunk, void *stream);

/*
 * fv_velocity -- the velocity pass alone (the v_theta of Eq. 1).
 *  buffer dev fp32 [batch][K][C][A] (read only), t dev fp32 [batch][K] (or
 *  NULL: the installed schedule), v_out dev fp32 [batch][K][C][A].  Uses the
 *  current mask mode and each stream's padding slots like fv_decode_step.
 * Same kernels, same order and same results as the pass inside fv_decode_step.
 * buffer and v_out must not overlap.  Errors: as fv_decode_step.
 */
fv_status fv_velocity(fv_handle h, const float *buffer, const float *t, float *v_out,
                      void *stream);

/*
 * fv_euler_shift -- the queue update of fv_decode_step for a caller-given
 * velocity v (dev fp32 [batch][K][C][A]); buffer, t and out_chunk as in
 * fv_decode_step.  Draws the tail noise at the current step and advances the
 * step counter.  Needs no prefix.  Errors: FV_ERR_INVALID_ARG, FV_ERR_HIP.
 */
fv_status fv_euler_shift(fv_handle h, float *buffer, const float *t, const float *v,
                         float *out_chunk, void *stream);

/*
 * fv_sequential_decode -- the isolated per-chunk decode the paper starts from
 * (Sec. 3.1: each chunk is denoised from pure noise by several sequential
 * expert passes conditioned on the same observation).  Needs a handle with
 * n_chunks == 1.  noise dev fp32 [batch][C][A] (read only); n_steps >= 1;
 * out_chunk dev fp32 [batch][C][A].  Runs x <- x - (t_j - t_{j+1}) v(x, t_j)
 * for t_j = (n_steps - j)/n_steps (fp32), j = 0..n_steps-1, t_{n_steps} = 0,
 * and writes the final x.  Does not touch the noise state.
 * Errors: FV_ERR_STATE (no prefix, or n_chunks != 1), FV_ERR_INVALID_ARG, FV_ERR_HIP.
 */
fv_status fv_sequential_decode(fv_handle h, const float *noise, int32_t n_steps,
                               float *out_chunk, void *stream);

/*
 * Noise state (seed and step counter) for bit-exact resume.  Both calls
 * synchronise the device first.  Errors: FV_ERR_INVALID_ARG (NULL pointer).
 */
fv_status fv_get_noise_state(fv_handle h, uint64_t *seed, uint64_t *step);
fv_status fv_set_noise_state(fv_handle h, uint64_t seed, uint64_t step);

/*
 * fv_set_mask_mode -- attention mask of the following passes (FV_MASK_*).
 * Drops the captured graphs (they are captured again on next use).
 * Errors: FV_ERR_INVALID_ARG (unknown mode).
 */
fv_status fv_set_mask_mode(fv_handle h, int32_t mode);

/*
 * fv_set_schedule -- static-schedule cache.  In steady state every step uses
 * the same per-slot noise levels, so the FiLM modulation of every norm (a
 * function of t only) is the same at every step.  Computes it once for
 *  t dev fp32 [batch][K] (the active batch, as fv_decode_step's t_per_chunk)
 * and keeps it, with a copy of t, in the handle; fv_decode_step and
 * fv_velocity called with t == NULL then skip the time embedding, the
 * time-MLP and the FiLM map products.  Results are bit-identical to passing
 * t.  The first call allocates the cache (max_batch * K * (6L+2) * W fp32);
 * later calls reuse it.  Stream-ordered.
 * Errors: FV_ERR_STATE (no prefix set), FV_ERR_INVALID_ARG, FV_ERR_OOM, FV_ERR_HIP.
 */
fv_status fv_set_schedule(fv_handle h, const float *t, void *stream);

/*
 * fv_cold_start -- start an episode for streams [first_stream, first_stream
 * + n_streams) of the active batch (Sec. 3.2, Algorithm 1, cold start): slots
 * 0..K-2 of their buffer become padding chunks (zeros, never attended to by a
 * valid chunk) and slot K-1 a fresh N(0, I) chunk drawn as fv_decode_step
 * draws its tail, at the current step counter; the step counter then advances
 * by one.  Those streams then have one valid slot; each fv_decode_step adds
 * one, and the first K-1 steps emit zeros.  Other streams are untouched.
 *  buffer dev fp32 [batch][K][C][A], in/out.  Stream-ordered; no graph.
 * Errors: FV_ERR_STATE (no prefix set), FV_ERR_INVALID_ARG (range outside the
 * active batch, NULL or misaligned buffer), FV_ERR_HIP.
 */
fv_status fv_cold_start(fv_handle h, float *buffer, int32_t first_stream, int32_t n_streams,
                        void *stream);

/*
 * fv_get_valid_slots -- number of valid (non-padding) slots of the first
 * `count` streams (K for a stream in steady state), into host int32
 * out[count].  Synchronises the device.
 * Errors: FV_ERR_INVALID_ARG (NULL out, count outside 1..max_batch).
 */
fv_status fv_get_valid_slots(fv_handle h, int32_t *out, int32_t count);

/*
 * fv_set_valid_slots -- set the valid (non-padding) slot count of the first
 * `count` streams from host int32 n_valid[count] (each 1..K; the last
 * n_valid slots of a stream are real chunks).  Restores a saved cold-start
 * state; fv_cold_start and fv_decode_step maintain the counts otherwise.
 * Synchronises the device.
 * Errors: FV_ERR_INVALID_ARG (NULL, count outside 1..max_batch, a count
 * outside 1..K).
 */
fv_status fv_set_valid_slots(fv_handle h, const int32_t *n_valid, int32_t count);

/*
 * fv_multibuffer_velocity -- forward pass of the packed multi-buffer sample
 * of Sec. 3.3 for one observation: the N = K buffer configurations that cold
 * start passes through, configuration j (j = 1..N) holding N - j padding
 * chunks followed by j real chunks, all attending to the same observation
 * and isolated from each other.  Configuration j runs as stream j - 1.
 *  k, v       dev [L][ld][Hkv][dh] (cfg dtype): the one observation prefix,
 *             installed for all N streams (prefix_len rows valid).
 *  buffers    dev fp32 [N][K][C][A]: configuration j at index j - 1.
 *  t          dev fp32 [N][K]: slot noise levels of every configuration.
 *  v_out      dev fp32 [N][K][C][A]: velocities (padding slots: unused values).
 * Leaves the handle with batch N, that prefix, and valid slot counts
 * 1..N.  Needs max_batch >= K.  Host-synchronous for the prefix install.
 * Errors: FV_ERR_INVALID_ARG (pointers, prefix_len, ld, max_batch < K),
 * FV_ERR_HIP.
 */
fv_status fv_multibuffer_velocity(fv_handle h, const void *k, const void *v, int32_t prefix_len,
                                  int32_t ld, const float *buffers, const float *t, float *v_out,
                                  void *stream);

/*
 * fv_set_graph_mode -- 1 (default): each step is one hipGraphLaunch of a
 * captured graph; 0: kernels are launched one by one on the caller's stream
 * (same kernels, same results).  Errors: FV_ERR_INVALID_ARG.
 */
fv_status fv_set_graph_mode(fv_handle h, int32_t enabled);

/*
 * fv_query -- host-side introspection of a handle; launches nothing.
 *  FV_QUERY_ATTN_SPLITS: number of key ranges the attention splits each
 *    query tile into at batch `batch` (1: no split, no combine kernel);
 *  FV_QUERY_DEVICE_BYTES: device memory the handle holds (weights, prefix
 *    arenas, scratch, workspace), in bytes; `batch` is ignored;
 *  FV_QUERY_NOALLOC_SCRATCH_BYTES: static scratch fv_decode_step_noalloc
 *    needs for a step at batch `batch` (accepted when at most
 *    FV_NOALLOC_SCRATCH_BYTES);
 *  FV_QUERY_OUT_PROJ_SPLITS: split-K factor of the output projection at batch
 *    `batch` (1: unsplit, the gated residual runs in the GEMM's epilogue;
 *    more: split partials reduced with the residual and the next norm).
 * `value` is a host pointer.  Errors: FV_ERR_INVALID_ARG (NULL handle or
 * value, unknown `what`, batch outside 1..max_batch for the split query).
 */
enum { FV_QUERY_ATTN_SPLITS = 1, FV_QUERY_DEVICE_BYTES = 2, FV_QUERY_NOALLOC_SCRATCH_BYTES = 3,
       FV_QUERY_OUT_PROJ_SPLITS = 4 };
fv_status fv_query(fv_handle h, int32_t what, int32_t batch, int64_t *value);

/* fv_destroy -- synchronise the device and free everything the handle owns. */
fv_status fv_destroy(fv_handle h);

/* Static description of a status code. */
const char *fv_status_string(fv_status s);

/* Message of the handle's last failed call; owned by the handle, valid until
 * its next call.  Returns "" for a NULL handle. */
const char *fv_last_error(fv_handle h);

/* FV_ABI_VERSION of the built library. */
int32_t fv_abi_version(void);

/*
 * fv_debug_forward -- inspection aid for tests: runs the velocity pass up to
 * and including layer n_layers_run - 1 (0 = embedding only) and copies out
 *  h_out   dev fp32 [batch][K*C][W]: the residual stream at that point, and
 *  mod_out dev fp32 [batch][K][(6L+2)*W] (may be NULL): every FiLM parameter,
 *          norm n < 2L at offset 3*W*n as [scale | shift | gate], the final
 *          norm at 6*L*W as [scale | shift].
 * Errors: as fv_velocity, plus FV_ERR_INVALID_ARG for n_layers_run > L.
 */
fv_status fv_debug_forward(fv_handle h, const float *buffer, const float *t,
                           int32_t n_layers_run, float *h_out, float *mod_out, void *stream);

/*
 * fv_debug_stage -- measurement aid: re-launches one kernel stage of the most
 * recent velocity pass (fv_velocity, fv_decode_step or fv_debug_forward with
 * the same batch) `reps` times on `stream`, reading the activations that pass
 * left in the handle's scratch memory.  `layer` selects the layer's weights
 * and arena; -1 makes repetition r use layer r mod L, as a step walks the
 * layers.  In graph mode (the default) the reps launches are captured once
 * into a HIP graph and replayed, so each launch is dispatched as inside a
 * step.  Stages 0-5 rewrite scratch memory only and give the same result on
 * every repetition; stages 6-11 add into the residual stream or rewrite the
 * normalised activations (timing aid only: run a velocity pass again before
 * reading results).
 *  stage 0: FiLM maps (cond -> every norm's [scale | shift | gate]);
 *  stage 1: packed QKV GEMM + rotary + K/V arena write;
 *  stage 2: chunk-causal attention (both kernels);
 *  stage 3: packed gate/up GEMM + GeGLU (or GELU);
 *  stage 4: attention score/value kernel alone (per-split partials);
 *  stage 5: attention split combine alone (no launch when nothing is split);
 *  stage 6: output projection + gated residual + next FiLM RMSNorm;
 *  stage 7: down projection + gated residual + next FiLM RMSNorm;
 *  stage 8: output projection GEMM alone (its split-K partials, or the GEMM
 *           with the gated residual in its epilogue when k is not split);
 *  stage 9: down projection GEMM alone (likewise);
 *  stage 10: the kernel after the output projection alone (split-K reduction
 *           + gated residual + FiLM norm, or the FiLM norm);
 *  stage 11: the kernel after the down projection alone (likewise).
 * Errors: FV_ERR_STATE (no prefix, or a staged observation pending),
 * FV_ERR_INVALID_ARG (stage 0..11, layer -1..L-1, reps 1..100000).
 */
fv_status fv_debug_stage(fv_handle h, int32_t stage, int32_t layer, int32_t reps, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FLASHVLA_H */
