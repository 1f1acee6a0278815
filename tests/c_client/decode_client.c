/*
 * A plain C99 client of the streaming action-decode library, used by the
 * tests: it reads an fp32 expert, an observation prefix, a buffer and its
 * noise levels from raw little-endian fp32 files, runs one velocity pass
 * (fv_velocity) and one decode step (fv_decode_step) through the C ABI, and
 * writes the velocity, the emitted chunk and the buffer after the step.
 *
 * usage: decode_client DIR L W Hq Hkv dh F A C K P
 *   DIR/weights.bin  every weight of fv_weights in declaration order (w_mod
 *                    and b_mod per norm n = 0..2L, the per-layer matrices
 *                    per layer), each [in][out] row-major
 *   DIR/prefix_k.bin, DIR/prefix_v.bin   [L][1][P][Hkv][dh]
 *   DIR/buffer.bin [1][K][C][A], DIR/t.bin [1][K]
 * writes DIR/v.bin, DIR/out.bin, DIR/buffer_after.bin.  Exit status 0 on
 * success; a failed call prints the library's message.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "flashvla.h"

static void die(const char *what) {
  fprintf(stderr, "decode_client: %s\n", what);
  exit(1);
}

static void check(fv_handle h, fv_status s, const char *call) {
  if (s != FV_OK) {
    fprintf(stderr, "decode_client: %s: %s (%s)\n", call, fv_status_string(s), fv_last_error(h));
    exit(1);
  }
}

static void hip_check(hipError_t e, const char *what) {
  if (e != hipSuccess) {
    fprintf(stderr, "decode_client: %s: %s\n", what, hipGetErrorString(e));
    exit(1);
  }
}

static float *read_floats(const char *dir, const char *name, size_t n) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE *f = fopen(path, "rb");
  if (!f) die(path);
  float *p = (float *)malloc(n * sizeof(float));
  if (!p || fread(p, sizeof(float), n, f) != n) die(path);
  fclose(f);
  return p;
}

static void write_floats(const char *dir, const char *name, const float *p, size_t n) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE *f = fopen(path, "wb");
  if (!f || fwrite(p, sizeof(float), n, f) != n) die(path);
  fclose(f);
}

static float *to_device(const float *host, size_t n) {
  void *d = NULL;
  hip_check(hipMalloc(&d, n * sizeof(float)), "hipMalloc");
  hip_check(hipMemcpy(d, host, n * sizeof(float), hipMemcpyHostToDevice), "hipMemcpy");
  return (float *)d;
}

static float *to_host(const float *dev, size_t n) {
  float *p = (float *)malloc(n * sizeof(float));
  if (!p) die("malloc");
  hip_check(hipMemcpy(p, dev, n * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy");
  return p;
}

int main(int argc, char **argv) {
  if (argc != 12) die("usage: decode_client DIR L W Hq Hkv dh F A C K P");
  const char *dir = argv[1];
  fv_cfg cfg;
  cfg.n_layers = atoi(argv[2]);
  cfg.width = atoi(argv[3]);
  cfg.n_q_heads = atoi(argv[4]);
  cfg.n_kv_heads = atoi(argv[5]);
  cfg.head_dim = atoi(argv[6]);
  cfg.mlp_dim = atoi(argv[7]);
  cfg.action_dim = atoi(argv[8]);
  cfg.chunk_len = atoi(argv[9]);
  cfg.n_chunks = atoi(argv[10]);
  cfg.max_prefix = atoi(argv[11]);
  cfg.max_batch = 1;
  cfg.dtype = FV_FP32;
  cfg.mlp_gated = 1;
  cfg.rms_eps = 1e-6f;
  cfg.rope_theta = 10000.0f;
  cfg.noise_seed = 0;
  const int L = cfg.n_layers, W = cfg.width, qd = cfg.n_q_heads * cfg.head_dim;
  const int kd = cfg.n_kv_heads * cfg.head_dim, F = cfg.mlp_dim, A = cfg.action_dim;
  const int C = cfg.chunk_len, K = cfg.n_chunks, P = cfg.max_prefix;

  /* the weights, in declaration order, each a view into one host array */
  size_t total = (size_t)A * W + W + 2 * ((size_t)W * W + W) + (2 * (size_t)L + 1) * (3 * (size_t)W * W + 3 * (size_t)W) +
                 (size_t)L * ((size_t)W * qd + 2 * (size_t)W * kd + (size_t)qd * W + 2 * (size_t)W * F + (size_t)F * W) +
                 (size_t)W * A + A;
  float *all = read_floats(dir, "weights.bin", total);
  const float **mods = (const float **)malloc((2 * L + 1) * 2 * sizeof(float *));
  const float **lay = (const float **)malloc((size_t)L * 7 * sizeof(float *));
  if (!mods || !lay) die("malloc");
  float *p = all;
  fv_weights w;
  w.w_in = p; p += (size_t)A * W;
  w.b_in = p; p += W;
  w.w_t1 = p; p += (size_t)W * W;
  w.b_t1 = p; p += W;
  w.w_t2 = p; p += (size_t)W * W;
  w.b_t2 = p; p += W;
  for (int n = 0; n < 2 * L + 1; ++n) { mods[n] = p; p += 3 * (size_t)W * W; }
  for (int n = 0; n < 2 * L + 1; ++n) { mods[2 * L + 1 + n] = p; p += 3 * (size_t)W; }
  w.w_mod = mods;
  w.b_mod = mods + 2 * L + 1;
  const size_t sizes[7] = {(size_t)W * qd, (size_t)W * kd, (size_t)W * kd, (size_t)qd * W,
                           (size_t)W * F, (size_t)W * F, (size_t)F * W};
  for (int m = 0; m < 7; ++m)
    for (int l = 0; l < L; ++l) { lay[m * L + l] = p; p += sizes[m]; }
  w.wq = lay; w.wk = lay + L; w.wv = lay + 2 * L; w.wo = lay + 3 * L;
  w.wg = lay + 4 * L; w.wu = lay + 5 * L; w.wd = lay + 6 * L;
  w.w_out = p; p += (size_t)W * A;
  w.b_out = p; p += A;
  if ((size_t)(p - all) != total) die("weight layout");

  fv_handle h = NULL;
  check(NULL, fv_create(&w, &cfg, &h), "fv_create");
  free(all);

  const size_t npre = (size_t)L * P * kd, nbuf = (size_t)K * C * A;
  float *hk = read_floats(dir, "prefix_k.bin", npre), *hv = read_floats(dir, "prefix_v.bin", npre);
  float *hx = read_floats(dir, "buffer.bin", nbuf), *ht = read_floats(dir, "t.bin", (size_t)K);
  float *dk = to_device(hk, npre), *dv = to_device(hv, npre);
  float *dx = to_device(hx, nbuf), *dt = to_device(ht, (size_t)K);
  float *dvel = to_device(hx, nbuf), *dout = to_device(hx, (size_t)C * A);
  const int32_t len = P;
  check(h, fv_set_prefix(h, dk, dv, &len, 1, P, NULL), "fv_set_prefix");
  /* an invalid call leaves the handle usable */
  if (fv_decode_step(h, NULL, dt, dout, NULL) != FV_ERR_INVALID_ARG) die("NULL buffer accepted");
  check(h, fv_velocity(h, dx, dt, dvel, NULL), "fv_velocity");
  check(h, fv_decode_step(h, dx, dt, dout, NULL), "fv_decode_step");
  hip_check(hipDeviceSynchronize(), "hipDeviceSynchronize");

  float *v = to_host(dvel, nbuf), *out = to_host(dout, (size_t)C * A), *after = to_host(dx, nbuf);
  write_floats(dir, "v.bin", v, nbuf);
  write_floats(dir, "out.bin", out, (size_t)C * A);
  write_floats(dir, "buffer_after.bin", after, nbuf);
  uint64_t seed = 0, step = 0;
  check(h, fv_get_noise_state(h, &seed, &step), "fv_get_noise_state");
  check(h, fv_destroy(h), "fv_destroy");
  printf("decode_client: ok (noise step %llu)\n", (unsigned long long)step);
  return 0;
}
