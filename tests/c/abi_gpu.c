/* The sensitivity profile driven from plain C: device memory from the HIP
 * runtime (hipMalloc / hipMemcpy), no Python or torch.  Reads a model, a batch
 * and the profile's arguments from a binary file written by
 * tests/test_gpu_c_abi.py, runs rk_sensitivity_profile and rk_layer_budgets, and
 * prints s and the budgets for the test to compare with the ctypes binding.
 *
 * File layout (little-endian): int32 n_layers, d_model, n_heads, n_kv_heads,
 * head_dim, d_ff, vocab, dtype, n_seqs, n_alpha; float32 rope_theta, rms_eps;
 * int64 offsets[n_seqs + 1]; float32 alphas[n_alpha]; then the weights as
 * stored on the device (model dtype for matrices, fp32 for norms): tok_emb,
 * per layer w_qkv, w_o, w_gate_up, w_down, attn_norm, mlp_norm, then
 * final_norm, lm_head; then int32 tokens[offsets[n_seqs]]. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "rk.h"

static FILE* in;

static void rd(void* p, size_t n) {
  if (fread(p, 1, n, in) != n) { fprintf(stderr, "short read\n"); exit(2); }
}

static void* dev(size_t n) {   /* read n bytes into a new device buffer */
  void* h = malloc(n);
  void* d = NULL;
  if (!h) exit(3);
  rd(h, n);
  if (hipMalloc(&d, n) != hipSuccess || hipMemcpy(d, h, n, hipMemcpyHostToDevice) != hipSuccess) {
    fprintf(stderr, "hip copy failed\n");
    exit(4);
  }
  free(h);
  return d;
}

int main(int argc, char** argv) {
  if (argc != 2 || !(in = fopen(argv[1], "rb"))) { fprintf(stderr, "usage: abi_gpu FILE\n"); return 1; }
  int32_t hdr[10];
  float fl[2];
  rd(hdr, sizeof hdr);
  rd(fl, sizeof fl);
  rk_model_config cfg = {hdr[0], hdr[1], hdr[2], hdr[3], hdr[4], hdr[5], hdr[6], fl[0], fl[1], (rk_dtype)hdr[7]};
  const int L = cfg.n_layers, n_seqs = hdr[8], n_alpha = hdr[9];
  const size_t a = cfg.dtype == RK_BF16 ? 2 : 4, d = (size_t)cfg.d_model;
  const size_t qkv = (size_t)(cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim, att = (size_t)cfg.n_heads * cfg.head_dim;
  int64_t* offs = malloc(sizeof(int64_t) * (n_seqs + 1));
  float* alphas = malloc(sizeof(float) * n_alpha);
  const void** wq = malloc(sizeof(void*) * L);
  const void** wo = malloc(sizeof(void*) * L);
  const void** wg = malloc(sizeof(void*) * L);
  const void** wd = malloc(sizeof(void*) * L);
  const float** an = malloc(sizeof(float*) * L);
  const float** mn = malloc(sizeof(float*) * L);
  int32_t* layers = malloc(sizeof(int32_t) * L);
  if (!offs || !alphas || !wq || !wo || !wg || !wd || !an || !mn || !layers) return 3;
  rd(offs, sizeof(int64_t) * (n_seqs + 1));
  rd(alphas, sizeof(float) * n_alpha);
  const void* emb = dev((size_t)cfg.vocab * d * a);
  for (int l = 0; l < L; ++l) {
    wq[l] = dev(qkv * d * a);
    wo[l] = dev(d * att * a);
    wg[l] = dev(2 * (size_t)cfg.d_ff * d * a);
    wd[l] = dev(d * (size_t)cfg.d_ff * a);
    an[l] = dev(d * 4);
    mn[l] = dev(d * 4);
    layers[l] = l;
  }
  const float* fn = dev(d * 4);
  const void* lm = dev((size_t)cfg.vocab * d * a);
  const int32_t* tokens = dev((size_t)offs[n_seqs] * 4);
  fclose(in);

  rk_model_weights w = {emb, wq, wo, wg, wd, an, mn, fn, lm};
  rk_model* m = NULL;
  if (rk_model_create(&cfg, &w, &m) != RK_OK) { fprintf(stderr, "%s\n", rk_last_error()); return 5; }
  const rk_batch batch = {tokens, offs, n_seqs, 0};
  const int64_t rows = offs[n_seqs];
  const size_t ws_bytes = rk_workspace_size(m, rows, L, RK_WS_CLEAN_STATE);
  void *ws = NULL, *s_dev = NULL;
  if (hipMalloc(&ws, ws_bytes) != hipSuccess || hipMalloc(&s_dev, sizeof(float) * n_alpha * L) != hipSuccess) return 4;
  const rk_perturb_params p = {2, 0, 0, 0, 0};
  rk_status st = rk_sensitivity_profile(m, &batch, layers, L, alphas, n_alpha, &p, rows, L, (float*)s_dev, NULL, ws,
                                        ws_bytes, NULL);
  if (st != RK_OK) { fprintf(stderr, "profile: %s\n", rk_last_error()); return 6; }
  float* s = malloc(sizeof(float) * n_alpha * L);
  double* sd = malloc(sizeof(double) * L);
  int64_t* b = malloc(sizeof(int64_t) * L);
  if (!s || !sd || !b) return 3;
  if (hipMemcpy(s, s_dev, sizeof(float) * n_alpha * L, hipMemcpyDeviceToHost) != hipSuccess) return 4;
  for (int k = 0; k < n_alpha; ++k) {
    printf("s%d", k);
    for (int l = 0; l < L; ++l) printf(" %.9g", s[k * L + l]);
    printf("\n");
  }
  for (int l = 0; l < L; ++l) sd[l] = s[(n_alpha - 1) * L + l];
  st = rk_layer_budgets(sd, L, 100 * (int64_t)L, 2.0, 0.0, 0.0, RK_ROUND_LARGEST_REMAINDER, NULL, b);
  printf("budgets %d", (int)st);
  for (int l = 0; l < L; ++l) printf(" %lld", (long long)b[l]);
  printf("\n");
  rk_model_destroy(m);
  return 0;
}
