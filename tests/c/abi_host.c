/* Host-side use of the C ABI from plain C99 (no GPU): the public structs' layout,
 * the budget mapping, Spearman's rho, the compressed-cache layout, model handles
 * and size queries, and an error path.  Prints "key value ..." lines that
 * tests/test_c_abi.py compares with the same calls made through ctypes. */
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>

#include "rk.h"

#define LAYOUT(T, f) printf("offset " #T "." #f " %zu\n", offsetof(T, f))

int main(void) {
  printf("sizeof rk_model_config %zu\n", sizeof(rk_model_config));
  printf("sizeof rk_model_weights %zu\n", sizeof(rk_model_weights));
  printf("sizeof rk_batch %zu\n", sizeof(rk_batch));
  printf("sizeof rk_perturb_params %zu\n", sizeof(rk_perturb_params));
  printf("sizeof rk_snapkv_params %zu\n", sizeof(rk_snapkv_params));
  LAYOUT(rk_model_config, rope_theta);
  LAYOUT(rk_model_config, dtype);
  LAYOUT(rk_model_weights, lm_head);
  LAYOUT(rk_batch, n_seqs);
  LAYOUT(rk_batch, seq_index0);
  LAYOUT(rk_perturb_params, window_start);
  LAYOUT(rk_perturb_params, flags);
  LAYOUT(rk_snapkv_params, pooling);

  /* budget mapping (Algorithm 1, allocation half) */
  const double s[5] = {0.5, 0.1, 0.3, 0.9, 0.3};
  double w[5];
  int64_t b[5];
  rk_status st = rk_layer_budgets(s, 5, 1000, 2.0, 0.0, 0.0, RK_ROUND_LARGEST_REMAINDER, w, b);
  printf("budgets_status %d\n", (int)st);
  printf("budgets");
  for (int i = 0; i < 5; ++i) printf(" %lld", (long long)b[i]);
  printf("\nweights");
  for (int i = 0; i < 5; ++i) printf(" %.17g", w[i]);
  printf("\n");
  st = rk_layer_budgets(s, 5, 1000, 4.0, 1.5, 0.0, RK_ROUND_NEAREST_EVEN, w, b);
  printf("budgets_clip_even %d", (int)st);
  for (int i = 0; i < 5; ++i) printf(" %lld", (long long)b[i]);
  printf("\n");

  /* Spearman's rho */
  const double x[6] = {1, 2, 2, 5, 3, 9}, y[6] = {0.1, 0.4, 0.3, 0.2, 0.9, 0.8};
  double rho = 0.0;
  st = rk_spearman(x, y, 6, &rho);
  printf("spearman %d %.17g\n", (int)st, rho);

  /* compressed-cache layout of three sequences, two layers */
  const int64_t offs[4] = {0, 40, 100, 105};
  rk_batch batch = {NULL, offs, 3, 0};
  const int64_t bud[6] = {10, 50, 70, 0, 3, 8};
  int64_t lay[7];
  const int64_t total = rk_snapkv_layout(&batch, 2, bud, lay);
  printf("layout %lld", (long long)total);
  for (int i = 0; i < 7; ++i) printf(" %lld", (long long)lay[i]);
  printf("\n");

  /* a model handle over placeholder pointers: sizes only, no device work */
  enum { L = 2 };
  static const char dummy[16];
  const void* mats[L] = {dummy, dummy};
  const float* norms[L] = {(const float*)dummy, (const float*)dummy};
  rk_model_config cfg = {L, 256, 4, 2, 64, 512, 1024, 1.0e4f, 1e-5f, RK_BF16};
  rk_model_weights wts = {dummy, mats, mats, mats, mats, norms, norms, (const float*)dummy, dummy};
  rk_model* m = NULL;
  st = rk_model_create(&cfg, &wts, &m);
  printf("create %d\n", (int)st);
  printf("sizes %zu %zu %zu %zu\n", rk_clean_state_size(m, 300), rk_window_state_size(m, 300),
         rk_workspace_size(m, 300, 4, RK_FLAG_CACHED_WINDOW), rk_snapkv_state_size(m, 300, 3, 16));
  rk_model_destroy(m);

  /* an error path: nothing created, a message recorded */
  cfg.head_dim = 96;
  m = NULL;
  st = rk_model_create(&cfg, &wts, &m);
  printf("create_bad %d %d %s\n", (int)st, m == NULL, rk_last_error()[0] ? "message" : "empty");
  return 0;
}
