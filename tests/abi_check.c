/* A C program built against the public headers alone (C99, no C++ and no
 * PyTorch): the headers are plain C, and the library's host-side entry
 * points answer as the headers state.  No call here reaches the device:
 * sizing, argument checks and NULL handles only. */
#include <stdio.h>
#include <string.h>

#include "mar_cache.h"
#include "mar_head.h"
#include "mar_kernels.h"

static int failures = 0;
#define CHECK(cond)                                                 \
  do {                                                              \
    if (!(cond)) {                                                  \
      printf("FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond);         \
      ++failures;                                                   \
    }                                                               \
  } while (0)

int main(void) {
  mar_dims d;
  mar_cache* h = (mar_cache*)&d; /* any non-NULL value: init must reset it */
  size_t n, cache;

  memset(&d, 0, sizeof d);
  d.n_layers = 32;
  d.d_model = 1024;
  d.n_heads = 16;
  d.d_mlp = 4096;
  d.seq_len = 320;
  d.max_slots = 128;
  d.full_prefix = 3;
  d.dtype = MAR_BF16;
  d.ln_eps = 1e-6f;

  /* the workspace holds at least the key/value caches of blocks P..L-1 */
  n = mar_workspace_bytes(&d);
  cache = (size_t)(32 - 3) * 2 * 128 * 320 * 1024 * 2;
  CHECK(n > cache);
  CHECK(n % 256 == 0);
  /* the feature score source adds its fp32 reference rows */
  d.score_source = MAR_SCORE_FEATURES;
  CHECK(mar_workspace_bytes(&d) >= n + (size_t)128 * 320 * 1024 * 4);
  d.score_source = 7;
  CHECK(mar_workspace_bytes(&d) == 0);
  CHECK(strstr(mar_last_error(), "score_source") != NULL);
  d.score_source = MAR_SCORE_VALUES;
  d.n_heads = 7; /* d_model not divisible */
  CHECK(mar_workspace_bytes(&d) == 0);
  d.n_heads = 16;
  d.seq_len = 4097;
  CHECK(mar_workspace_bytes(&d) == 0);
  d.seq_len = 320;
  /* 32-bit offsets: MAR-H shapes fit 327 slots, not 330 (the widest
   * product, fc1 on every row of a full step, would reach 2 GiB) */
  d.n_layers = 40;
  d.d_model = 1280;
  d.d_mlp = 5120;
  d.max_slots = 327;
  CHECK(mar_workspace_bytes(&d) > 0);
  d.max_slots = 330;
  CHECK(mar_workspace_bytes(&d) == 0);
  CHECK(strstr(mar_last_error(), "2 GiB") != NULL);
  CHECK(mar_cache_init(&d, NULL, NULL, 0, NULL, &h) == MAR_E_SHAPE);
  d.n_layers = 32;
  d.d_model = 1024;
  d.d_mlp = 4096;
  d.max_slots = 128;

  /* argument checks come before any device work */
  CHECK(mar_cache_init(&d, NULL, NULL, 0, NULL, &h) == MAR_E_ARG);
  CHECK(h == NULL);
  CHECK(mar_cache_init(&d, NULL, NULL, 0, NULL, NULL) == MAR_E_ARG);
  CHECK(mar_step(NULL, NULL, NULL, 0, 1, MAR_FULL, 0, NULL, NULL) == MAR_E_ARG);
  CHECK(mar_cfg_combine(NULL, NULL, NULL, 0, 1, MAR_CFG_STORE, 1.0f, NULL, NULL, NULL) == MAR_E_ARG);
  CHECK(mar_k_select(NULL, 1, 8, 2, NULL, NULL) == MAR_E_ARG);
  CHECK(mar_k_select_most_similar(NULL, 1, 8, 2, NULL, NULL) == MAR_E_ARG);
  CHECK(mar_cache_destroy(NULL) == MAR_OK);
  CHECK(mar_output(NULL) == NULL);
  CHECK(mar_k_gemm_variant(16) == MAR_E_ARG);
  CHECK(mar_k_gemm_variant(-1) == MAR_OK);

  /* the diffusion head: sizing and host-side checks */
  {
    mar_head_dims hd;
    mar_head* hh = (mar_head*)&hd;
    memset(&hd, 0, sizeof hd);
    hd.width = 1280;
    hd.depth = 8;
    hd.cond_dim = 1024;
    hd.token_dim = 16;
    hd.steps = 100;
    hd.train_steps = 1000;
    hd.freq_dim = 256;
    hd.max_rows = 1024;
    hd.dtype = MAR_BF16;
    hd.beta_start = 1e-4f;
    hd.beta_end = 0.02f;
    hd.ln_eps = 1e-6f;
    CHECK(mar_head_workspace_bytes(&hd) > 0);
    hd.dtype = MAR_F32;
    CHECK(mar_head_workspace_bytes(&hd) == 0);
    CHECK(strstr(mar_last_error(), "bf16") != NULL);
    hd.dtype = MAR_BF16;
    hd.max_rows = 16384; /* the modulation rows would pass 32-bit offsets */
    CHECK(mar_head_workspace_bytes(&hd) == 0);
    hd.max_rows = 1024;
    CHECK(mar_head_init(&hd, NULL, NULL, 0, NULL, &hh) == MAR_E_ARG);
    CHECK(hh == NULL);
    CHECK(mar_head_sample(NULL, NULL, NULL, 1, NULL, NULL, 1, NULL, NULL, 1.0f, NULL, NULL, NULL, NULL) ==
          MAR_E_ARG);
    CHECK(mar_head_destroy(NULL) == MAR_OK);
  }

  printf("abi check: %s (%d failures)\n", failures ? "FAILED" : "ok", failures);
  return failures != 0;
}
