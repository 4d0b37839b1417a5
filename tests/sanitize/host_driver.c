/* Drives the host code of libpnerf on the CPU, for a build with the host
 * pass under AddressSanitizer and UndefinedBehaviorSanitizer: batch planning
 * over many shapes, argument validation of every entry point, and field
 * creation up to its first device allocation (parameter checks, level
 * tables, fp16 weight conversion and the MFMA weight-tile layout run first;
 * without a GPU the allocation then fails and the partial field is
 * released).  Exits 0 when every call returned the status expected. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pnerf.h"

static int failures = 0;
#define EXPECT(cond)                                                  \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

static uint32_t rng = 12345u;
static uint32_t next(void) {
  rng ^= rng << 13;
  rng ^= rng >> 17;
  rng ^= rng << 5;
  return rng;
}

static void planning(void) {
  for (int trial = 0; trial < 20000; ++trial) {
    int32_t K = 1 + (int32_t)(next() % 70000), P = 1 + (int32_t)(next() % (1 << 22));
    int32_t cap = 1 + (int32_t)(next() % 8192), kr = -1;
    pnerf_status st = pnerf_plan_counted_batch(K, P, cap, &kr);
    if (st == PNERF_OK) {
      EXPECT(kr >= 1 && kr <= K);
      EXPECT((int64_t)kr * P <= ((int64_t)1 << 21));
      EXPECT((int64_t)kr * P * cap < ((int64_t)1 << 31));
    } else {
      EXPECT(st == PNERF_ERR_CAPACITY && kr == 0);
    }
  }
  enum { N = 300 };
  int32_t h[N], cut[N + 1];
  int64_t sums[N];
  for (int trial = 0; trial < 2000; ++trial) {
    int32_t n = 1 + (int32_t)(next() % N), c = 0;
    for (int i = 0; i < n; ++i) h[i] = (int32_t)(next() % 100000);
    int64_t capacity = 1 + (int64_t)(next() % 300000), goal = 1 + (int64_t)(next() % 300000);
    pnerf_status st = pnerf_plan_chunks(h, n, capacity, goal, cut, sums, &c);
    if (st == PNERF_OK) {
      EXPECT(c >= 1 && c <= n && cut[0] == 0 && cut[c] == n);
      for (int i = 0; i < c; ++i) EXPECT(sums[i] <= capacity && cut[i + 1] > cut[i]);
    } else {
      EXPECT(st == PNERF_ERR_CAPACITY);
    }
  }
  EXPECT(pnerf_plan_chunks(NULL, 3, 10, 10, cut, sums, &(int32_t){0}) == PNERF_ERR_INVALID_ARG);
}

static void validation(void) {
  pnerf_adam_params ap = {5e-3f, 3e-3f, 0.9f, 0.999f, 1e-8f, 0.33f, 256, 0, 0, 0};
  EXPECT(pnerf_step_momentum(0, NULL, NULL, NULL, 0.1f, 0.9f, NULL) == PNERF_ERR_INVALID_ARG);
  EXPECT(pnerf_step_adam(4, NULL, NULL, NULL, 0, &ap, NULL) == PNERF_ERR_INVALID_ARG);
  ap.beta1 = 1.0f;
  EXPECT(pnerf_step_adam(4, NULL, NULL, NULL, 0, &ap, NULL) == PNERF_ERR_INVALID_ARG);
  EXPECT(pnerf_resample_hypotheses(70000, NULL, NULL, 6, NULL, 0.5f, 0.1f, 0.1f, 1, 0, NULL) ==
         PNERF_ERR_INVALID_ARG);
  EXPECT(pnerf_resample_hypotheses_noalloc(4, NULL, NULL, 6, NULL, 0.5f, 0.1f, 0.1f, 1, 0,
                                           NULL) == PNERF_ERR_INVALID_ARG);
  EXPECT(pnerf_render_loss_grad(NULL, 4, NULL, 8, NULL, NULL, NULL, NULL, NULL, NULL) ==
         PNERF_ERR_INVALID_ARG);
  EXPECT(pnerf_render(NULL, 4, NULL, 8, NULL, NULL, NULL, NULL) == PNERF_ERR_INVALID_ARG);
  EXPECT(pnerf_field_inspect(NULL, 0, NULL, 0, NULL) == PNERF_ERR_INVALID_ARG);
  EXPECT(strlen(pnerf_last_error()) > 0);
  pnerf_destroy_field(NULL);
}

/* A tiny field in float32 or float16 storage. */
static void creation(int f16, int march_mode, int L, int mlp_precision) {
  const int T = 1 << 10, din = 2 * L;
  int32_t res[16];
  for (int l = 0; l < L; ++l) res[l] = 4 + 3 * l;
  size_t el = f16 ? 2 : 4;
  void* table = calloc((size_t)L * T * 2, el);
  void* w[5];
  size_t wn[5] = {(size_t)din * 64, 64 * 16, 32 * 64, 64 * 64, 64 * 3};
  for (int i = 0; i < 5; ++i) {
    w[i] = malloc(wn[i] * el);
    for (size_t k = 0; k < wn[i]; ++k) {
      if (f16)
        ((uint16_t*)w[i])[k] = (uint16_t)(0x3000u + (next() & 0x3FFu) + ((next() & 1u) << 15));
      else
        ((float*)w[i])[k] = (float)((int)(next() % 2001) - 1000) * 1e-3f;
    }
  }
  pnerf_field_params p;
  memset(&p, 0, sizeof(p));
  p.n_levels = L;
  p.n_features = 2;
  p.log2_table_size = 10;
  p.level_res = res;
  p.dense_coarse_levels = 1;
  p.param_dtype = f16;
  p.table = table;
  p.w_density1 = w[0];
  p.w_density2 = w[1];
  p.w_color1 = w[2];
  p.w_color2 = w[3];
  p.w_color3 = w[4];
  p.density_bias = -1.0f;
  for (int a = 0; a < 3; ++a) {
    p.aabb_min[a] = -0.5f;
    p.aabb_max[a] = 0.5f;
  }
  p.march_mode = march_mode;
  p.n_uniform = 32;
  p.step = 0.01f;
  p.max_samples = 100;
  p.occ_res = march_mode ? 8 : 0;
  p.loss_param = 0.1f;
  p.mlp_precision = mlp_precision;
  pnerf_field* F = NULL;
  pnerf_status st = pnerf_create_field(&p, NULL, &F);
  /* without a GPU the first device allocation fails after the host work */
  EXPECT(st == PNERF_OK || st == PNERF_ERR_DEVICE || st == PNERF_ERR_OUT_OF_MEMORY);
  if (st == PNERF_OK) pnerf_destroy_field(F);
  else EXPECT(F == NULL);
  /* invalid parameters are refused before anything else */
  p.n_levels = 5;
  EXPECT(pnerf_create_field(&p, NULL, &F) == PNERF_ERR_NOT_SUPPORTED);
  p.n_levels = L;
  p.loss_type = 9;
  EXPECT(pnerf_create_field(&p, NULL, &F) == PNERF_ERR_INVALID_ARG);
  p.loss_type = 0;
  p.backward = 3;
  EXPECT(pnerf_create_field(&p, NULL, &F) == PNERF_ERR_INVALID_ARG);
  p.backward = 0;
  p.mlp_precision = 2;
  EXPECT(pnerf_create_field(&p, NULL, &F) == PNERF_ERR_INVALID_ARG);
  p.mlp_precision = mlp_precision;
  p.step = 1e-9f;
  p.march_mode = 1;
  EXPECT(pnerf_create_field(&p, NULL, &F) == PNERF_ERR_INVALID_ARG);
  free(table);
  for (int i = 0; i < 5; ++i) free(w[i]);
}

int main(void) {
  planning();
  validation();
  for (int L = 4; L <= 16; L += 4) {
    for (int mlp = 0; mlp <= 1; ++mlp) {
      creation(0, 0, L, mlp);
      creation(1, 1, L, mlp);
    }
  }
  if (failures) fprintf(stderr, "%d failures\n", failures);
  printf("host driver done\n");
  return failures ? 1 : 0;
}
