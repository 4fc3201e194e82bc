/*
 * Drives every entry point of the CPU oracle on small inputs, including the
 * edge cases (empty batch, k = m, every expert selected, a kept set of k,
 * masks, exactly k eligible experts, rejected arguments), with every buffer
 * a heap allocation of its exact size.  Built with AddressSanitizer and
 * UndefinedBehaviorSanitizer by tests/test_oracle_asan.py: a read or write
 * past any buffer, a use of uninitialised heap through an index, or an
 * integer overflow ends the run with a report.  Exit status 0 means every
 * call behaved and returned what it should.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "swo.h"

static uint64_t g_state = 0x9E3779B97F4A7C15ull;

static uint64_t next_u64(void) {
  /* splitmix64 (Steele, Lea and Flood, OOPSLA 2014): test data only */
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static float uniform_pm1(void) { return (float)((next_u64() >> 40) * (1.0 / 16777216.0)) * 2.0f - 1.0f; }

static uint16_t bf16_of(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

static void* xmalloc(size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p) {
    fprintf(stderr, "out of memory\n");
    exit(2);
  }
  return p;
}

static int failures = 0;
#define EXPECT(cond)                                                    \
  do {                                                                  \
    if (!(cond)) {                                                      \
      fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      failures++;                                                       \
    }                                                                   \
  } while (0)

/* one layer through prune, route, dispatch, forward (fp32 and fp64), the
 * shared expert and the routing mass, on exactly sized buffers */
static void run_case(int H, int I, int m, int k, int T, int n_keep, int use_mask, int use_bias) {
  size_t n13 = (size_t)m * 2 * I * H, n2 = (size_t)m * H * I;
  uint16_t* x = xmalloc((size_t)T * H * 2);
  uint16_t* w13 = xmalloc(n13 * 2);
  uint16_t* w2 = xmalloc(n2 * 2);
  float* wr = xmalloc((size_t)m * H * 4);
  float* bias = use_bias ? xmalloc((size_t)m * 4) : NULL;
  float* imp = xmalloc((size_t)m * 4);
  for (size_t i = 0; i < (size_t)T * H; i++) x[i] = bf16_of(uniform_pm1());
  for (size_t i = 0; i < n13; i++) w13[i] = bf16_of(0.05f * uniform_pm1());
  for (size_t i = 0; i < n2; i++) w2[i] = bf16_of(0.05f * uniform_pm1());
  for (size_t i = 0; i < (size_t)m * H; i++) wr[i] = 0.05f * uniform_pm1();
  for (int e = 0; e < m; e++) imp[e] = uniform_pm1();
  if (bias)
    for (int e = 0; e < m; e++) bias[e] = 0.3f * uniform_pm1();

  int32_t* kept = xmalloc((size_t)n_keep * 4);
  int32_t* remap = xmalloc((size_t)m * 4);
  uint8_t* mask = xmalloc((size_t)m);
  uint16_t* w13c = xmalloc((size_t)n_keep * 2 * I * H * 2);
  uint16_t* w2c = xmalloc((size_t)n_keep * H * I * 2);
  float* wrc = xmalloc((size_t)n_keep * H * 4);
  float* biasc = bias ? xmalloc((size_t)n_keep * 4) : NULL;
  EXPECT(swo_prune_compact(H, I, m, k, imp, n_keep, w13, w2, wr, bias, kept, remap, mask, w13c,
                           w2c, wrc, biasc) == 0);
  /* mask-only mode */
  EXPECT(swo_prune_compact(H, I, m, k, imp, n_keep, NULL, NULL, NULL, NULL, kept, remap, mask,
                           NULL, NULL, NULL, NULL) == 0);

  int32_t* ids = xmalloc((size_t)T * k * 4);
  float* w = xmalloc((size_t)T * k * 4);
  float* gap = xmalloc((size_t)T * 4);
  float* logits = xmalloc((size_t)T * m * 4);
  const uint8_t* mk = use_mask ? mask : NULL;
  EXPECT(swo_route(H, m, k, x, T, wr, bias, mk, ids, w, gap, logits) == 0);
  EXPECT(swo_route(H, m, k, x, T, wr, bias, mk, ids, w, NULL, NULL) == 0);
  for (int t = 0; t < T; t++) {
    float s = 0.0f;
    for (int j = 0; j < k; j++) {
      EXPECT(ids[t * k + j] >= 0 && ids[t * k + j] < m);
      if (mk) EXPECT(mk[ids[t * k + j]] == 1);
      s += w[t * k + j];
    }
    EXPECT(fabsf(s - 1.0f) < 1e-5f);
    int n_elig = mk ? n_keep : m;
    if (n_elig == k) EXPECT(isinf(gap[t]) && gap[t] > 0);
  }

  int32_t* counts = xmalloc((size_t)m * 4);
  int32_t* offsets = xmalloc((size_t)(m + 1) * 4);
  int32_t* perm = xmalloc((size_t)T * k * 4);
  int32_t* active = xmalloc((size_t)m * 4);
  int32_t na = -5;
  EXPECT(swo_dispatch(m, k, ids, T, counts, offsets, perm, active, &na) == 0);
  EXPECT(offsets[m] == T * k);
  EXPECT(na >= 0 && na <= m);

  float* out = xmalloc((size_t)T * H * 4);
  double* out64 = xmalloc((size_t)T * H * 8);
  EXPECT(swo_forward(H, I, m, k, x, T, w13, w2, ids, w, out) == 0);
  EXPECT(swo_forward_f64(H, I, m, k, x, T, w13, w2, ids, w, out64) == 0);
  for (size_t i = 0; i < (size_t)T * H; i++) EXPECT(fabs((double)out[i] - out64[i]) < 1e-3);

  /* the shared expert: one expert of width I behind a sigmoid gate */
  float* gate_w = xmalloc((size_t)H * 4);
  for (int h = 0; h < H; h++) gate_w[h] = 0.05f * uniform_pm1();
  EXPECT(swo_shared_expert(H, I, x, T, w13, w2, gate_w, out) == 0);

  float* ms = xmalloc((size_t)m * 4);
  float* mt = xmalloc((size_t)m * 4);
  memset(ms, 0, (size_t)m * 4);
  memset(mt, 0, (size_t)m * 4);
  EXPECT(swo_routing_mass(H, m, k, x, T, wr, bias, mk, ms, mt) == 0);
  EXPECT(swo_routing_mass(H, m, k, x, T, wr, bias, mk, NULL, mt) == 0);

  /* rejected arguments: k above the eligible count, an out-of-range id */
  if (T > 0) {
    EXPECT(swo_route(H, m, m + 1, x, T, wr, bias, NULL, ids, w, gap, NULL) != 0);
    int32_t saved = ids[0];
    ids[0] = m;
    EXPECT(swo_forward(H, I, m, k, x, T, w13, w2, ids, w, out) != 0);
    ids[0] = saved;
  }

  free(x); free(w13); free(w2); free(wr); free(bias); free(imp); free(kept); free(remap);
  free(mask); free(w13c); free(w2c); free(wrc); free(biasc); free(ids); free(w); free(gap);
  free(logits); free(counts); free(offsets); free(perm); free(active); free(out); free(out64);
  free(gate_w); free(ms); free(mt);
}

int main(void) {
  /* H, I, m, k, T, n_keep, mask, bias */
  run_case(64, 32, 8, 2, 5, 4, 1, 0);      /* masked, half the pool */
  run_case(72, 8, 5, 5, 3, 5, 0, 1);       /* k = m: every expert selected */
  run_case(40, 24, 6, 3, 4, 3, 1, 1);      /* kept set of exactly k: gap = +inf */
  run_case(256, 16, 33, 8, 9, 17, 1, 1);   /* ragged sizes */
  run_case(32, 8, 4, 1, 1, 1, 1, 0);       /* one token, top-1, one kept expert */
  run_case(48, 16, 7, 2, 0, 4, 1, 1);      /* empty batch */
  if (failures) {
    fprintf(stderr, "%d expectation(s) failed\n", failures);
    return 1;
  }
  printf("oracle asan driver: all cases ok\n");
  return 0;
}
