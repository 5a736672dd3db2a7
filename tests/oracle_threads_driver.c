/*
 * Driver for the ThreadSanitizer run of the CPU oracle (tests only).
 *
 * Builds a small seeded ensemble and pool in plain C, scores the pool with
 * ml2o_validity / ml2o_perf on 1 thread and on several thread counts that do
 * not divide the pool size, and exits non-zero if any output byte differs.
 * Compiled together with oracle/ml2_oracle.c under -fsanitize=thread, so a
 * data race between the worker threads is reported by the sanitizer.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t num_trees;
  int32_t num_features;
  float base_score;
  const int64_t *offsets;
  const int32_t *left;
  const int32_t *right;
  const int32_t *feature;
  const float *threshold;
  const float *value;
  const uint8_t *default_left;
} ml2o_ensemble;

void ml2o_validity(const ml2o_ensemble *v, const float *X, int64_t n, int64_t ld,
                   uint8_t *valid, float *margin, int32_t nthreads);
void ml2o_perf(const ml2o_ensemble *p, const float *X, int64_t n, int64_t ld,
               const uint8_t *valid, float *score, int32_t nthreads);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) { /* xorshift64*: any fixed sequence will do */
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 0x2545F4914F6CDD1Dull) >> 32);
}

enum { T = 24, D = 4, F = 9, N = 1013 };

int main(void) {
  const int nodes = (2 << D) - 1; /* perfect tree: 2^(D+1) - 1 nodes */
  int64_t off[T + 1];
  int32_t *left = malloc(sizeof(int32_t) * T * nodes), *right = malloc(sizeof(int32_t) * T * nodes);
  int32_t *feat = malloc(sizeof(int32_t) * T * nodes);
  float *thr = malloc(sizeof(float) * T * nodes), *val = malloc(sizeof(float) * T * nodes);
  for (int t = 0; t < T; ++t) {
    off[t] = (int64_t)t * nodes;
    for (int j = 0; j < nodes; ++j) {
      const int g = t * nodes + j;
      const int internal = j < (1 << D) - 1;
      left[g] = internal ? 2 * j + 1 : -1;
      right[g] = internal ? 2 * j + 2 : -1;
      feat[g] = (int32_t)(next_u32() % F);
      thr[g] = (float)(next_u32() % 9);
      val[g] = ((float)(next_u32() % 2001) - 1000.0f) / 512.0f;
    }
  }
  off[T] = (int64_t)T * nodes;
  ml2o_ensemble e = {T, F, 0.25f, off, left, right, feat, thr, val, NULL};
  float *X = malloc(sizeof(float) * N * F);
  for (int i = 0; i < N * F; ++i) X[i] = (float)(next_u32() % 9);
  uint8_t *v1 = malloc(N), *vt = malloc(N);
  float *m1 = malloc(sizeof(float) * N), *mt = malloc(sizeof(float) * N);
  float *s1 = malloc(sizeof(float) * N), *st = malloc(sizeof(float) * N);
  ml2o_validity(&e, X, N, F, v1, m1, 1);
  ml2o_perf(&e, X, N, F, v1, s1, 1);
  const int threads[] = {2, 3, 7, 16, 64};
  for (size_t k = 0; k < sizeof threads / sizeof threads[0]; ++k) {
    memset(vt, 0xAB, N);
    memset(mt, 0xAB, sizeof(float) * N);
    memset(st, 0xAB, sizeof(float) * N);
    ml2o_validity(&e, X, N, F, vt, mt, threads[k]);
    ml2o_perf(&e, X, N, F, vt, st, threads[k]);
    if (memcmp(v1, vt, N) || memcmp(m1, mt, sizeof(float) * N) ||
        memcmp(s1, st, sizeof(float) * N)) {
      fprintf(stderr, "outputs on %d threads differ from 1 thread\n", threads[k]);
      return 1;
    }
  }
  printf("threads ok\n");
  free(left); free(right); free(feat); free(thr); free(val);
  free(X); free(v1); free(vt); free(m1); free(mt); free(s1); free(st);
  return 0;
}
