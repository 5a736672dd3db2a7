/*
 * CPU oracle for candidate scoring -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg use
 * this file.  It shares no code with the GPU library: it walks the general
 * child-pointer trees directly, one candidate and one tree at a time, and
 * selects by a full sort.
 *
 * What it computes (ML2Tuner, Section 2):
 *   - model V predicts whether a configuration is valid; the explorer never
 *     passes on a configuration V rejects ("ML Model V");
 *   - model P predicts performance from the same features; the explorer keeps
 *     the configurations with the highest predicted performance among those V
 *     accepts, until (alpha+1)*N are held ("ML Model V", "Hidden Feature
 *     Extractor & ML Model A").  On a fixed pool this is the top-k by P among
 *     the V-accepted candidates with k = (alpha+1)*N;
 *   - model A re-ranks the configurations held, using the hidden features as
 *     well, and keeps the N it predicts best ("Hidden Feature Extractor & ML
 *     Model A"): ml2o_rerank;
 *   - the models are XGBoost tree ensembles (Section 3 "Experimental Setup";
 *     Table 3): V uses the binary hinge objective, whose class decision is 1
 *     exactly when the raw margin is positive; P uses squared-error
 *     regression, whose prediction is the raw margin.
 *
 * Readings taken where the paper is silent:
 *   - a split sends x LEFT iff x[feature] < threshold (XGBoost's rule), so a
 *     tie goes right; a missing (NaN) feature takes the node's default
 *     direction, left where default_left is set, right otherwise (XGBoost's
 *     missing-value rule; without default_left every NaN goes right);
 *   - the margin is base_score + leaf_0 + leaf_1 + ... summed in float32, left
 *     to right in tree-index order, round-to-nearest-even, no fused operations,
 *     subnormals kept;
 *   - valid  <=> margin > 0 (strict);
 *   - invalid candidates get score -inf;
 *   - top-k: included candidates (valid and score not NaN) ordered by score
 *     descending, then index ascending (lower index wins ties, -0 == +0);
 *     min(k, #included) entries, unused slots get index -1 and score -inf.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t num_trees;
  int32_t num_features;
  float base_score;
  const int64_t *offsets;   /* [num_trees + 1] */
  const int32_t *left;      /* tree-local child ids, -1 on both for a leaf */
  const int32_t *right;
  const int32_t *feature;
  const float *threshold;
  const float *value;       /* leaf values */
  const uint8_t *default_left; /* NULL, or nonzero: a NaN feature goes left */
} ml2o_ensemble;

/* Leaf value tree t assigns to the feature vector x.  Returns NaN if the tree
 * is malformed (a walk longer than the tree has nodes). */
float ml2o_tree_leaf(const ml2o_ensemble *e, int32_t t, const float *x) {
  const int64_t base = e->offsets[t];
  const int64_t size = e->offsets[t + 1] - base;
  int64_t node = 0;
  for (int64_t steps = 0; steps <= size; ++steps) {
    int32_t l = e->left[base + node];
    int32_t r = e->right[base + node];
    if (l < 0 && r < 0) return e->value[base + node];
    float xv = x[e->feature[base + node]];
    if (isnan(xv))
      node = (e->default_left && e->default_left[base + node]) ? l : r;
    else
      node = (xv < e->threshold[base + node]) ? l : r;
  }
  return NAN;
}

/* Per-tree leaf values for one candidate (for tests). */
void ml2o_leaves(const ml2o_ensemble *e, const float *x, float *out) {
  for (int32_t t = 0; t < e->num_trees; ++t) out[t] = ml2o_tree_leaf(e, t, x);
}

/* The raw margin: base + leaf_0 + ... + leaf_{T-1}, float32 left fold. */
float ml2o_margin(const ml2o_ensemble *e, const float *x) {
  float m = e->base_score;
  for (int32_t t = 0; t < e->num_trees; ++t) {
    float leaf = ml2o_tree_leaf(e, t, x);
    m = m + leaf;
  }
  return m;
}

/* ---- serial bodies over a candidate range --------------------------------- */

static void validity_range(const ml2o_ensemble *v, const float *X, int64_t lo, int64_t hi,
                           int64_t ld, uint8_t *valid, float *margin) {
  for (int64_t i = lo; i < hi; ++i) {
    float m = ml2o_margin(v, X + i * ld);
    valid[i] = (m > 0.0f) ? 1 : 0;
    if (margin) margin[i] = m;
  }
}

static void perf_range(const ml2o_ensemble *p, const float *X, int64_t lo, int64_t hi,
                       int64_t ld, const uint8_t *valid, float *score) {
  for (int64_t i = lo; i < hi; ++i) {
    if (valid && !valid[i])
      score[i] = -INFINITY;
    else
      score[i] = ml2o_margin(p, X + i * ld);
  }
}

/* ---- the same bodies over contiguous ranges on nthreads threads ---------- */

typedef struct {
  int kind;
  const ml2o_ensemble *e;
  const float *X;
  int64_t lo, hi, ld;
  const uint8_t *valid_in;
  uint8_t *valid_out;
  float *out;
} job;

static void *worker(void *p) {
  job *j = (job *)p;
  if (j->kind == 0)
    validity_range(j->e, j->X, j->lo, j->hi, j->ld, j->valid_out, j->out);
  else
    perf_range(j->e, j->X, j->lo, j->hi, j->ld, j->valid_in, j->out);
  return NULL;
}

static void run(int kind, const ml2o_ensemble *e, const float *X, int64_t n, int64_t ld,
                const uint8_t *valid_in, uint8_t *valid_out, float *out, int32_t nthreads) {
  if (n <= 0) return;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if ((int64_t)nthreads > n) nthreads = (int32_t)n;
  pthread_t th[256];
  job jobs[256];
  for (int32_t t = 0; t < nthreads; ++t) {
    jobs[t].kind = kind;
    jobs[t].e = e;
    jobs[t].X = X;
    jobs[t].lo = n * t / nthreads;
    jobs[t].hi = n * (t + 1) / nthreads;
    jobs[t].ld = ld;
    jobs[t].valid_in = valid_in;
    jobs[t].valid_out = valid_out;
    jobs[t].out = out;
  }
  for (int32_t t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, worker, &jobs[t]);
  worker(&jobs[0]);
  for (int32_t t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
}

/* valid[i] = (margin_i > 0); margin may be NULL. */
void ml2o_validity(const ml2o_ensemble *v, const float *X, int64_t n, int64_t ld,
                   uint8_t *valid, float *margin, int32_t nthreads) {
  run(0, v, X, n, ld, NULL, valid, margin, nthreads);
}

/* score[i] = margin_i under p, or -inf where valid[i] == 0 (valid may be NULL). */
void ml2o_perf(const ml2o_ensemble *p, const float *X, int64_t n, int64_t ld,
               const uint8_t *valid, float *score, int32_t nthreads) {
  run(1, p, X, n, ld, valid, NULL, score, nthreads);
}

/* ---- selection ------------------------------------------------------------ */

typedef struct {
  float s;
  int64_t i;
} pair;

static int by_score_then_index(const void *a, const void *b) {
  const pair *x = (const pair *)a, *y = (const pair *)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->i < y->i) ? -1 : (x->i > y->i) ? 1 : 0;
}

/*
 * Top-k of the included candidates (valid[i] != 0 or valid == NULL, and
 * score not NaN) by (score desc, index asc).  Writes min(k, #included) entries
 * to idx/out_score, pads the rest of the k slots with -1 / -inf, and returns
 * the number written.  Returns -1 on allocation failure.
 */
int64_t ml2o_topk(const uint8_t *valid, const float *score, int64_t n, int64_t k,
                  int32_t *idx, float *out_score) {
  int64_t m = 0;
  pair *all = (pair *)malloc((size_t)(n > 0 ? n : 1) * sizeof(pair));
  if (!all) return -1;
  for (int64_t i = 0; i < n; ++i) {
    if (valid && !valid[i]) continue;
    if (isnan(score[i])) continue;
    all[m].s = score[i];
    all[m].i = i;
    ++m;
  }
  qsort(all, (size_t)m, sizeof(pair), by_score_then_index);
  int64_t sel = m < k ? m : k;
  for (int64_t j = 0; j < k; ++j) {
    if (j < sel) {
      idx[j] = (int32_t)all[j].i;
      out_score[j] = all[j].s;
    } else {
      idx[j] = -1;
      out_score[j] = -INFINITY;
    }
  }
  free(all);
  return sel;
}

/*
 * Second level, model A (Section 2, "Hidden Feature Extractor & ML Model A"):
 * of the configurations the explorer holds, the ones model A -- which also
 * sees the hidden features -- predicts to perform best are kept.
 * rows[0..m) list pool rows of X (n rows, stride ld).  Entry i with
 * 0 <= rows[i] < n gets row_scores[i] = margin under a; any other entry gets
 * -inf and is skipped.  The scored entries are ordered by (score desc, row
 * asc; -0 == +0), a row listed twice counting twice, and the first
 * min(keep, #scored) are written with the row and that entry's score as
 * computed (sign of zero included); the other keep slots get -1 / -inf.
 * Returns the number written, -1 on allocation failure.
 */
int64_t ml2o_rerank(const ml2o_ensemble *a, const float *X, int64_t n, int64_t ld,
                    const int32_t *rows, int64_t m, int64_t keep, float *row_scores,
                    int32_t *idx, float *out_score) {
  pair *all = (pair *)malloc((size_t)(m > 0 ? m : 1) * sizeof(pair));
  if (!all) return -1;
  int64_t c = 0;
  for (int64_t i = 0; i < m; ++i) {
    const int32_t r = rows[i];
    if (r < 0 || (int64_t)r >= n) {
      row_scores[i] = -INFINITY;
      continue;
    }
    const float s = ml2o_margin(a, X + (int64_t)r * ld);
    row_scores[i] = s;
    if (isnan(s)) continue;
    all[c].s = s;
    all[c].i = r;
    ++c;
  }
  qsort(all, (size_t)c, sizeof(pair), by_score_then_index);
  const int64_t sel = c < keep ? c : keep;
  for (int64_t j = 0; j < keep; ++j) {
    if (j < sel) {
      idx[j] = (int32_t)all[j].i;
      out_score[j] = all[j].s;
    } else {
      idx[j] = -1;
      out_score[j] = -INFINITY;
    }
  }
  free(all);
  return sel;
}
