/*
 * Seeded synthetic inputs for candidate scoring: candidate feature matrices
 * and perfect binary tree ensembles in the general (child-pointer) form.
 *
 * This file holds input generation only: no tree walking, no summation,
 * no selection.  Both the GPU path and the CPU oracle take their inputs from
 * here, byte for byte.
 *
 * Stand-ins for the paper's workloads (Section 3 "Experimental Setup",
 * Appendix A.3 and Table 5): visible features are schedule knobs (tile sizes,
 * virtual-thread counts), modelled as log2 knob values uniform on {0..8};
 * hidden compiler features are modelled as lognormal(0,1) values.  Tree
 * ensembles follow the XGBoost gbtree shape of Table 3 (perfect trees of a
 * given depth, breadth-first node order).
 *
 * Random numbers are counter-based: every value is a pure function of
 * (seed, stream, counter), so the output does not depend on the thread count.
 *   hash  : SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014) applied to
 *           a per-(seed, stream) key plus counter * 0x9E3779B97F4A7C15.
 *   u24   : the top 24 bits of a hash.
 *   knob  : floor(9 * u24 / 2^24), an exact integer in {0..8}.
 *   normal: Box-Muller, z = sqrt(-2 ln u1) cos(2 pi u2), in double, with
 *           u1 in (0,1] and u2 in [0,1) from two 53-bit draws.
 *   lognormal: (float) exp(z).
 * Streams: 0 = features, 1 = validity ensemble, 2 = performance ensemble
 * (callers may use others, e.g. 3 for a second-level ensemble).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

uint64_t ml2gen_hash(uint64_t seed, uint64_t stream, uint64_t ctr) {
  uint64_t key = mix64(seed * 0x9E3779B97F4A7C15ULL +
                       stream * 0xD1B54A32D192ED03ULL + 0x632BE59BD9B4E019ULL);
  return mix64(key + ctr * 0x9E3779B97F4A7C15ULL);
}

static inline uint32_t u24(uint64_t h) { return (uint32_t)(h >> 40); }

static inline int32_t knob_of(uint64_t h) {
  return (int32_t)(((uint64_t)u24(h) * 9u) >> 24);
}

static inline int32_t index_of(uint64_t h, int32_t m) {
  return (int32_t)(((uint64_t)u24(h) * (uint64_t)m) >> 24);
}

static double normal_of(uint64_t h1, uint64_t h2) {
  const double two53 = 9007199254740992.0;
  double u1 = ((double)(h1 >> 11) + 1.0) / two53; /* (0, 1] */
  double u2 = (double)(h2 >> 11) / two53;         /* [0, 1) */
  return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
}

/* One feature value: column f < K is a knob, otherwise lognormal. */
static float feature_value(uint64_t seed, uint64_t ctr, int32_t f, int32_t K) {
  if (f < K) return (float)knob_of(ml2gen_hash(seed, 0, 2 * ctr));
  double z = normal_of(ml2gen_hash(seed, 0, 2 * ctr), ml2gen_hash(seed, 0, 2 * ctr + 1));
  return (float)exp(z);
}

typedef struct {
  uint64_t seed;
  const int64_t *rows; /* NULL: rows row0 .. row0+n-1 */
  int64_t row0, lo, hi;
  int32_t F, K;
  int64_t ld;
  float *X;
  uint32_t missing_u24; /* hidden values are NaN with probability missing_u24 / 2^24 */
} feat_job;

#define STREAM_MISSING 4

static void *feat_worker(void *p) {
  feat_job *j = (feat_job *)p;
  for (int64_t r = j->lo; r < j->hi; ++r) {
    int64_t row = j->rows ? j->rows[r] : j->row0 + r;
    float *dst = j->X + r * j->ld;
    for (int32_t f = 0; f < j->F; ++f) {
      const uint64_t ctr = (uint64_t)row * (uint64_t)j->F + (uint64_t)f;
      if (f >= j->K && j->missing_u24 &&
          u24(ml2gen_hash(j->seed, STREAM_MISSING, ctr)) < j->missing_u24)
        dst[f] = NAN;
      else
        dst[f] = feature_value(j->seed, ctr, f, j->K);
    }
  }
  return NULL;
}

/*
 * Write m rows of the N x F feature matrix of `seed` into X (row stride ld
 * floats).  Row r of the output is global row rows[r], or row0 + r when rows
 * is NULL.  Columns F..ld-1 are left untouched.  With missing > 0 each hidden
 * value (column >= K) is NaN -- a missing value -- with that probability
 * (stream 4, one draw per element).
 */
void ml2gen_features(uint64_t seed, const int64_t *rows, int64_t row0, int64_t m,
                     int32_t F, int32_t K, int64_t ld, float *X, int32_t nthreads,
                     double missing) {
  const uint32_t miss = missing <= 0.0 ? 0u
                      : missing >= 1.0 ? (1u << 24)
                                       : (uint32_t)(missing * 16777216.0);
  if (m <= 0) return;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if ((int64_t)nthreads > m) nthreads = (int32_t)m;
  pthread_t th[256];
  feat_job jobs[256];
  for (int32_t t = 0; t < nthreads; ++t) {
    jobs[t].seed = seed;
    jobs[t].rows = rows;
    jobs[t].row0 = row0;
    jobs[t].lo = m * t / nthreads;
    jobs[t].hi = m * (t + 1) / nthreads;
    jobs[t].F = F;
    jobs[t].K = K;
    jobs[t].ld = ld;
    jobs[t].X = X;
    jobs[t].missing_u24 = miss;
  }
  for (int32_t t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, feat_worker, &jobs[t]);
  feat_worker(&jobs[0]);
  for (int32_t t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
}

/*
 * T perfect trees of the given depth (depth split levels: 2^depth - 1
 * internal nodes and 2^depth leaves per tree), in breadth-first order with
 * children 2i+1 and 2i+2, written in the general child-pointer form:
 *   off[T+1]           tree t owns nodes off[t] .. off[t+1]-1 (tree-local ids)
 *   left[], right[]    tree-local child ids, -1 on both for a leaf
 *   feat[], thr[]      split feature (uniform over 0..F-1) and threshold drawn
 *                      from that feature's own distribution (knob or lognormal)
 *   leaf[]             leaf value sigma * N(0,1); 0 on internal nodes
 * Internal nodes of leaves carry feat = -1, thr = 0.
 */
void ml2gen_perfect_trees(uint64_t seed, uint64_t stream, int32_t T, int32_t depth,
                          int32_t F, int32_t K, double leaf_sigma, int64_t *off,
                          int32_t *left, int32_t *right, int32_t *feat, float *thr,
                          float *leaf) {
  const int64_t nodes = ((int64_t)2 << depth) - 1;
  const int64_t internal = ((int64_t)1 << depth) - 1;
  for (int32_t t = 0; t <= T; ++t) off[t] = (int64_t)t * nodes;
  for (int32_t t = 0; t < T; ++t) {
    for (int64_t i = 0; i < nodes; ++i) {
      const int64_t g = (int64_t)t * nodes + i;
      const uint64_t c = ((uint64_t)t << 32) + (uint64_t)i;
      if (i < internal) {
        int32_t f = index_of(ml2gen_hash(seed, stream, 4 * c), F);
        float th;
        if (f < K)
          th = (float)knob_of(ml2gen_hash(seed, stream, 4 * c + 1));
        else
          th = (float)exp(normal_of(ml2gen_hash(seed, stream, 4 * c + 2),
                                    ml2gen_hash(seed, stream, 4 * c + 3)));
        left[g] = (int32_t)(2 * i + 1);
        right[g] = (int32_t)(2 * i + 2);
        feat[g] = f;
        thr[g] = th;
        leaf[g] = 0.0f;
      } else {
        left[g] = -1;
        right[g] = -1;
        feat[g] = -1;
        thr[g] = 0.0f;
        leaf[g] = (float)(leaf_sigma * normal_of(ml2gen_hash(seed, stream, 4 * c),
                                                  ml2gen_hash(seed, stream, 4 * c + 1)));
      }
    }
  }
}

/*
 * T ragged trees grown breadth-first (the shape of XGBoost trees trained to a
 * maximum depth): the root splits, a node at depth d in 1..max_depth-1 splits
 * with probability p_split * decay^(d-1), a node at max_depth is a leaf, and a
 * split that would take the tree past max_nodes nodes becomes a leaf.  Node
 * ids are breadth-first (the children of a node are adjacent, left first).
 * Split features are uniform over 0..F-1 with thresholds from the feature's
 * own distribution, as for perfect trees; default_left is 1 with probability
 * p_left on internal nodes.  Per node i of tree t the draws use counters
 * 8*c + {0: feature, 1: knob threshold, 2-3: lognormal threshold, 4: split,
 * 5: default direction, 6-7: leaf}, c = (t << 32) + i.  Arrays hold room
 * for T * max_nodes nodes; returns the number of nodes written.
 */
int64_t ml2gen_ragged_trees(uint64_t seed, uint64_t stream, int32_t T, int32_t max_depth,
                            int32_t max_nodes, double p_split, double decay, double p_left,
                            int32_t F, int32_t K, double leaf_sigma, int64_t *off,
                            int32_t *left, int32_t *right, int32_t *feat, float *thr,
                            float *leaf, uint8_t *dleft) {
  int32_t *depth = (int32_t *)malloc((size_t)(max_nodes > 0 ? max_nodes : 1) * sizeof(int32_t));
  if (!depth) return -1;
  int64_t g0 = 0;
  for (int32_t t = 0; t < T; ++t) {
    off[t] = g0;
    int32_t count = 1;
    depth[0] = 0;
    for (int32_t i = 0; i < count; ++i) {
      const int64_t g = g0 + i;
      const uint64_t c = ((uint64_t)t << 32) + (uint64_t)i;
      const int32_t d = depth[i];
      int split = 0;
      if (d == 0) {
        split = max_depth > 0;
      } else if (d < max_depth) {
        const double p = p_split * pow(decay, (double)(d - 1));
        split = (double)u24(ml2gen_hash(seed, stream, 8 * c + 4)) < p * 16777216.0;
      }
      if (split && count + 2 > max_nodes) split = 0;
      if (split) {
        const int32_t f = index_of(ml2gen_hash(seed, stream, 8 * c), F);
        float th;
        if (f < K)
          th = (float)knob_of(ml2gen_hash(seed, stream, 8 * c + 1));
        else
          th = (float)exp(normal_of(ml2gen_hash(seed, stream, 8 * c + 2),
                                    ml2gen_hash(seed, stream, 8 * c + 3)));
        left[g] = count;
        right[g] = count + 1;
        feat[g] = f;
        thr[g] = th;
        leaf[g] = 0.0f;
        dleft[g] = (double)u24(ml2gen_hash(seed, stream, 8 * c + 5)) < p_left * 16777216.0;
        depth[count] = d + 1;
        depth[count + 1] = d + 1;
        count += 2;
      } else {
        left[g] = -1;
        right[g] = -1;
        feat[g] = -1;
        thr[g] = 0.0f;
        dleft[g] = 0;
        leaf[g] = (float)(leaf_sigma * normal_of(ml2gen_hash(seed, stream, 8 * c + 6),
                                                  ml2gen_hash(seed, stream, 8 * c + 7)));
      }
    }
    g0 += count;
  }
  off[T] = g0;
  free(depth);
  return g0;
}
