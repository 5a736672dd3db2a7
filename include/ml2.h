/*
 * ml2.h -- C ABI of the candidate-scoring library (gfx950).
 *
 * The library implements the data-parallel step of ML2Tuner's configuration
 * explorer (Section 2 and Fig. 1): every candidate configuration of a pool is
 * scored by a validity model V and, where V accepts it, by a performance
 * model P; the explorer then keeps the top (alpha+1)*N candidates by
 * predicted performance among those V accepts ("ML Model V"; "Hidden Feature
 * Extractor & ML Model A").  Both models are XGBoost gbtree ensembles
 * (Section 3 "Experimental Setup"; Table 3: V uses the binary hinge
 * objective, P the squared-error regression objective).
 *
 * Conventions shared by every call:
 *   - A split sends a candidate LEFT iff x[feature] < threshold (XGBoost's
 *     rule): a tie goes right.  A NaN feature is a missing value and takes
 *     the node's default direction (XGBoost's missing-value rule): left
 *     where the ensemble's default_left is set, right otherwise.
 *   - A margin is base_score + leaf(tree 0) + leaf(tree 1) + ... computed in
 *     float32 as a left fold in tree-index order, round-to-nearest-even, no
 *     fused operations, subnormals kept.  Results are bit-identical to that
 *     definition, whatever the launch shape.
 *   - Candidate pools are row-major float32 matrices X[n][ld] in DEVICE
 *     memory; row i is candidate i; only columns 0..num_features-1 are read.
 *   - Every pointer argument except desc/out/bytes is a DEVICE pointer owned
 *     by the caller; the library never frees caller memory.
 *   - stream is a hipStream_t passed as void* (NULL = the null stream).  Work
 *     is enqueued asynchronously on it; arguments are validated
 *     synchronously before anything is enqueued, and a call that returns an
 *     error has enqueued nothing.  Faults inside kernels surface at the
 *     caller's next synchronisation of the stream.
 *   - The device is the HIP device current on the calling thread.
 *   - The scoring, selection and re-rank calls allocate nothing and only
 *     enqueue kernels, so they may be captured into a HIP graph on the
 *     stream, once each has run outside the capture on that device (its
 *     first call sets kernel attributes).  Replays read and write the
 *     buffers given at capture.
 *   - Errors are returned as status codes; ml2_last_error() gives a
 *     thread-local description of the last non-OK status.
 */
#ifndef ML2_H
#define ML2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ML2_OK = 0,
  ML2_ERR_INVALID_ARG = 1,   /* malformed descriptor, bad pointer/size/stride */
  ML2_ERR_UNSUPPORTED = 2,   /* valid input beyond this library's limits */
  ML2_ERR_OUT_OF_MEMORY = 3, /* device or host allocation failed */
  ML2_ERR_HIP = 4            /* a HIP runtime call or kernel launch failed */
} ml2_status;

/* Library limits (checked at load / call time, ML2_ERR_UNSUPPORTED beyond). */
#define ML2_MAX_DEPTH 32        /* longest root-to-leaf path, in splits */
#define ML2_MAX_TREE_NODES 3062 /* nodes of one tree in the ragged layout */
#define ML2_MAX_FEATURES 256    /* num_features of an ensemble */
#define ML2_MAX_TOPK 16384      /* k of ml2_filter_topk; m and keep of ml2_rerank */
#define ML2_MAX_STREAM_K 4096   /* k of ml2_stream_explorer_create */

typedef struct ml2_ensemble ml2_ensemble; /* opaque; immutable after load */

/*
 * A tree ensemble in XGBoost's general form (host arrays, read during
 * ml2_load_ensemble only).
 *   num_trees       T >= 1
 *   num_features    F in [1, ML2_MAX_FEATURES]; split features lie in [0, F)
 *   base_score      margin bias, the first term of the fold (finite)
 *   tree_node_offset[T+1]  tree t owns global nodes off[t] .. off[t+1]-1;
 *                   off[0] = 0, strictly increasing; node ids inside a tree
 *                   are tree-local (0 = root)
 *   left_child, right_child  tree-local child ids; -1 on BOTH marks a leaf;
 *                   an internal node has both children in range
 *   split_feature, split_threshold  internal nodes only (threshold not NaN;
 *                   +-inf allowed)
 *   leaf_value      leaves only; finite
 *   default_left    NULL, or per node: nonzero sends a missing (NaN) feature
 *                   value left at that internal node (ignored on leaves);
 *                   with NULL every missing value goes right
 * Every node of a tree must be reachable from its root exactly once (no
 * cycles, no shared or orphan nodes), and no root-to-leaf path may have more
 * than ML2_MAX_DEPTH splits.  The sum T * max|leaf| + |base_score| must stay
 * below FLT_MAX / 2 so that no partial sum overflows.
 * Device layouts: ensembles whose paths have at most 12 splits and no
 * default-left node are padded to perfect trees unless that is more than
 * four times their node count; the others are packed tree by tree into
 * 24 KiB chunks, which holds trees of at most ML2_MAX_TREE_NODES nodes
 * (Table 3's depth-14 models trained on the paper's data are far smaller).
 */
typedef struct {
  int32_t num_trees;
  int32_t num_features;
  float base_score;
  const int64_t *tree_node_offset;
  const int32_t *left_child;
  const int32_t *right_child;
  const int32_t *split_feature;
  const float *split_threshold;
  const float *leaf_value;
  const uint8_t *default_left;
} ml2_ensemble_desc;

/*
 * Validate desc and build the device form of the ensemble on the current
 * device (synchronous).  Models V, P and A of Section 2 are each loaded this
 * way.  On success *out owns its device tables until ml2_free_ensemble; a
 * loaded ensemble may be used from several threads and streams at once.
 * Errors: INVALID_ARG (NULL pointers, malformed trees, out-of-range feature,
 * NaN threshold, non-finite leaf, overflow bound), UNSUPPORTED (depth, F or
 * tree size beyond the limits), OUT_OF_MEMORY, HIP.  *out is set to NULL on error.
 */
ml2_status ml2_load_ensemble(const ml2_ensemble_desc *desc, ml2_ensemble **out);

/* Release an ensemble (NULL is ignored).  The caller must have finished
 * every call that uses it (work enqueued on a stream counts until that
 * stream has passed it).  The device memory is returned with hipFree, which
 * waits for the device. */
void ml2_free_ensemble(ml2_ensemble *e);

/* Number of features / trees / depth (the longest path, or the padded depth
 * of the perfect layout) of a loaded ensemble (-1 on NULL). */
int32_t ml2_ensemble_num_features(const ml2_ensemble *e);
int32_t ml2_ensemble_num_trees(const ml2_ensemble *e);
int32_t ml2_ensemble_depth(const ml2_ensemble *e);

/*
 * Validity filter (model V, Section 2 "ML Model V"; hinge decision of
 * Table 3): for i in [0, n)
 *   margin_i     = fold of v over row i of X
 *   valid_out[i] = (margin_i > 0) ? 1 : 0          (uint8)
 *   margin_out[i]= margin_i                        (if margin_out != NULL)
 * X: float32 [n][ld] device, ld >= num_features(v), 4-byte aligned.
 * valid_out: uint8 [n] device.  margin_out: float32 [n] device or NULL.
 * n = 0 enqueues nothing.  Errors: INVALID_ARG (NULL ensemble/pointers with
 * n > 0, n < 0 or n > INT32_MAX, ld < F, misaligned X), HIP.
 */
ml2_status ml2_score_validity(const ml2_ensemble *v, const float *X, int64_t n, int64_t ld,
                              uint8_t *valid_out, float *margin_out, void *stream);

/*
 * Performance prediction over the candidates V accepted (model P, Section 2
 * "ML Model P"; regression objective of Table 3): for i in [0, n)
 *   score_out[i] = fold of p over row i of X   if valid == NULL or valid[i] != 0
 *                = -infinity                   otherwise
 * Only accepted rows are read from X and walked.
 * X as in ml2_score_validity; valid: uint8 [n] device or NULL (all accepted);
 * score_out: float32 [n] device.  Errors as ml2_score_validity.
 */
ml2_status ml2_score_perf(const ml2_ensemble *p, const float *X, int64_t n, int64_t ld,
                          const uint8_t *valid, float *score_out, void *stream);

/*
 * Validity and performance prediction in one call (models V and P of
 * Section 2, "ML Model V" / "ML Model P"): the same outputs, bit for bit, as
 * ml2_score_validity(v, X, n, ld, valid_out, margin_out) followed by
 * ml2_score_perf(p, X, n, ld, valid_out, score_out).  Where both ensembles
 * are perfect trees of one depth (at most 8) and fit one workgroup's LDS
 * together, and the rows are 16-byte aligned with a multiple of 4 and at most
 * 128 features, one kernel reads every row once and walks V and then P on
 * it (P on every row, which costs nothing in HBM traffic; rejected rows
 * still get -infinity); otherwise the two walks run one after the other.
 * ml2_score_single_pass says which (1: one pass).  Arguments and errors as
 * the two calls; X must hold the features of both ensembles.
 */
ml2_status ml2_score(const ml2_ensemble *v, const ml2_ensemble *p, const float *X, int64_t n,
                     int64_t ld, uint8_t *valid_out, float *margin_out, float *score_out,
                     void *stream);
int32_t ml2_score_single_pass(const ml2_ensemble *v, const ml2_ensemble *p, const float *X,
                              int64_t n, int64_t ld);

/* Device workspace bytes ml2_filter_topk needs for (n, k).  Errors:
 * INVALID_ARG (NULL bytes, n < 0, k < 0), UNSUPPORTED (k > ML2_MAX_TOPK). */
ml2_status ml2_topk_workspace_bytes(int64_t n, int32_t k, size_t *bytes);

/*
 * Selection of the configurations to pass on (Section 2: the explorer keeps
 * the highest predicted performance among the candidates V accepts, until
 * (alpha+1)*N are held; here k = (alpha+1)*N on a fixed pool).
 * A candidate is included iff (valid == NULL or valid[i] != 0) and
 * scores[i] is not NaN.  The included candidates are ordered by score
 * descending, then index ascending (-0.0 and +0.0 are equal, so ties between
 * them go to the lower index).  Writes
 *   topk_idx[j], topk_score[j]  for j < min(k, #included): index and its
 *                               score value (bit-exact copy of scores[idx])
 *   topk_idx[j] = -1, topk_score[j] = -inf for the remaining slots
 *   *num_selected = min(k, #included)          (int32, device)
 * valid: uint8 [n] device or NULL; scores: float32 [n] device;
 * topk_idx: int32 [k], topk_score: float32 [k], num_selected: int32 [1],
 * workspace: >= ml2_topk_workspace_bytes(n, k) bytes of device memory,
 * 256-byte aligned, used exclusively by this call until it completes.
 * Errors: INVALID_ARG (NULL pointers, n/k out of range, small workspace),
 * UNSUPPORTED (k > ML2_MAX_TOPK), HIP.
 */
ml2_status ml2_filter_topk(const uint8_t *valid, const float *scores, int64_t n, int32_t k,
                           int32_t *topk_idx, float *topk_score, int32_t *num_selected,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * ml2_filter_topk for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same selection and outputs as ml2_filter_topk, with the workspace
 * taken from a static array in the library's device code instead of an
 * argument.  The array (246,016 bytes, the workspace of k = ML2_MAX_TOPK) is
 * held by each device the library runs on until the process ends; its
 * device address is looked up on the first call on a device.  This call
 * allocates nothing.
 * Calls on one device share that device's array: two calls whose work
 * overlaps on the device (on different streams, or from different threads,
 * without ordering between them) race and give wrong results; calls ordered
 * on one stream are safe.  Each call starts by clearing the state it uses.
 * Arguments and errors as ml2_filter_topk without the workspace;
 * UNSUPPORTED for k > ML2_MAX_TOPK (beyond the static array).
 */
ml2_status ml2_filter_topk_noalloc(const uint8_t *valid, const float *scores, int64_t n,
                                   int32_t k, int32_t *topk_idx, float *topk_score,
                                   int32_t *num_selected, void *stream);

/*
 * Second-level selection (model A, Section 2 "Hidden Feature Extractor & ML
 * Model A"): of the (alpha+1)*N configurations the explorer holds, model A,
 * which sees the hidden features as well as the visible ones, picks the N
 * expected to perform best.  For i in [0, m):
 *   row_scores[i] = fold of a over row rows[i] of X   if 0 <= rows[i] < n
 *                 = -infinity                          otherwise (skipped)
 * The listed rows in range are ordered by row_scores descending, then pool
 * row ascending (-0.0 and +0.0 are equal; a row listed twice is taken twice).
 * Writes
 *   out_idx[j], out_score[j]  for j < min(keep, #in range): pool row and its
 *                             score (bit-exact copy of the entry's row_scores
 *                             value, sign of zero included)
 *   out_idx[j] = -1, out_score[j] = -inf for the remaining slots
 *   *num_selected = min(keep, #in range)        (int32, device)
 * X: float32 [n][ld] device, as in ml2_score_validity (a's features may be
 * more columns than those V and P use); rows: int32 [m] device, e.g. the
 * topk_idx of ml2_filter_topk (its -1 padding is skipped); row_scores:
 * float32 [m] device; out_idx: int32 [keep], out_score: float32 [keep],
 * num_selected: int32 [1], all device; workspace: at least
 * ml2_rerank_workspace_bytes(a, m) bytes of device memory, used by this
 * call until it completes.  The trees are walked in parallel over the
 * listed rows (a few rows still occupy the whole GPU) and each row's leaves
 * are then added in tree order.
 * Errors: INVALID_ARG (NULL pointers, m < 0, keep < 0, n out of range,
 * ld < F, misaligned X, small workspace), UNSUPPORTED (m or keep >
 * ML2_MAX_TOPK), HIP.
 */
ml2_status ml2_rerank(const ml2_ensemble *a, const float *X, int64_t n, int64_t ld,
                      const int32_t *rows, int32_t m, int32_t keep, float *row_scores,
                      int32_t *out_idx, float *out_score, int32_t *num_selected,
                      void *workspace, size_t workspace_bytes, void *stream);

/* Device workspace bytes ml2_rerank needs for m listed rows of ensemble a
 * (one float per tree and row).  Errors: INVALID_ARG (NULL a or bytes,
 * m < 0), UNSUPPORTED (m > ML2_MAX_TOPK). */
ml2_status ml2_rerank_workspace_bytes(const ml2_ensemble *a, int32_t m, size_t *bytes);

/*
 * The configuration explorer's rounds over one pool (Section 2: the
 * explorer proposes N configurations per iteration; it applies V and P until
 * (alpha+1)*N are held and model A keeps N; configurations proposed before
 * are not proposed again).  An explorer owns the device buffers of one pool
 * of n candidates (mask, scores, top-k state, the list of proposed rows) and
 * refers to, but does not own, its ensembles, which must outlive it.
 *   v, p: validity and performance ensembles; a: second-level ensemble or
 *   NULL (then the k held rows keep P's order); k = (alpha+1)*N rows held
 *   per round, keep = N rows proposed per round, max_rounds rounds before a
 *   reset.  Allocates device memory on the current device (synchronously).
 * Errors: INVALID_ARG (NULL out/v/p, n < 1, keep < 1 or > k, max_rounds < 1,
 * ensembles on another device), UNSUPPORTED (k > ML2_MAX_TOPK),
 * OUT_OF_MEMORY, HIP.
 */
typedef struct ml2_explorer ml2_explorer;
ml2_status ml2_explorer_create(const ml2_ensemble *v, const ml2_ensemble *p,
                               const ml2_ensemble *a, int64_t n, int32_t k, int32_t keep,
                               int32_t max_rounds, ml2_explorer **out);
/* Releases the explorer's memory (NULL is a no-op); as ml2_free_ensemble, the
 * caller must have finished every round enqueued on it. */
void ml2_explorer_free(ml2_explorer *ex);
/* Forgets every proposed row and the stored scores (INVALID_ARG if NULL). */
ml2_status ml2_explorer_reset(ml2_explorer *ex);
/* Rounds run since creation or the last reset (-1 for NULL). */
int32_t ml2_explorer_rounds(const ml2_explorer *ex);

/*
 * One round over the pool X (float32 [n][ld] device, ld >= every ensemble's
 * feature count, the same pool in every round):
 *   1. with rescore != 0 (the models changed) or in the first round:
 *      validity mask and performance scores of every row, as
 *      ml2_score_validity and ml2_score_perf; otherwise the stored ones;
 *   2. rows proposed in earlier rounds leave the mask;
 *   3. the k best remaining accepted rows, as ml2_filter_topk;
 *   4. the keep best of those by model A's score (or by P's without A),
 *      as ml2_rerank; written to out_idx/out_score (int32/float32 [keep],
 *      device; -1/-inf padding once the pool runs dry), *num_selected
 *      (int32, device), and recorded as proposed.
 * All of it is enqueued on `stream`; nothing waits for the device.  Calls
 * on one explorer must not overlap.  Errors: INVALID_ARG (NULL pointers,
 * ld too small, misaligned X, every round used), UNSUPPORTED, HIP.
 */
ml2_status ml2_explorer_round(ml2_explorer *ex, const float *X, int64_t ld, int32_t rescore,
                              int32_t *out_idx, float *out_score, int32_t *num_selected,
                              void *stream);

/*
 * The configuration explorer over a pool that arrives in chunks of rows
 * (Section 2, "Configuration Explorer": the explorer applies V and P to the
 * candidate configurations until (alpha+1)*N are held, model A keeps N, and a
 * configuration proposed once is not proposed again).  For search spaces that
 * are generated, read or copied to the device a piece at a time instead of
 * held in one resident matrix.  A round is
 *   ml2_stream_explorer_begin, ml2_stream_explorer_chunk for every chunk of
 *   the pool, ml2_stream_explorer_end;
 * its result is the same, bit for bit, as that of a round of ml2_explorer
 * over the pool of the distinct rows the chunks carry, in row order
 * (a row is identified by its pool row number; the k held are the best
 * accepted, not yet proposed rows by (P score desc, pool row asc), model A
 * or P's order keeps `keep`).  A chunk holds pool rows row0 .. row0+m-1; chunks
 * may come in any order, leave gaps and overlap: a row that arrives twice in
 * a round is held once (its features must be the same in every chunk).
 * Model A scores each chunk's selection while the chunk is on the device, so
 * no chunk is needed after its call returns (the caller may reuse its
 * memory once the stream has passed the call).
 * v, p, a: ensembles as for ml2_explorer_create (a may be NULL);
 * max_chunk_rows: the largest m of any chunk; k = (alpha+1)*N held, keep = N
 * proposed per round, max_rounds rounds before a reset.  The explorer owns
 * its device buffers (about 5 bytes per chunk row plus the selection's
 * workspace); it refers to, but does not own, its ensembles.
 * Errors: INVALID_ARG (NULL out/v/p, max_chunk_rows < 1, keep < 1 or > k,
 * max_rounds < 1, ensembles on another device), UNSUPPORTED
 * (k > ML2_MAX_STREAM_K), OUT_OF_MEMORY, HIP.
 */
typedef struct ml2_stream_explorer ml2_stream_explorer;
ml2_status ml2_stream_explorer_create(const ml2_ensemble *v, const ml2_ensemble *p,
                                      const ml2_ensemble *a, int64_t max_chunk_rows, int32_t k,
                                      int32_t keep, int32_t max_rounds,
                                      ml2_stream_explorer **out);
/* Releases the explorer's memory (NULL is a no-op); the caller must have
 * finished every call enqueued on it. */
void ml2_stream_explorer_free(ml2_stream_explorer *ex);
/* Forgets every proposed row and any open round (INVALID_ARG if NULL). */
ml2_status ml2_stream_explorer_reset(ml2_stream_explorer *ex);
/* Rounds ended since creation or the last reset (-1 for NULL). */
int32_t ml2_stream_explorer_rounds(const ml2_stream_explorer *ex);
/* Opens a round: nothing is held (enqueued on `stream`).  INVALID_ARG if a
 * round is open or every round is used, or on another device; HIP. */
ml2_status ml2_stream_explorer_begin(ml2_stream_explorer *ex, void *stream);
/* Scores chunk X (float32 [m][ld] device, ld >= every ensemble's feature
 * count, 4-byte aligned; pool rows row0 .. row0+m-1) and updates the held
 * set: its accepted rows not proposed in earlier rounds compete with those
 * held.  m = 0 does nothing.  All of it is enqueued on `stream`; calls on one
 * explorer must be ordered on one stream.  INVALID_ARG (no open round, m < 0
 * or > max_chunk_rows, row0 < 0 or row0 + m > 2^31 - 1, NULL X with m > 0,
 * ld too small, misaligned X), UNSUPPORTED, HIP. */
ml2_status ml2_stream_explorer_chunk(ml2_stream_explorer *ex, const float *X, int64_t m,
                                     int64_t ld, int64_t row0, void *stream);
/* Closes the round: writes the keep rows proposed (out_idx int32 [keep],
 * pool rows; out_score float32 [keep], model A's scores, or P's without A,
 * bit for bit; -1 / -inf padding once the pool runs dry; *num_selected, all
 * device) and records them as proposed.  INVALID_ARG (NULL outputs, no open
 * round), HIP. */
ml2_status ml2_stream_explorer_end(ml2_stream_explorer *ex, int32_t *out_idx, float *out_score,
                                   int32_t *num_selected, void *stream);

/* Thread-local description of the last non-OK status on this thread. */
const char *ml2_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ML2_H */
