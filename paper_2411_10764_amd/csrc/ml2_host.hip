// C-ABI entry points: argument validation, ensemble loading (validation,
// padding to perfect trees, packing into the device tree records) and the
// launches.  Everything here runs on the host; the arithmetic of the method
// runs in walk_kernels.hip and topk_kernels.hip.
#include <float.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "ml2_internal.h"
#include "pack.h"

using ml2::pack_ragged;
using ml2::pad_identity_tree;
using ml2::pad_tree;
using ml2::RaggedPack;
using ml2::TreeView;
#include "ml2_probe.h"

struct ml2_ensemble {
  ml2::Forest f;
};

// Device state of an explorer over one pool (see ml2_explorer_create).
struct ml2_explorer {
  const ml2_ensemble *v, *p, *a;  // not owned
  int device;
  int64_t n;
  int32_t k, keep, max_rounds, rounds;
  bool scored;  // valid/score hold the models' view of the pool
  void *block;  // one allocation holding every buffer below
  uint8_t *valid;
  float *score;
  int32_t *tk_idx;
  float *tk_score;
  int32_t *tk_num;
  float *a_scores;
  int32_t *proposed;  // [max_rounds * keep] rows proposed so far (-1 padding)
  void *ws;           // top-k workspace
  size_t ws_bytes;
  void *a_ws;         // second-level leaves
};

// Device state of a streamed explorer (see ml2_stream_explorer_create).
struct ml2_stream_explorer {
  const ml2_ensemble *v, *p, *a;  // not owned
  int device;
  int64_t max_rows;   // rows of the largest chunk
  int32_t k, keep, max_rounds, rounds;
  bool open;          // a round has begun and not ended
  int cur;            // which held set is current (0 or 1)
  void *block;        // one allocation holding every buffer below
  uint8_t *valid;     // [max_rows] chunk mask
  float *score;       // [max_rows] chunk P scores
  int32_t *tk_idx;    // [k] chunk selection (chunk-local rows)
  float *tk_score;
  int32_t *tk_num;
  float *a_scores;    // [k] model A's scores of the chunk selection
  int32_t *held_id[2];
  float *held_p[2], *held_a[2];
  int32_t *held_n[2];
  int32_t *proposed;  // [max_rounds * keep] pool rows proposed so far (-1 padding)
  void *ws;           // top-k workspace
  size_t ws_bytes;
  void *a_ws;         // second-level leaves
};

namespace {

thread_local std::string g_last_error;

ml2_status fail(ml2_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

ml2_status hip_fail(hipError_t e, const char *what) {
  return fail(ML2_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Compute-unit count per device, queried once.
int cu_count(int device) {
  static std::mutex mu;
  static std::vector<int> cache;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= device) cache.resize(device + 1, 0);
  if (cache[device] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
        v <= 0)
      v = 256;
    cache[device] = v;
  }
  return cache[device];
}

ml2_status current_device(int *dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  return ML2_OK;
}

// ---- descriptor validation ------------------------------------------------

// Checks that tree t is a proper binary tree rooted at 0 and returns its depth.
ml2_status check_tree(const ml2_ensemble_desc &d, int32_t t, const TreeView &tv, int *depth_out,
                      double *max_abs_leaf) {
  std::vector<uint8_t> seen((size_t)tv.size, 0);
  std::vector<std::pair<int32_t, int>> stack;
  stack.emplace_back(0, 0);
  seen[0] = 1;
  int64_t visited = 1;
  int depth = 0;
  while (!stack.empty()) {
    const auto [node, lvl] = stack.back();
    stack.pop_back();
    const int32_t l = tv.left[node], r = tv.right[node];
    if (l == -1 && r == -1) {
      const float v = tv.val[node];
      if (!isfinite(v))
        return fail(ML2_ERR_INVALID_ARG, "tree %d node %d: leaf value is not finite", t, node);
      if (fabs((double)v) > *max_abs_leaf) *max_abs_leaf = fabs((double)v);
      if (lvl > depth) depth = lvl;
      continue;
    }
    if (l < 0 || r < 0 || l >= tv.size || r >= tv.size)
      return fail(ML2_ERR_INVALID_ARG, "tree %d node %d: child ids (%d, %d) out of range", t,
                  node, l, r);
    const int32_t f = tv.feat[node];
    if (f < 0 || f >= d.num_features)
      return fail(ML2_ERR_INVALID_ARG, "tree %d node %d: split feature %d outside [0, %d)", t,
                  node, f, d.num_features);
    if (isnan(tv.thr[node]))
      return fail(ML2_ERR_INVALID_ARG, "tree %d node %d: split threshold is NaN", t, node);
    if (lvl + 1 > ML2_MAX_DEPTH)
      return fail(ML2_ERR_UNSUPPORTED, "tree %d: depth exceeds %d", t, ML2_MAX_DEPTH);
    for (int32_t c : {l, r}) {
      if (seen[c])
        return fail(ML2_ERR_INVALID_ARG, "tree %d: node %d reached twice (cycle or shared node)",
                    t, c);
      seen[c] = 1;
      ++visited;
      stack.emplace_back(c, lvl + 1);
    }
  }
  if (visited != tv.size)
    return fail(ML2_ERR_INVALID_ARG, "tree %d: %lld of %lld nodes unreachable from the root", t,
                (long long)(tv.size - visited), (long long)tv.size);
  *depth_out = depth;
  return ML2_OK;
}


ml2_status check_stream_args(const ml2_ensemble *e, const float *X, int64_t n, int64_t ld,
                             const void *out, const char *what, int *dev) {
  if (!e) return fail(ML2_ERR_INVALID_ARG, "%s: ensemble is NULL", what);
  if (n < 0 || n > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "%s: n = %lld outside [0, 2^31-1]", what, (long long)n);
  if (ld < e->f.num_features)
    return fail(ML2_ERR_INVALID_ARG, "%s: ld = %lld < num_features = %d", what, (long long)ld,
                e->f.num_features);
  if (n > 0 && (!X || !out)) return fail(ML2_ERR_INVALID_ARG, "%s: NULL device pointer", what);
  if (X && (reinterpret_cast<uintptr_t>(X) & 3u))
    return fail(ML2_ERR_INVALID_ARG, "%s: X is not 4-byte aligned", what);
  ml2_status st = current_device(dev);
  if (st != ML2_OK) return st;
  if (*dev != e->f.device)
    return fail(ML2_ERR_INVALID_ARG, "%s: ensemble lives on device %d, current device is %d",
                what, e->f.device, *dev);
  return ML2_OK;
}

}  // namespace

// Microbenchmark timing (ml2_probe.h).
namespace {

// One untimed and one timed launch of `launch` (which writes to a buffer of
// out_bytes device bytes) on the null stream; *ms: the timed launch.
template <typename Launch>
ml2_status time_probe(const char *what, size_t out_bytes, double *ms, double *work,
                      Launch launch) {
  void *out = nullptr;
  hipError_t e = hipMalloc(&out, out_bytes);
  if (e != hipSuccess) return fail(ML2_ERR_OUT_OF_MEMORY, "%s: hipMalloc(%zu)", what, out_bytes);
  hipEvent_t t0 = nullptr, t1 = nullptr;
  float elapsed = 0.0f;
  e = hipEventCreate(&t0);
  if (e == hipSuccess) e = hipEventCreate(&t1);
  if (e == hipSuccess) e = launch(out, work, nullptr);
  if (e == hipSuccess) e = hipEventRecord(t0, nullptr);
  if (e == hipSuccess) e = launch(out, work, nullptr);
  if (e == hipSuccess) e = hipEventRecord(t1, nullptr);
  if (e == hipSuccess) e = hipEventSynchronize(t1);
  if (e == hipSuccess) e = hipEventElapsedTime(&elapsed, t0, t1);
  if (t0) (void)hipEventDestroy(t0);
  if (t1) (void)hipEventDestroy(t1);
  (void)hipFree(out);
  if (e != hipSuccess) return hip_fail(e, what);
  *ms = elapsed;
  return ML2_OK;
}

ml2_status check_probe(const char *what, int32_t iters, int32_t blocks, const double *ms,
                       const double *work) {
  if (!ms || !work) return fail(ML2_ERR_INVALID_ARG, "%s: NULL output", what);
  if (iters < 1 || iters > (1 << 20))
    return fail(ML2_ERR_INVALID_ARG, "%s: iters = %d outside [1, 2^20]", what, iters);
  if (blocks < 1 || blocks > 65536)
    return fail(ML2_ERR_INVALID_ARG, "%s: blocks = %d outside [1, 65536]", what, blocks);
  return ML2_OK;
}

}  // namespace

namespace ml2 {

hipError_t ensure_dynamic_lds(const void *fn, size_t bytes) {
  static std::mutex mu;
  static std::unordered_map<const void *, std::vector<size_t>> set;  // per kernel, per device
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  std::vector<size_t> &v = set[fn];
  if ((int)v.size() <= dev) v.resize((size_t)dev + 1, 0);
  if (bytes > v[(size_t)dev]) {
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
    v[(size_t)dev] = bytes;
  }
  return hipSuccess;
}

}  // namespace ml2

extern "C" {

const char *ml2_last_error(void) { return g_last_error.c_str(); }

ml2_status ml2_load_ensemble(const ml2_ensemble_desc *desc, ml2_ensemble **out) {
  if (!out) return fail(ML2_ERR_INVALID_ARG, "ml2_load_ensemble: out is NULL");
  *out = nullptr;
  if (!desc) return fail(ML2_ERR_INVALID_ARG, "ml2_load_ensemble: desc is NULL");
  const ml2_ensemble_desc &d = *desc;
  if (d.num_trees < 1) return fail(ML2_ERR_INVALID_ARG, "num_trees = %d < 1", d.num_trees);
  if (d.num_features < 1) return fail(ML2_ERR_INVALID_ARG, "num_features = %d < 1", d.num_features);
  if (d.num_features > ML2_MAX_FEATURES)
    return fail(ML2_ERR_UNSUPPORTED, "num_features = %d > %d", d.num_features, ML2_MAX_FEATURES);
  if (!d.tree_node_offset || !d.left_child || !d.right_child || !d.split_feature ||
      !d.split_threshold || !d.leaf_value)
    return fail(ML2_ERR_INVALID_ARG, "ml2_load_ensemble: NULL array in the descriptor");
  if (!isfinite(d.base_score)) return fail(ML2_ERR_INVALID_ARG, "base_score is not finite");
  if (d.tree_node_offset[0] != 0)
    return fail(ML2_ERR_INVALID_ARG, "tree_node_offset[0] = %lld, expected 0",
                (long long)d.tree_node_offset[0]);
  int depth = 1;
  double max_leaf = 0.0;
  int64_t total_nodes = 0, max_nodes = 0;
  bool any_default_left = false;
  std::vector<TreeView> views((size_t)d.num_trees);
  std::vector<int> depths((size_t)d.num_trees);
  for (int32_t t = 0; t < d.num_trees; ++t) {
    const int64_t a = d.tree_node_offset[t], b = d.tree_node_offset[t + 1];
    if (b <= a || b - a > (int64_t)INT32_MAX)
      return fail(ML2_ERR_INVALID_ARG, "tree %d: node range [%lld, %lld) is empty or too large",
                  t, (long long)a, (long long)b);
    TreeView tv{d.left_child + a, d.right_child + a, d.split_feature + a,
                d.split_threshold + a, d.leaf_value + a,
                d.default_left ? d.default_left + a : nullptr, b - a};
    int dt = 0;
    ml2_status st = check_tree(d, t, tv, &dt, &max_leaf);
    if (st != ML2_OK) return st;
    if (dt > depth) depth = dt;
    depths[(size_t)t] = dt;
    views[(size_t)t] = tv;
    total_nodes += tv.size;
    if (tv.size > max_nodes) max_nodes = tv.size;
    if (tv.dl)
      for (int64_t i = 0; i < tv.size && !any_default_left; ++i)
        any_default_left = tv.left[i] != -1 && tv.dl[i] != 0;
  }
  if ((double)d.num_trees * max_leaf + fabs((double)d.base_score) >= (double)FLT_MAX / 2)
    return fail(ML2_ERR_INVALID_ARG, "num_trees * max|leaf| + |base| may overflow float32");

  // Layout: perfect padded trees where they represent the ensemble and are
  // not much larger than its nodes; ragged slots otherwise (deeper than the
  // perfect limit, default directions, or sparse trees).  The tuning
  // override (ml2_tune_layout) forces a layout that can represent it.
  const int64_t tpad16 = (d.num_trees + ml2::kTreePad - 1) / ml2::kTreePad * ml2::kTreePad;
  const bool perfect_ok = depth <= ml2::kMaxPerfectDepth && !any_default_left;
  const bool ragged_ok = max_nodes <= ML2_MAX_TREE_NODES;
  bool ragged = !perfect_ok ||
                (ragged_ok && (double)tpad16 * ml2::record_bytes(depth) > 4.0 * 12.0 * total_nodes);
  const int forced = ml2::get_tune(ml2::kTuneLayout);
  if (forced == 2 && ragged_ok) ragged = true;
  if (forced == 1 && perfect_ok) ragged = false;
  if (ragged && !ragged_ok)
    return fail(ML2_ERR_UNSUPPORTED,
                "a tree of %lld nodes needs the ragged layout (deeper than %d levels or default "
                "directions), which holds at most %d nodes per tree",
                (long long)max_nodes, ml2::kMaxPerfectDepth, ML2_MAX_TREE_NODES);

  ml2::Forest f{};
  ml2_status st = current_device(&f.device);
  if (st != ML2_OK) return st;
  f.num_trees = d.num_trees;
  f.num_features = d.num_features;
  f.base = d.base_score;
  f.ragged = ragged ? 1 : 0;
  std::vector<char> host;
  size_t bytes = 0;
  if (ragged) {
    RaggedPack pk;
    try {
      pack_ragged(views, depths, &pk);
    } catch (const std::bad_alloc &) {
      return fail(ML2_ERR_OUT_OF_MEMORY, "host staging of the ragged layout failed");
    }
    f.num_trees_padded = pk.trees;
    f.records = pk.slots;
    f.depth = pk.depth;
    f.rec_bytes = ml2::record_bytes(0);
    host.swap(pk.bytes);
    bytes = host.size();
  } else {
    f.num_trees_padded = (int32_t)tpad16;
    f.records = f.num_trees_padded;
    f.depth = depth;
    f.rec_bytes = ml2::record_bytes(depth);
    bytes = (size_t)f.num_trees_padded * f.rec_bytes;
    try {
      host.assign(bytes, 0);
    } catch (const std::bad_alloc &) {
      return fail(ML2_ERR_OUT_OF_MEMORY, "host staging of %zu bytes failed", bytes);
    }
    for (int32_t t = 0; t < f.num_trees_padded; ++t) {
      char *rec = host.data() + (size_t)t * f.rec_bytes;
      if (t < d.num_trees)
        pad_tree(views[(size_t)t], depth, rec);
      else
        pad_identity_tree(depth, rec);
    }
  }
  // The tree table is followed by kTreeSlack zero bytes: chunk staging reads
  // whole register sets, past the end of the last chunk.
  hipError_t e = hipMalloc(&f.d_trees, bytes + ml2::kTreeSlack);
  if (e == hipErrorOutOfMemory)
    return fail(ML2_ERR_OUT_OF_MEMORY, "hipMalloc(%zu)", bytes + ml2::kTreeSlack);
  if (e != hipSuccess) return hip_fail(e, "hipMalloc");
  e = hipMemset(f.d_trees, 0, bytes + ml2::kTreeSlack);
  if (e == hipSuccess) e = hipMemcpy(f.d_trees, host.data(), bytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(f.d_trees);
    return hip_fail(e, "hipMemcpy");
  }
  ml2_ensemble *h = new (std::nothrow) ml2_ensemble;
  if (!h) {
    (void)hipFree(f.d_trees);
    return fail(ML2_ERR_OUT_OF_MEMORY, "handle allocation failed");
  }
  h->f = f;
  *out = h;
  return ML2_OK;
}

void ml2_free_ensemble(ml2_ensemble *e) {
  if (!e) return;
  int cur = 0;
  const bool other = hipGetDevice(&cur) == hipSuccess && cur != e->f.device;
  if (other) (void)hipSetDevice(e->f.device);
  (void)hipFree(e->f.d_trees);
  if (other) (void)hipSetDevice(cur);
  delete e;
}

int32_t ml2_ensemble_num_features(const ml2_ensemble *e) { return e ? e->f.num_features : -1; }
int32_t ml2_ensemble_num_trees(const ml2_ensemble *e) { return e ? e->f.num_trees : -1; }
int32_t ml2_ensemble_depth(const ml2_ensemble *e) { return e ? e->f.depth : -1; }

ml2_status ml2_score_validity(const ml2_ensemble *v, const float *X, int64_t n, int64_t ld,
                              uint8_t *valid_out, float *margin_out, void *stream) {
  int dev = 0;
  ml2_status st = check_stream_args(v, X, n, ld, valid_out, "ml2_score_validity", &dev);
  if (st != ML2_OK) return st;
  if (n == 0) return ML2_OK;
  ml2::WalkPlan p;
  const char *why = nullptr;
  if (!ml2::plan_walk(v->f, n, cu_count(dev), &p, &why))
    return fail(ML2_ERR_UNSUPPORTED, "ml2_score_validity: %s", why);
  hipError_t e = ml2::launch_validity(v->f, p, X, n, ld, valid_out, margin_out,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "validity kernel launch");
  return ML2_OK;
}

ml2_status ml2_score_perf(const ml2_ensemble *p_ens, const float *X, int64_t n, int64_t ld,
                          const uint8_t *valid, float *score_out, void *stream) {
  int dev = 0;
  ml2_status st = check_stream_args(p_ens, X, n, ld, score_out, "ml2_score_perf", &dev);
  if (st != ML2_OK) return st;
  if (n == 0) return ML2_OK;
  ml2::WalkPlan p;
  const char *why = nullptr;
  if (!ml2::plan_walk(p_ens->f, n, cu_count(dev), &p, &why, valid != nullptr))
    return fail(ML2_ERR_UNSUPPORTED, "ml2_score_perf: %s", why);
  hipError_t e = ml2::launch_perf(p_ens->f, p, X, n, ld, valid, score_out,
                                  static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "perf kernel launch");
  return ML2_OK;
}

namespace {

ml2_status check_score_args(const ml2_ensemble *v, const ml2_ensemble *p, const float *X,
                            int64_t n, int64_t ld, const void *valid_out, const void *score_out,
                            const char *what, int *dev) {
  ml2_status st = check_stream_args(v, X, n, ld, valid_out, what, dev);
  if (st != ML2_OK) return st;
  st = check_stream_args(p, X, n, ld, score_out, what, dev);
  if (st != ML2_OK) return st;
  return ML2_OK;
}

}  // namespace

ml2_status ml2_score(const ml2_ensemble *v, const ml2_ensemble *p, const float *X, int64_t n,
                     int64_t ld, uint8_t *valid_out, float *margin_out, float *score_out,
                     void *stream) {
  int dev = 0;
  ml2_status st = check_score_args(v, p, X, n, ld, valid_out, score_out, "ml2_score", &dev);
  if (st != ML2_OK) return st;
  if (n == 0) return ML2_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  ml2::WalkPlan pl;
  int nv = 0, np = 0;
  if (ml2::plan_fused(v->f, p->f, n, ld, X, cu_count(dev), &pl, &nv, &np)) {
    hipError_t e = ml2::launch_fused(v->f, p->f, pl, nv, np, X, n, ld, valid_out, margin_out,
                                     score_out, s);
    if (e != hipSuccess) return hip_fail(e, "ml2_score: launch");
    return ML2_OK;
  }
  ml2::WalkPlan pv, pp;
  const char *why = nullptr;
  if (!ml2::plan_walk(v->f, n, cu_count(dev), &pv, &why) ||
      !ml2::plan_walk(p->f, n, cu_count(dev), &pp, &why, true))
    return fail(ML2_ERR_UNSUPPORTED, "ml2_score: %s", why);
  hipError_t e = ml2::launch_validity(v->f, pv, X, n, ld, valid_out, margin_out, s);
  if (e == hipSuccess) e = ml2::launch_perf(p->f, pp, X, n, ld, valid_out, score_out, s);
  if (e != hipSuccess) return hip_fail(e, "ml2_score: launch");
  return ML2_OK;
}

int32_t ml2_score_single_pass(const ml2_ensemble *v, const ml2_ensemble *p, const float *X,
                              int64_t n, int64_t ld) {
  if (!v || !p || n < 1 || ld < v->f.num_features || ld < p->f.num_features) return 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  ml2::WalkPlan pl;
  int nv = 0, np = 0;
  return ml2::plan_fused(v->f, p->f, n, ld, X, cu_count(dev), &pl, &nv, &np) ? 1 : 0;
}

ml2_status ml2_topk_workspace_bytes(int64_t n, int32_t k, size_t *bytes) {
  if (!bytes) return fail(ML2_ERR_INVALID_ARG, "ml2_topk_workspace_bytes: bytes is NULL");
  if (n < 0 || n > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "ml2_topk_workspace_bytes: n = %lld out of range",
                (long long)n);
  if (k < 0) return fail(ML2_ERR_INVALID_ARG, "ml2_topk_workspace_bytes: k = %d < 0", k);
  if (k > ML2_MAX_TOPK)
    return fail(ML2_ERR_UNSUPPORTED, "ml2_topk_workspace_bytes: k = %d > %d", k, ML2_MAX_TOPK);
  *bytes = ml2::topk_workspace_bytes(n, k);
  return ML2_OK;
}

ml2_status ml2_filter_topk(const uint8_t *valid, const float *scores, int64_t n, int32_t k,
                           int32_t *topk_idx, float *topk_score, int32_t *num_selected,
                           void *workspace, size_t workspace_bytes, void *stream) {
  if (n < 0 || n > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: n = %lld out of range", (long long)n);
  if (k < 0) return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: k = %d < 0", k);
  if (k > ML2_MAX_TOPK)
    return fail(ML2_ERR_UNSUPPORTED, "ml2_filter_topk: k = %d > %d", k, ML2_MAX_TOPK);
  if (!num_selected || !workspace)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: NULL num_selected or workspace");
  if (n > 0 && !scores) return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: scores is NULL");
  if (k > 0 && (!topk_idx || !topk_score))
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: NULL output array");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: workspace is not 256-byte aligned");
  const size_t need = ml2::topk_workspace_bytes(n, k);
  if (workspace_bytes < need)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk: workspace %zu < %zu bytes",
                workspace_bytes, need);
  int dev = 0;
  ml2_status st = current_device(&dev);
  if (st != ML2_OK) return st;
  hipError_t e = ml2::launch_topk(valid, scores, n, k, topk_idx, topk_score, num_selected,
                                  workspace, cu_count(dev), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "top-k kernel launch");
  return ML2_OK;
}

ml2_status ml2_filter_topk_noalloc(const uint8_t *valid, const float *scores, int64_t n,
                                   int32_t k, int32_t *topk_idx, float *topk_score,
                                   int32_t *num_selected, void *stream) {
  if (n < 0 || n > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk_noalloc: n = %lld out of range",
                (long long)n);
  if (k < 0) return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk_noalloc: k = %d < 0", k);
  if (k > ML2_MAX_TOPK)
    return fail(ML2_ERR_UNSUPPORTED,
                "ml2_filter_topk_noalloc: k = %d > %d (the static scratch holds the workspace "
                "of k <= %d)", k, ML2_MAX_TOPK, ML2_MAX_TOPK);
  if (!num_selected)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk_noalloc: num_selected is NULL");
  if (n > 0 && !scores)
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk_noalloc: scores is NULL");
  if (k > 0 && (!topk_idx || !topk_score))
    return fail(ML2_ERR_INVALID_ARG, "ml2_filter_topk_noalloc: NULL output array");
  const size_t need = ml2::topk_workspace_bytes(n, k);
  if (need > ml2::static_scratch_bytes())
    return fail(ML2_ERR_UNSUPPORTED, "ml2_filter_topk_noalloc: workspace %zu > static %zu bytes",
                need, ml2::static_scratch_bytes());
  int dev = 0;
  ml2_status st = current_device(&dev);
  if (st != ML2_OK) return st;
  void *ws = nullptr;
  hipError_t e = ml2::static_scratch(dev, &ws);
  if (e != hipSuccess) return hip_fail(e, "ml2_filter_topk_noalloc: hipGetSymbolAddress");
  e = ml2::launch_topk(valid, scores, n, k, topk_idx, topk_score, num_selected, ws, cu_count(dev),
                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "top-k kernel launch");
  return ML2_OK;
}

ml2_status ml2_rerank_workspace_bytes(const ml2_ensemble *a, int32_t m, size_t *bytes) {
  if (!a || !bytes) return fail(ML2_ERR_INVALID_ARG, "ml2_rerank_workspace_bytes: NULL argument");
  if (m < 0) return fail(ML2_ERR_INVALID_ARG, "ml2_rerank_workspace_bytes: m = %d < 0", m);
  if (m > ML2_MAX_TOPK)
    return fail(ML2_ERR_UNSUPPORTED, "ml2_rerank_workspace_bytes: m = %d > %d", m, ML2_MAX_TOPK);
  *bytes = ml2::rows_workspace_bytes(a->f, m);
  return ML2_OK;
}

ml2_status ml2_rerank(const ml2_ensemble *a, const float *X, int64_t n, int64_t ld,
                      const int32_t *rows, int32_t m, int32_t keep, float *row_scores,
                      int32_t *out_idx, float *out_score, int32_t *num_selected,
                      void *workspace, size_t workspace_bytes, void *stream) {
  int dev = 0;
  ml2_status st = check_stream_args(a, X, n, ld, X, "ml2_rerank", &dev);
  if (st != ML2_OK) return st;
  if (m < 0) return fail(ML2_ERR_INVALID_ARG, "ml2_rerank: m = %d < 0", m);
  if (keep < 0) return fail(ML2_ERR_INVALID_ARG, "ml2_rerank: keep = %d < 0", keep);
  if (m > ML2_MAX_TOPK || keep > ML2_MAX_TOPK)
    return fail(ML2_ERR_UNSUPPORTED, "ml2_rerank: m = %d or keep = %d > %d", m, keep,
                ML2_MAX_TOPK);
  if (!num_selected) return fail(ML2_ERR_INVALID_ARG, "ml2_rerank: num_selected is NULL");
  if (m > 0 && (!rows || !row_scores))
    return fail(ML2_ERR_INVALID_ARG, "ml2_rerank: NULL rows or row_scores");
  if (keep > 0 && (!out_idx || !out_score))
    return fail(ML2_ERR_INVALID_ARG, "ml2_rerank: NULL output array");
  const size_t need = ml2::rows_workspace_bytes(a->f, m);
  if (m > 0 && n > 0 && (!workspace || workspace_bytes < need))
    return fail(ML2_ERR_INVALID_ARG, "ml2_rerank: workspace %zu < %zu bytes", workspace_bytes,
                need);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (m > 0 && n > 0) {
    hipError_t e = ml2::launch_rows(a->f, X, n, ld, rows, m, row_scores, workspace, cu_count(dev),
                                    s);
    if (e != hipSuccess) return hip_fail(e, "rerank walk launch");
  }
  if (m > 0 && n == 0) {  // no listed row is in range (and X may be NULL)
    hipError_t e = hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(row_scores), 0xFF800000u,
                                     (size_t)m, s);
    if (e != hipSuccess) return hip_fail(e, "rerank score fill");
  }
  hipError_t e = ml2::launch_rerank_select(rows, row_scores, m, n, keep, out_idx, out_score,
                                           num_selected, s);
  if (e != hipSuccess) return hip_fail(e, "rerank select launch");
  return ML2_OK;
}

ml2_status ml2_explorer_create(const ml2_ensemble *v, const ml2_ensemble *p,
                               const ml2_ensemble *a, int64_t n, int32_t k, int32_t keep,
                               int32_t max_rounds, ml2_explorer **out) {
  if (!out) return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_create: out is NULL");
  *out = nullptr;
  if (!v || !p) return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_create: NULL V or P ensemble");
  if (n < 1 || n > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_create: n = %lld outside [1, 2^31-1]",
                (long long)n);
  if (k < 1 || keep < 1 || keep > k || max_rounds < 1)
    return fail(ML2_ERR_INVALID_ARG,
                "ml2_explorer_create: need 1 <= keep <= k and max_rounds >= 1 (k = %d, keep = "
                "%d, max_rounds = %d)", k, keep, max_rounds);
  if (k > ML2_MAX_TOPK)
    return fail(ML2_ERR_UNSUPPORTED, "ml2_explorer_create: k = %d > %d", k, ML2_MAX_TOPK);
  if ((int64_t)max_rounds * keep > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_create: max_rounds * keep overflows");
  int dev = 0;
  ml2_status st = current_device(&dev);
  if (st != ML2_OK) return st;
  if (v->f.device != dev || p->f.device != dev || (a && a->f.device != dev))
    return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_create: ensembles not on device %d", dev);
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t ws = ml2::topk_workspace_bytes(n, k);
  const size_t a_ws = a ? ml2::rows_workspace_bytes(a->f, k) : 0;
  const size_t sizes[] = {up((size_t)n), up(4 * (size_t)n), up(4 * (size_t)k), up(4 * (size_t)k),
                          up(4), up(4 * (size_t)k), up(4 * (size_t)max_rounds * keep), up(ws),
                          up(a_ws)};
  size_t total = 0;
  for (size_t b : sizes) total += b;
  ml2_explorer *ex = new (std::nothrow) ml2_explorer{};
  if (!ex) return fail(ML2_ERR_OUT_OF_MEMORY, "ml2_explorer_create: handle allocation failed");
  hipError_t e = hipMalloc(&ex->block, total);
  if (e != hipSuccess) {
    delete ex;
    if (e == hipErrorOutOfMemory)
      return fail(ML2_ERR_OUT_OF_MEMORY, "ml2_explorer_create: hipMalloc(%zu)", total);
    return hip_fail(e, "ml2_explorer_create: hipMalloc");
  }
  char *c = static_cast<char *>(ex->block);
  ex->valid = reinterpret_cast<uint8_t *>(c);            c += sizes[0];
  ex->score = reinterpret_cast<float *>(c);              c += sizes[1];
  ex->tk_idx = reinterpret_cast<int32_t *>(c);           c += sizes[2];
  ex->tk_score = reinterpret_cast<float *>(c);           c += sizes[3];
  ex->tk_num = reinterpret_cast<int32_t *>(c);           c += sizes[4];
  ex->a_scores = reinterpret_cast<float *>(c);           c += sizes[5];
  ex->proposed = reinterpret_cast<int32_t *>(c);         c += sizes[6];
  ex->ws = c;                                            c += sizes[7];
  ex->ws_bytes = sizes[7];
  ex->a_ws = c;
  ex->v = v;
  ex->p = p;
  ex->a = a;
  ex->device = dev;
  ex->n = n;
  ex->k = k;
  ex->keep = keep;
  ex->max_rounds = max_rounds;
  ex->rounds = 0;
  ex->scored = false;
  *out = ex;
  return ML2_OK;
}

void ml2_explorer_free(ml2_explorer *ex) {
  if (!ex) return;
  int cur = 0;
  const bool other = hipGetDevice(&cur) == hipSuccess && cur != ex->device;
  if (other) (void)hipSetDevice(ex->device);
  (void)hipFree(ex->block);
  if (other) (void)hipSetDevice(cur);
  delete ex;
}

ml2_status ml2_explorer_reset(ml2_explorer *ex) {
  if (!ex) return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_reset: explorer is NULL");
  ex->rounds = 0;
  ex->scored = false;
  return ML2_OK;
}

int32_t ml2_explorer_rounds(const ml2_explorer *ex) { return ex ? ex->rounds : -1; }

ml2_status ml2_explorer_round(ml2_explorer *ex, const float *X, int64_t ld, int32_t rescore,
                              int32_t *out_idx, float *out_score, int32_t *num_selected,
                              void *stream) {
  if (!ex) return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_round: explorer is NULL");
  if (!out_idx || !out_score || !num_selected)
    return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_round: NULL output array");
  if (ex->rounds >= ex->max_rounds)
    return fail(ML2_ERR_INVALID_ARG, "ml2_explorer_round: all %d rounds used (reset first)",
                ex->max_rounds);
  int dev = 0;
  const ml2_ensemble *models[3] = {ex->v, ex->p, ex->a};
  for (const ml2_ensemble *m : models) {
    if (!m) continue;
    ml2_status st = check_stream_args(m, X, ex->n, ld, X, "ml2_explorer_round", &dev);
    if (st != ML2_OK) return st;
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int cus = cu_count(dev);
  const int32_t held = ex->rounds * ex->keep;  // rows proposed in earlier rounds
  hipError_t e = hipSuccess;
  if (rescore || !ex->scored) {
    ml2::WalkPlan pv, pp;
    const char *why = nullptr;
    if (!ml2::plan_walk(ex->v->f, ex->n, cus, &pv, &why) ||
        !ml2::plan_walk(ex->p->f, ex->n, cus, &pp, &why, true))
      return fail(ML2_ERR_UNSUPPORTED, "ml2_explorer_round: %s", why);
    e = ml2::launch_validity(ex->v->f, pv, X, ex->n, ld, ex->valid, nullptr, s);
    if (e == hipSuccess) e = ml2::launch_exclude(ex->valid, ex->n, ex->proposed, held, s);
    if (e == hipSuccess) e = ml2::launch_perf(ex->p->f, pp, X, ex->n, ld, ex->valid, ex->score, s);
    if (e != hipSuccess) return hip_fail(e, "explorer scoring launch");
  } else if (ex->rounds > 0) {
    // same scores: only the previous round's rows leave the pool
    e = ml2::launch_exclude(ex->valid, ex->n, ex->proposed + held - ex->keep, ex->keep, s);
    if (e != hipSuccess) return hip_fail(e, "explorer exclusion launch");
  }
  e = ml2::launch_topk(ex->valid, ex->score, ex->n, ex->k, ex->tk_idx, ex->tk_score, ex->tk_num,
                       ex->ws, cus, s);
  if (e != hipSuccess) return hip_fail(e, "explorer top-k launch");
  const float *by = ex->tk_score;  // without model A the k held keep their P order
  if (ex->a) {
    e = ml2::launch_rows(ex->a->f, X, ex->n, ld, ex->tk_idx, ex->k, ex->a_scores, ex->a_ws, cus,
                         s);
    if (e != hipSuccess) return hip_fail(e, "explorer re-rank launch");
    by = ex->a_scores;
  }
  e = ml2::launch_rerank_select(ex->tk_idx, by, ex->k, ex->n, ex->keep, out_idx, out_score,
                                num_selected, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(ex->proposed + held, out_idx, sizeof(int32_t) * ex->keep,
                       hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "explorer selection launch");
  ex->rounds += 1;
  ex->scored = true;
  return ML2_OK;
}

// ---- the explorer over a streamed pool -------------------------------------------

ml2_status ml2_stream_explorer_create(const ml2_ensemble *v, const ml2_ensemble *p,
                                      const ml2_ensemble *a, int64_t max_chunk_rows, int32_t k,
                                      int32_t keep, int32_t max_rounds,
                                      ml2_stream_explorer **out) {
  if (!out) return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_create: out is NULL");
  *out = nullptr;
  if (!v || !p)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_create: NULL V or P ensemble");
  if (max_chunk_rows < 1 || max_chunk_rows > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG,
                "ml2_stream_explorer_create: max_chunk_rows = %lld outside [1, 2^31-1]",
                (long long)max_chunk_rows);
  if (k < 1 || keep < 1 || keep > k || max_rounds < 1)
    return fail(ML2_ERR_INVALID_ARG,
                "ml2_stream_explorer_create: need 1 <= keep <= k and max_rounds >= 1 (k = %d, "
                "keep = %d, max_rounds = %d)", k, keep, max_rounds);
  if (k > ML2_MAX_STREAM_K)
    return fail(ML2_ERR_UNSUPPORTED, "ml2_stream_explorer_create: k = %d > %d", k,
                ML2_MAX_STREAM_K);
  if ((int64_t)max_rounds * keep > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_create: max_rounds * keep overflows");
  int dev = 0;
  ml2_status st = current_device(&dev);
  if (st != ML2_OK) return st;
  if (v->f.device != dev || p->f.device != dev || (a && a->f.device != dev))
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_create: ensembles not on device %d",
                dev);
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t n = (size_t)max_chunk_rows, kk = (size_t)k;
  const size_t ws = ml2::topk_workspace_bytes(max_chunk_rows, k);
  const size_t a_ws = a ? ml2::rows_workspace_bytes(a->f, k) : 0;
  const size_t sizes[] = {up(n), up(4 * n), up(4 * kk), up(4 * kk), up(4), up(4 * kk),
                          up(4 * kk), up(4 * kk), up(4 * kk), up(4),
                          up(4 * kk), up(4 * kk), up(4 * kk), up(4),
                          up(4 * (size_t)max_rounds * keep), up(ws), up(a_ws)};
  size_t total = 0;
  for (size_t b : sizes) total += b;
  ml2_stream_explorer *ex = new (std::nothrow) ml2_stream_explorer{};
  if (!ex)
    return fail(ML2_ERR_OUT_OF_MEMORY, "ml2_stream_explorer_create: handle allocation failed");
  hipError_t e = hipMalloc(&ex->block, total);
  if (e != hipSuccess) {
    delete ex;
    if (e == hipErrorOutOfMemory)
      return fail(ML2_ERR_OUT_OF_MEMORY, "ml2_stream_explorer_create: hipMalloc(%zu)", total);
    return hip_fail(e, "ml2_stream_explorer_create: hipMalloc");
  }
  char *c = static_cast<char *>(ex->block);
  size_t i = 0;
  auto take = [&](size_t) {
    char *q = c;
    c += sizes[i++];
    return q;
  };
  ex->valid = reinterpret_cast<uint8_t *>(take(0));
  ex->score = reinterpret_cast<float *>(take(0));
  ex->tk_idx = reinterpret_cast<int32_t *>(take(0));
  ex->tk_score = reinterpret_cast<float *>(take(0));
  ex->tk_num = reinterpret_cast<int32_t *>(take(0));
  ex->a_scores = reinterpret_cast<float *>(take(0));
  for (int h = 0; h < 2; ++h) {
    ex->held_id[h] = reinterpret_cast<int32_t *>(take(0));
    ex->held_p[h] = reinterpret_cast<float *>(take(0));
    ex->held_a[h] = reinterpret_cast<float *>(take(0));
    ex->held_n[h] = reinterpret_cast<int32_t *>(take(0));
  }
  ex->proposed = reinterpret_cast<int32_t *>(take(0));
  ex->ws_bytes = sizes[i];
  ex->ws = take(0);
  ex->a_ws = take(0);
  ex->v = v;
  ex->p = p;
  ex->a = a;
  ex->device = dev;
  ex->max_rows = max_chunk_rows;
  ex->k = k;
  ex->keep = keep;
  ex->max_rounds = max_rounds;
  *out = ex;
  return ML2_OK;
}

void ml2_stream_explorer_free(ml2_stream_explorer *ex) {
  if (!ex) return;
  int cur = 0;
  const bool other = hipGetDevice(&cur) == hipSuccess && cur != ex->device;
  if (other) (void)hipSetDevice(ex->device);
  (void)hipFree(ex->block);
  if (other) (void)hipSetDevice(cur);
  delete ex;
}

ml2_status ml2_stream_explorer_reset(ml2_stream_explorer *ex) {
  if (!ex) return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_reset: explorer is NULL");
  ex->rounds = 0;
  ex->open = false;
  return ML2_OK;
}

int32_t ml2_stream_explorer_rounds(const ml2_stream_explorer *ex) {
  return ex ? ex->rounds : -1;
}

ml2_status ml2_stream_explorer_begin(ml2_stream_explorer *ex, void *stream) {
  if (!ex) return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_begin: explorer is NULL");
  if (ex->open)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_begin: the round has begun already");
  if (ex->rounds >= ex->max_rounds)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_begin: all %d rounds used (reset first)",
                ex->max_rounds);
  int dev = 0;
  ml2_status st = current_device(&dev);
  if (st != ML2_OK) return st;
  if (dev != ex->device)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_begin: explorer lives on device %d",
                ex->device);
  const int h = ex->cur;
  hipError_t e = ml2::launch_held_reset(ex->held_id[h], ex->held_p[h], ex->held_a[h],
                                        ex->held_n[h], ex->k, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "ml2_stream_explorer_begin: launch");
  ex->open = true;
  return ML2_OK;
}

ml2_status ml2_stream_explorer_chunk(ml2_stream_explorer *ex, const float *X, int64_t m,
                                     int64_t ld, int64_t row0, void *stream) {
  if (!ex) return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_chunk: explorer is NULL");
  if (!ex->open)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_chunk: no round has begun");
  if (m < 0 || m > ex->max_rows)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_chunk: m = %lld outside [0, %lld]",
                (long long)m, (long long)ex->max_rows);
  if (row0 < 0 || row0 + m > (int64_t)INT32_MAX)
    return fail(ML2_ERR_INVALID_ARG,
                "ml2_stream_explorer_chunk: rows [%lld, %lld) outside [0, 2^31-1)",
                (long long)row0, (long long)(row0 + m));
  int dev = 0;
  const ml2_ensemble *models[3] = {ex->v, ex->p, ex->a};
  for (const ml2_ensemble *e : models) {
    if (!e) continue;
    ml2_status st = check_stream_args(e, X, m, ld, X, "ml2_stream_explorer_chunk", &dev);
    if (st != ML2_OK) return st;
  }
  if (m == 0) return ML2_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int cus = cu_count(dev);
  ml2::WalkPlan pv, pp;
  const char *why = nullptr;
  if (!ml2::plan_walk(ex->v->f, m, cus, &pv, &why) ||
      !ml2::plan_walk(ex->p->f, m, cus, &pp, &why, true))
    return fail(ML2_ERR_UNSUPPORTED, "ml2_stream_explorer_chunk: %s", why);
  const int h = ex->cur;
  hipError_t e = ml2::launch_validity(ex->v->f, pv, X, m, ld, ex->valid, nullptr, s);
  if (e == hipSuccess)
    e = ml2::launch_exclude_range(ex->valid, row0, m, ex->proposed, ex->rounds * ex->keep, s);
  if (e == hipSuccess) e = ml2::launch_perf(ex->p->f, pp, X, m, ld, ex->valid, ex->score, s);
  if (e == hipSuccess)
    e = ml2::launch_topk(ex->valid, ex->score, m, ex->k, ex->tk_idx, ex->tk_score, ex->tk_num,
                         ex->ws, cus, s);
  if (e == hipSuccess && ex->a)
    e = ml2::launch_rows(ex->a->f, X, m, ld, ex->tk_idx, ex->k, ex->a_scores, ex->a_ws, cus, s);
  if (e == hipSuccess)
    e = ml2::launch_merge_held(ex->held_id[h], ex->held_p[h], ex->held_a[h], ex->held_n[h],
                               ex->tk_idx, ex->tk_score, ex->a ? ex->a_scores : nullptr,
                               ex->tk_num, row0, ex->k, ex->held_id[1 - h], ex->held_p[1 - h],
                               ex->held_a[1 - h], ex->held_n[1 - h], s);
  if (e != hipSuccess) return hip_fail(e, "ml2_stream_explorer_chunk: launch");
  ex->cur = 1 - h;
  return ML2_OK;
}

ml2_status ml2_stream_explorer_end(ml2_stream_explorer *ex, int32_t *out_idx, float *out_score,
                                   int32_t *num_selected, void *stream) {
  if (!ex) return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_end: explorer is NULL");
  if (!out_idx || !out_score || !num_selected)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_end: NULL output array");
  if (!ex->open) return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_end: no round has begun");
  int dev = 0;
  ml2_status st = current_device(&dev);
  if (st != ML2_OK) return st;
  if (dev != ex->device)
    return fail(ML2_ERR_INVALID_ARG, "ml2_stream_explorer_end: explorer lives on device %d",
                ex->device);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int h = ex->cur;
  // held rows past the held count carry row -1 and are skipped
  hipError_t e = ml2::launch_rerank_select(ex->held_id[h], ex->held_a[h], ex->k, INT32_MAX,
                                           ex->keep, out_idx, out_score, num_selected, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(ex->proposed + (size_t)ex->rounds * ex->keep, out_idx,
                       sizeof(int32_t) * ex->keep, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "ml2_stream_explorer_end: launch");
  ex->rounds += 1;
  ex->open = false;
  return ML2_OK;
}

// ---- tuning overrides (ml2_probe.h) ------------------------------------------

ml2_status ml2_tune_walk_plan(int32_t split, int32_t group, int32_t waves, int32_t nbuf,
                              int32_t chunk) {
  if (split < 0 || split > 2 || group < 0 || group > 16 || waves < 0 || waves > 8 || nbuf < 0 ||
      nbuf > 2 || chunk < 0 || chunk > 4096)
    return fail(ML2_ERR_INVALID_ARG,
                "ml2_tune_walk_plan: split %d, group %d, waves %d, nbuf %d, chunk %d out of range",
                split, group, waves, nbuf, chunk);
  ml2::set_tune(ml2::kTuneSplit, split);
  ml2::set_tune(ml2::kTuneGroup, group);
  ml2::set_tune(ml2::kTuneWaves, waves);
  ml2::set_tune(ml2::kTuneNbuf, nbuf);
  ml2::set_tune(ml2::kTuneChunk, chunk);
  return ML2_OK;
}

ml2_status ml2_tune_layout(int32_t layout) {
  if (layout < 0 || layout > 2)
    return fail(ML2_ERR_INVALID_ARG, "ml2_tune_layout: layout = %d outside [0, 2]", layout);
  ml2::set_tune(ml2::kTuneLayout, layout);
  return ML2_OK;
}

// ---- microbenchmarks (ml2_probe.h) -------------------------------------------

ml2_status ml2_probe_visit(int32_t depth, int32_t trees_per_lane, int32_t lanes_per_candidate,
                           int32_t waves, int32_t features, int32_t iters, int32_t blocks,
                           double *ms, double *visits) {
  ml2_status st = check_probe("ml2_probe_visit", iters, blocks, ms, visits);
  if (st != ML2_OK) return st;
  const int G = trees_per_lane, S = lanes_per_candidate;
  const bool shape_ok = (depth == 6 || depth == 8 || depth == 10) &&
                        (G == 1 || G == 2 || G == 4 || G == 8) && (S == 1 || S == 2) &&
                        waves >= 1 && waves <= 8 && (features == 64 || features == 128);
  if (!shape_ok)
    return fail(ML2_ERR_INVALID_ARG,
                "ml2_probe_visit: shape depth %d, %d trees per lane, %d lanes per candidate, %d "
                "waves, %d features not built",
                depth, G, S, waves, features);
  const size_t lds = (size_t)waves * features * 4 * (64 / S) + (size_t)G * S * ml2::record_bytes(depth);
  if (lds > ml2::kLdsBudget)
    return fail(ML2_ERR_INVALID_ARG, "ml2_probe_visit: %zu bytes of LDS needed (%zu available)",
                lds, (size_t)ml2::kLdsBudget);
  return time_probe("ml2_probe_visit", (size_t)blocks * 512 * sizeof(float), ms, visits,
                    [&](void *out, double *w, hipStream_t s) {
                      return ml2::launch_visit_probe(depth, G, S, waves, features, iters, blocks,
                                                     static_cast<float *>(out), w, s);
                    });
}

ml2_status ml2_probe_lds(int32_t mode, int32_t iters, int32_t blocks, double *ms, double *bytes) {
  ml2_status st = check_probe("ml2_probe_lds", iters, blocks, ms, bytes);
  if (st != ML2_OK) return st;
  if (mode < 0 || mode > 5)
    return fail(ML2_ERR_INVALID_ARG, "ml2_probe_lds: mode = %d outside [0, 5]", mode);
  return time_probe("ml2_probe_lds", (size_t)blocks * 256 * sizeof(uint32_t), ms, bytes,
                    [&](void *out, double *w, hipStream_t s) {
                      return ml2::launch_lds_probe(mode, iters, blocks,
                                                   static_cast<uint32_t *>(out), w, s);
                    });
}

ml2_status ml2_probe_valu(int32_t iters, int32_t blocks, double *ms, double *lane_ops) {
  ml2_status st = check_probe("ml2_probe_valu", iters, blocks, ms, lane_ops);
  if (st != ML2_OK) return st;
  return time_probe("ml2_probe_valu", (size_t)blocks * 256 * sizeof(uint32_t), ms, lane_ops,
                    [&](void *out, double *w, hipStream_t s) {
                      return ml2::launch_valu_probe(iters, blocks, static_cast<uint32_t *>(out),
                                                    w, s);
                    });
}

}  // extern "C"
