// C-ABI entry points: argument validation, ensemble loading (validation,
// padding to perfect trees, packing into the device tree records) and the
// launches.  Everything here runs on the host; the arithmetic of the method
// runs in walk_kernels.hip and topk_kernels.hip.
#include <float.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ml2_internal.h"

struct ml2_ensemble {
  ml2::Forest f;
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

// ---- descriptor validation and padding ------------------------------------

struct TreeView {
  const int32_t *left, *right, *feat;
  const float *thr, *val;
  int64_t size;
};

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

// Fill the perfect-tree record of depth D from the general tree (replicating
// leaves that sit above depth D into dummy subtrees).
void pad_tree(const TreeView &tv, int D, char *rec) {
  const uint32_t L = 1u << D;
  uint2 *nodes = reinterpret_cast<uint2 *>(rec);              // nodes[j], 1 <= j < L
  float *leaves = reinterpret_cast<float *>(rec + 4u * L);    // leaves[j], L <= j < 2L
  struct Item {
    int32_t node;
    uint32_t pos;
  };
  std::vector<Item> stack;
  stack.push_back({0, 1u});
  while (!stack.empty()) {
    const Item it = stack.back();
    stack.pop_back();
    const bool leaf = tv.left[it.node] == -1 && tv.right[it.node] == -1;
    if (it.pos >= L) {  // only leaves reach depth D
      leaves[it.pos] = tv.val[it.node];
      continue;
    }
    if (leaf) {
      nodes[it.pos] = make_uint2(0u, 0u);  // feature 0, threshold +0: both sides equal
      stack.push_back({it.node, 2 * it.pos});
      stack.push_back({it.node, 2 * it.pos + 1});
    } else {
      uint32_t tb;
      memcpy(&tb, &tv.thr[it.node], 4);
      nodes[it.pos] = make_uint2((uint32_t)tv.feat[it.node], tb);
      stack.push_back({tv.left[it.node], 2 * it.pos + 1});
      stack.push_back({tv.right[it.node], 2 * it.pos});
    }
  }
}

void pad_identity_tree(int D, char *rec) {  // every leaf -0.0
  const uint32_t L = 1u << D;
  float *leaves = reinterpret_cast<float *>(rec + 4u * L);
  for (uint32_t j = L; j < 2 * L; ++j) leaves[j] = -0.0f;
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
  std::vector<TreeView> views((size_t)d.num_trees);
  for (int32_t t = 0; t < d.num_trees; ++t) {
    const int64_t a = d.tree_node_offset[t], b = d.tree_node_offset[t + 1];
    if (b <= a || b - a > (int64_t)INT32_MAX)
      return fail(ML2_ERR_INVALID_ARG, "tree %d: node range [%lld, %lld) is empty or too large",
                  t, (long long)a, (long long)b);
    TreeView tv{d.left_child + a, d.right_child + a, d.split_feature + a,
                d.split_threshold + a, d.leaf_value + a, b - a};
    int dt = 0;
    ml2_status st = check_tree(d, t, tv, &dt, &max_leaf);
    if (st != ML2_OK) return st;
    if (dt > depth) depth = dt;
    views[(size_t)t] = tv;
  }
  if ((double)d.num_trees * max_leaf + fabs((double)d.base_score) >= (double)FLT_MAX / 2)
    return fail(ML2_ERR_INVALID_ARG, "num_trees * max|leaf| + |base| may overflow float32");

  ml2::Forest f{};
  ml2_status st = current_device(&f.device);
  if (st != ML2_OK) return st;
  f.num_trees = d.num_trees;
  f.num_trees_padded = (d.num_trees + ml2::kTreePad - 1) / ml2::kTreePad * ml2::kTreePad;
  f.num_features = d.num_features;
  f.depth = depth;
  f.base = d.base_score;
  f.rec_bytes = ml2::record_bytes(depth);
  const size_t bytes = (size_t)f.num_trees_padded * f.rec_bytes;
  std::vector<char> host;
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
  if (hipGetDevice(&cur) == hipSuccess && cur != e->f.device) {
    (void)hipSetDevice(e->f.device);
    (void)hipDeviceSynchronize();
    (void)hipFree(e->f.d_trees);
    (void)hipSetDevice(cur);
  } else {
    (void)hipDeviceSynchronize();
    (void)hipFree(e->f.d_trees);
  }
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
  if (!ml2::plan_walk(p_ens->f, n, cu_count(dev), &p, &why))
    return fail(ML2_ERR_UNSUPPORTED, "ml2_score_perf: %s", why);
  hipError_t e = ml2::launch_perf(p_ens->f, p, X, n, ld, valid, score_out,
                                  static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "perf kernel launch");
  return ML2_OK;
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

ml2_status ml2_rerank(const ml2_ensemble *a, const float *X, int64_t n, int64_t ld,
                      const int32_t *rows, int32_t m, int32_t keep, float *row_scores,
                      int32_t *out_idx, float *out_score, int32_t *num_selected, void *stream) {
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
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (m > 0 && n > 0) {
    ml2::WalkPlan p;
    const char *why = nullptr;
    if (!ml2::plan_walk(a->f, m, cu_count(dev), &p, &why))
      return fail(ML2_ERR_UNSUPPORTED, "ml2_rerank: %s", why);
    hipError_t e = ml2::launch_rows(a->f, p, X, n, ld, rows, m, row_scores, s);
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

}  // extern "C"
