// Internal declarations shared by the host entry points and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ml2.h"

namespace ml2 {

// Device form of an ensemble.  Every tree is padded to a perfect tree of the
// ensemble's depth D (a leaf above depth D is replicated into a dummy subtree
// whose every split leads to the same value, which leaves every walk's result
// unchanged), and the tree count is padded to a multiple of kTreePad with
// trees whose leaves are -0.0 (x + (-0.0) == x for every float x, so the
// fold is unchanged).
//
// Tree record (rec_bytes, 16-byte aligned), breadth-first, 0-based heap:
//   node[i]  i in [0, 2^D - 1): uint2 {feature index, threshold bits}
//   leaf[j]  j in [0, 2^D):     float, at byte 8 * (2^D - 1) + 4 * j
// Children of node i are 2i+1 (taken iff x[feature] < threshold) and 2i+2.
constexpr int kTreePad = 8;

inline constexpr uint32_t record_bytes(int depth) {
  const uint32_t ni = (1u << depth) - 1u;
  const uint32_t raw = 8u * ni + 4u * (ni + 1u);
  return (raw + 15u) & ~15u;
}

struct Forest {
  int device;
  int32_t num_trees;        // trees in the descriptor
  int32_t num_trees_padded; // multiple of kTreePad
  int32_t num_features;
  int32_t depth;            // D >= 1
  float base;
  uint32_t rec_bytes;
  void *d_trees;            // num_trees_padded * rec_bytes bytes
};

// Launch parameters of a walk (chosen on the host from D and F).
struct WalkPlan {
  int waves;        // waves per workgroup; each wave owns 64 candidates
  int group;        // trees walked concurrently per lane (ILP)
  int chunk_trees;  // trees per LDS chunk (multiple of group)
  int nbuf;         // chunk buffers: 2 (double-buffered) or 1
  size_t lds_bytes; // dynamic LDS per workgroup
  int grid;         // workgroups
};

// Returns false (and sets *why) if no plan fits the LDS of one workgroup.
bool plan_walk(const Forest &f, int64_t n_work, int cu_count, WalkPlan *plan, const char **why);

hipError_t launch_validity(const Forest &f, const WalkPlan &p, const float *X, int64_t n,
                           int64_t ld, uint8_t *valid_out, float *margin_out, hipStream_t s);
hipError_t launch_perf(const Forest &f, const WalkPlan &p, const float *X, int64_t n,
                       int64_t ld, const uint8_t *valid, float *score_out, hipStream_t s);

size_t topk_workspace_bytes(int64_t n, int32_t k);
hipError_t launch_topk(const uint8_t *valid, const float *scores, int64_t n, int32_t k,
                       int32_t *idx, float *score, int32_t *num, void *ws, int cu_count,
                       hipStream_t s);

}  // namespace ml2
