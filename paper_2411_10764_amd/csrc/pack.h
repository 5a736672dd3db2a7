// Host packing of validated trees into the device layout of layout.h.
// Plain C++17 (no HIP): the library links it, and the checked host build
// (-DML2_CHECKED, under the address and undefined-behaviour sanitizers)
// compiles it on its own to test every index it writes.
#pragma once

#include <stdint.h>

#include <vector>

#include "layout.h"

namespace ml2 {

// One tree of a descriptor: node arrays of `size` entries, node 0 the root,
// leaves marked by left == right == -1 (the caller has checked that the
// nodes form one binary tree and that features lie in [0, 256)).
struct TreeView {
  const int32_t *left, *right, *feat;
  const float *thr, *val;
  const uint8_t *dl;  // NULL: every missing value goes right
  int64_t size;
};

// Fill the perfect-tree record of depth D (record_bytes(D) zeroed bytes at
// rec) from a tree of depth <= D, replicating leaves that sit above depth D
// into dummy subtrees.
void pad_tree(const TreeView &tv, int D, char *rec);

// A record of depth D whose every leaf is -0.0 (pads the tree count).
void pad_identity_tree(int D, char *rec);

// Trees packed into fixed chunk slots of kRaggedChunkBytes (breadth-first,
// siblings adjacent).  depths[i]: the deepest path of views[i].  Every tree
// must fit one slot with its header (the caller checks the node count).
struct RaggedPack {
  std::vector<char> bytes;
  int32_t slots = 0;
  int32_t trees = 0;  // with the padding trees
  int32_t depth = 0;  // deepest path over all trees
};
void pack_ragged(const std::vector<TreeView> &views, const std::vector<int> &depths,
                 RaggedPack *out);

}  // namespace ml2
