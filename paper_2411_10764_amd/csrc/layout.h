// Byte layout of an ensemble in device memory: the contract between the
// host packing (pack.cpp) and the walk kernels.  Plain C++ (no HIP), so the
// packing also builds on its own for the checked host build.
#pragma once

#include <stdint.h>

namespace ml2 {

// Device form of an ensemble.  Every tree is padded to a perfect tree of the
// ensemble's depth D (a leaf above depth D is replicated into a dummy subtree
// whose every split leads to the same value, which leaves every walk's result
// unchanged), and the tree count is padded to a multiple of kTreePad with
// trees whose leaves are -0.0 (x + (-0.0) == x for every float x, so the
// fold is unchanged).
//
// Tree record (rec_bytes bytes, 16-byte aligned), 1-based heap of depth D,
// with L = 2^D:
//   node j, 1 <= j < L  at byte 8*j:      uint2 {feature index, threshold bits}
//   leaf j, L <= j < 2L at byte 4*L + 4*j: float   (byte 8*L .. 12*L)
// The children of node j are 2j+1, taken iff x[feature] < threshold, and 2j,
// taken otherwise, so a walk moves with u <- 2u + [x < t].  Byte 0..7 is
// unused.
constexpr int kTreePad = 16;  // >= the trees of the largest walk group
constexpr int kMaxPerfectDepth = 12;  // deeper ensembles use the ragged layout

// Ragged layout (deep or sparse trees, or per-node default directions for
// missing values): the ensemble is cut into chunks of whole trees, each in a
// fixed slot of kRaggedChunkBytes bytes:
//   byte 0   uint4 {trees in the chunk (a multiple of kRaggedGroup), deepest
//            path of those trees, the sentinel's node index, global index of
//            the chunk's first tree}
//   byte 16  uint32 root node index of each tree (node u at byte 8u of the
//            slot), then two entries that point to the sentinel
//   then 8-byte nodes, each tree breadth-first (siblings adjacent):
//     split: word 0 bit 31 default-left, bits 30..16 signed offset in nodes
//            from the node to its left child (the right child follows it;
//            trees have at most 3062 nodes), bits 15..8 split feature,
//            bits 7..0 zero (bits 15..0: the feature's byte offset in a
//            256-byte-row tile); word 1 threshold bits
//     leaf:  word 0 bits 31..16 0x7FFF (offset -1), bits 15..0 the byte
//            offset in the slot of the next tree's root node (the
//            sentinel's after the last tree; the sentinel's own); word 1 the
//            leaf value.  A walk treats a leaf as "go right", i.e. onto
//            itself, so a lockstep walk may run past it
// Trees padded onto a chunk are single leaves of value -0.0; the sentinel,
// after the last tree, is one more such leaf.
constexpr uint32_t kRaggedChunkBytes = 24 * 1024;
constexpr int kRaggedGroup = 4;

// Bytes of one staged record: a perfect tree of `depth` levels, or (depth 0)
// one ragged chunk slot.
inline constexpr uint32_t record_bytes(int depth) {
  if (depth == 0) return kRaggedChunkBytes;
  const uint32_t raw = 12u << depth;
  return (raw + 15u) & ~15u;
}

}  // namespace ml2
