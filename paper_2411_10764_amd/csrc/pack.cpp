// Host packing of trees into the device layout (layout.h).  Built with
// -DML2_CHECKED, every byte written is first checked to lie inside its record
// or slot and every encoded field to fit its bits (the checked host build,
// run under the address and undefined-behaviour sanitizers by the tests).
#include "pack.h"

#include <string.h>

#ifdef ML2_CHECKED
#include <stdio.h>
#include <stdlib.h>
#define ML2_CHECK(cond)                                                                   \
  do {                                                                                    \
    if (!(cond)) {                                                                        \
      fprintf(stderr, "%s:%d: layout check failed: %s\n", __FILE__, __LINE__, #cond);     \
      abort();                                                                            \
    }                                                                                     \
  } while (0)
#else
#define ML2_CHECK(cond) \
  do {                  \
  } while (0)
#endif

namespace ml2 {
namespace {

uint32_t float_bits(float v) {
  uint32_t b;
  memcpy(&b, &v, 4);
  return b;
}

// The 8-byte node {w0, w1} at byte `at` of a buffer of `cap` bytes.
void put_node(char *base, size_t cap, size_t at, uint32_t w0, uint32_t w1) {
  ML2_CHECK(at % 8 == 0 && at + 8 <= cap);
  (void)cap;
  const uint32_t w[2] = {w0, w1};
  memcpy(base + at, w, 8);
}

void put_word(char *base, size_t cap, size_t at, uint32_t w) {
  ML2_CHECK(at % 4 == 0 && at + 4 <= cap);
  (void)cap;
  memcpy(base + at, &w, 4);
}

}  // namespace

void pad_tree(const TreeView &tv, int D, char *rec) {
  const uint32_t L = 1u << D;
  const size_t cap = record_bytes(D);
  struct Item {
    int32_t node;
    uint32_t pos;  // heap position, 1-based
  };
  std::vector<Item> stack;
  stack.push_back({0, 1u});
  while (!stack.empty()) {
    const Item it = stack.back();
    stack.pop_back();
    ML2_CHECK(it.node >= 0 && it.node < tv.size && it.pos >= 1 && it.pos < 2 * L);
    const bool leaf = tv.left[it.node] == -1 && tv.right[it.node] == -1;
    if (it.pos >= L) {  // only leaves reach depth D
      ML2_CHECK(leaf);
      put_word(rec, cap, 4u * L + 4u * it.pos, float_bits(tv.val[it.node]));  // byte 8L .. 12L
      continue;
    }
    if (leaf) {  // feature 0, threshold +0: both sides lead to the same value
      put_node(rec, cap, 8u * it.pos, 0u, 0u);
      stack.push_back({it.node, 2 * it.pos});
      stack.push_back({it.node, 2 * it.pos + 1});
    } else {
      put_node(rec, cap, 8u * it.pos, (uint32_t)tv.feat[it.node], float_bits(tv.thr[it.node]));
      stack.push_back({tv.left[it.node], 2 * it.pos + 1});  // taken iff x < threshold
      stack.push_back({tv.right[it.node], 2 * it.pos});
    }
  }
}

void pad_identity_tree(int D, char *rec) {
  const uint32_t L = 1u << D;
  const size_t cap = record_bytes(D);
  for (uint32_t j = L; j < 2 * L; ++j) put_word(rec, cap, 4u * L + 4u * j, float_bits(-0.0f));
}

void pack_ragged(const std::vector<TreeView> &views, const std::vector<int> &depths,
                 RaggedPack *out) {
  constexpr uint32_t CAP = kRaggedChunkBytes;
  constexpr int GRP = kRaggedGroup;
  // a leaf's first word: offset -1 (the node itself) and, in the low half,
  // the byte offset in the slot of the next tree's root (the sentinel after
  // the last tree)
  auto leaf_word0 = [](uint32_t next_root) {
    ML2_CHECK(8u * next_root + 8u <= CAP && 8u * next_root <= 0xFFFFu);
    return (0x7FFFu << 16) | (8u * next_root);
  };
  size_t t = 0;
  int32_t tree_index = 0;
  while (t < views.size()) {
    // choose the trees of this slot: header + roots + 8 bytes per node,
    // with room left for padding the tree count to a multiple of GRP
    // (two more root entries and one more node: the sentinel)
    size_t first = t, nodes = 0;
    auto need = [&](size_t ntrees, size_t nnodes) {
      const size_t ntr = (ntrees + GRP - 1) / GRP * GRP;
      const size_t head = (16 + 4 * (ntr + 2) + 15) & ~(size_t)15;
      return head + 8 * (nnodes + (ntr - ntrees) + 1);
    };
    while (t < views.size() && need(t + 1 - first, nodes + (size_t)views[t].size) <= CAP) {
      nodes += (size_t)views[t].size;
      ++t;
    }
    const size_t real = t - first;
    ML2_CHECK(real >= 1);  // every tree fits a slot of its own
    const size_t ntr = (real + GRP - 1) / GRP * GRP;
    const uint32_t head = (uint32_t)((16 + 4 * (ntr + 2) + 15) & ~(size_t)15);
    const size_t slot0 = out->bytes.size();
    out->bytes.resize(slot0 + CAP, 0);
    char *slot = out->bytes.data() + slot0;
    auto put_root = [&](size_t i, uint32_t u) {
      ML2_CHECK(16 + 4 * (i + 1) <= head);
      put_word(slot, CAP, 16 + 4 * i, u);
    };
    auto put = [&](uint32_t j, uint32_t w0, uint32_t w1) {  // node j of the slot's node array
      put_node(slot, CAP, head + 8 * (size_t)j, w0, w1);
    };
    int depth = 0;
    uint32_t next = 0;  // next free node index in the slot's node array
    std::vector<int32_t> order;
    for (size_t i = 0; i < ntr; ++i) {
      put_root(i, head / 8u + next);
      if (i >= real) {  // padding: one leaf of value -0.0
        put(next, leaf_word0(head / 8u + next + 1), float_bits(-0.0f));
        ++next;
        continue;
      }
      const TreeView &tv = views[first + i];
      if (depths[first + i] > depth) depth = depths[first + i];
      // breadth-first ids: order[k] = original node of new id k
      order.assign(1, 0);
      std::vector<int32_t> newid((size_t)tv.size, -1);
      newid[0] = 0;
      for (size_t k = 0; k < order.size(); ++k) {
        const int32_t o = order[k];
        if (tv.left[o] == -1) continue;
        newid[(size_t)tv.left[o]] = (int32_t)order.size();
        order.push_back(tv.left[o]);
        newid[(size_t)tv.right[o]] = (int32_t)order.size();
        order.push_back(tv.right[o]);
      }
      ML2_CHECK((int64_t)order.size() == tv.size);
      for (size_t k = 0; k < order.size(); ++k) {
        const int32_t o = order[k];
        const uint32_t j = next + (uint32_t)k;
        if (tv.left[o] == -1) {
          put(j, leaf_word0(head / 8u + next + (uint32_t)order.size()), float_bits(tv.val[o]));
        } else {
          const int32_t rel = newid[(size_t)tv.left[o]] - (int32_t)k;  // nodes, > 0
          ML2_CHECK(rel >= 1 && rel <= 0x3FFF);                         // 15-bit signed field
          ML2_CHECK(newid[(size_t)tv.right[o]] == newid[(size_t)tv.left[o]] + 1);
          ML2_CHECK(tv.feat[o] >= 0 && tv.feat[o] < 256);
          const uint32_t dl = (tv.dl && tv.dl[o]) ? 1u : 0u;
          put(j,
              (dl << 31) | (((uint32_t)rel & 0x7FFFu) << 16) | ((uint32_t)tv.feat[o] << 8),
              float_bits(tv.thr[o]));
        }
      }
      next += (uint32_t)order.size();
    }
    // the sentinel: a leaf of value -0.0 that the two entries after the last
    // root point to (a walk past its last tree moves onto it; adding -0.0
    // changes no float)
    const uint32_t sentinel = head / 8u + next;
    put(next, leaf_word0(sentinel), float_bits(-0.0f));
    put_root(ntr, sentinel);
    put_root(ntr + 1, sentinel);
    ++next;
    const uint32_t hdr[4] = {(uint32_t)ntr, (uint32_t)depth, sentinel, (uint32_t)tree_index};
    memcpy(slot, hdr, sizeof hdr);
    tree_index += (int32_t)ntr;
    if (depth > out->depth) out->depth = depth;
    out->slots += 1;
  }
  out->trees = tree_index;
}

}  // namespace ml2
