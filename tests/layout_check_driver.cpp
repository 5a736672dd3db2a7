// Checked host build of the tree packing (pack.cpp, built with -DML2_CHECKED
// under the address and undefined-behaviour sanitizers): packs random trees
// into the device layout of layout.h and walks every packed tree on the host
// with the kernels' index arithmetic, checking each address against its
// record or slot, each feature index against F, the header fields and the
// leaf chain, and that every walk ends on the leaf the unpacked tree gives
// (bit for bit; missing values by the node's default direction).
//
//   layout_check_driver            all cases; prints one line per case
//   layout_check_driver corrupt    damages packed bytes and expects the
//                                  walker to reject them
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <random>
#include <string>
#include <vector>

#include "pack.h"

using ml2::TreeView;

namespace {

struct Tree {
  std::vector<int32_t> left, right, feat;
  std::vector<float> thr, val;
  std::vector<uint8_t> dl;
  int depth = 0;
  TreeView view() const {
    return TreeView{left.data(), right.data(), feat.data(), thr.data(), val.data(), dl.data(),
                    (int64_t)left.size()};
  }
};

// A random binary tree of `splits` splits and depth <= max_depth: leaves are
// split at random (chains when `chain`), then node ids are shuffled (root
// kept at 0) so that the packing must renumber them.
Tree random_tree(std::mt19937_64 &rng, int splits, int max_depth, int F, bool chain,
                 const std::vector<float> &pool) {
  struct N {
    int l = -1, r = -1, d = 0;
  };
  std::vector<N> nodes(1);
  std::vector<int> leaves{0};
  for (int s = 0; s < splits && !leaves.empty(); ++s) {
    const size_t pick = chain ? leaves.size() - 1 : rng() % leaves.size();
    const int id = leaves[pick];
    if (nodes[id].d >= max_depth) {
      leaves.erase(leaves.begin() + (long)pick);
      --s;
      continue;
    }
    leaves.erase(leaves.begin() + (long)pick);
    const int l = (int)nodes.size(), r = l + 1;
    nodes.push_back({-1, -1, nodes[id].d + 1});
    nodes.push_back({-1, -1, nodes[id].d + 1});
    nodes[id].l = l;
    nodes[id].r = r;
    leaves.push_back(l);
    leaves.push_back(r);
  }
  const int n = (int)nodes.size();
  std::vector<int> perm(n);
  for (int i = 0; i < n; ++i) perm[i] = i;
  for (int i = n - 1; i > 1; --i) std::swap(perm[i], perm[1 + rng() % i]);  // perm[0] = 0
  Tree t;
  t.left.assign(n, -1);
  t.right.assign(n, -1);
  t.feat.assign(n, 0);
  t.thr.assign(n, 0.0f);
  t.val.assign(n, 0.0f);
  t.dl.assign(n, 0);
  std::uniform_real_distribution<float> u(-2.0f, 2.0f);
  for (int i = 0; i < n; ++i) {
    const int p = perm[i];
    if (nodes[i].d > t.depth) t.depth = nodes[i].d;
    if (nodes[i].l < 0) {
      t.val[p] = (rng() % 17 == 0) ? -0.0f : u(rng);
    } else {
      t.left[p] = perm[nodes[i].l];
      t.right[p] = perm[nodes[i].r];
      t.feat[p] = (int32_t)(rng() % (uint64_t)F);
      t.thr[p] = pool[rng() % pool.size()];
      t.dl[p] = (uint8_t)(rng() & 1u);
    }
  }
  return t;
}

// The unpacked tree's leaf for x (x < threshold goes left; a missing value
// goes left where the node's default direction says so when `missing`,
// right otherwise).
float walk_tree(const Tree &t, const float *x, bool missing) {
  int u = 0;
  while (t.left[u] != -1) {
    const float v = x[t.feat[u]];
    const bool left = (v < t.thr[u]) || (missing && isnan(v) && t.dl[u]);
    u = left ? t.left[u] : t.right[u];
  }
  return t.val[u];
}

uint32_t word(const char *base, size_t at) {
  uint32_t w;
  memcpy(&w, base + at, 4);
  return w;
}

bool same_bits(float a, float b) { return memcmp(&a, &b, 4) == 0; }

#define REQUIRE(cond)                                                                 \
  do {                                                                                \
    if (!(cond)) {                                                                    \
      snprintf(why, sizeof why, "line %d: %s", __LINE__, #cond);                      \
      return false;                                                                   \
    }                                                                                 \
  } while (0)

char why[256];

// The perfect walk: D levels of u <- 2u + [x < t] from u = 1, then the leaf
// at byte 4L + 4u (the validity and perf kernels' index arithmetic).
bool walk_perfect(const char *rec, int D, int F, const float *x, float *out) {
  const uint32_t L = 1u << D;
  const size_t cap = ml2::record_bytes(D);
  uint32_t u = 1;
  for (int l = 0; l < D; ++l) {
    REQUIRE(u >= 1 && u < L && 8u * u + 8u <= cap);
    const uint32_t f = word(rec, 8u * u);
    REQUIRE(f < (uint32_t)F);
    float t;
    memcpy(&t, rec + 8u * u + 4u, 4);
    u = 2u * u + ((x[f] < t) ? 1u : 0u);
  }
  REQUIRE(u >= L && u < 2u * L && 4u * L + 4u * u + 4u <= cap);
  memcpy(out, rec + 4u * L + 4u * u, 4);
  return true;
}

// The ragged walk of tree i of a slot, as the kernels step it: a split's
// word 0 holds the default direction (bit 31), the offset to the left child
// (bits 30..16, signed) and the feature's byte offset in a 256-byte tile row
// (bits 15..0); a leaf's holds offset -1 and the byte offset of the next
// tree's root.  Returns the leaf value; checks that the walk stays in the
// slot and in the tree, ends within `depth` splits and hands over to the
// next root.
bool walk_ragged(const char *slot, size_t i, int F, const float *x, float *out) {
  constexpr size_t CAP = ml2::kRaggedChunkBytes;
  const uint32_t ntr = word(slot, 0), depth = word(slot, 4), sentinel = word(slot, 8);
  const uint32_t head = (uint32_t)((16 + 4 * (ntr + 2) + 15) & ~15u);
  REQUIRE(i < ntr);
  uint32_t u = word(slot, 16 + 4 * i);
  const uint32_t next_root = word(slot, 16 + 4 * (i + 1));
  REQUIRE(u >= head / 8u && u < next_root && next_root <= sentinel);
  for (uint32_t steps = 0;; ++steps) {
    REQUIRE(steps <= depth);
    REQUIRE(8u * u + 8u <= CAP && u >= head / 8u && u < next_root);
    const uint32_t w0 = word(slot, 8u * u);
    const int32_t off = (int32_t)(w0 << 1) >> 17;  // bits 30..16, signed
    if ((w0 >> 16) == 0x7FFFu) {                     // a leaf
      REQUIRE((w0 & 0xFFFFu) == 8u * next_root);
      REQUIRE((int64_t)u + off + 1 == (int64_t)u);  // "go right" stays on the leaf
      memcpy(out, slot + 8u * u + 4u, 4);
      return true;
    }
    REQUIRE((w0 & 0xFFu) == 0u);
    const uint32_t f = (w0 & 0xFFFFu) >> 8;
    REQUIRE(f < (uint32_t)F && 256u * f + 4u <= 256u * (uint32_t)F);
    float t;
    memcpy(&t, slot + 8u * u + 4u, 4);
    const float v = x[f];
    const bool dl = (w0 >> 31) != 0;
    const bool right = !(v < t) && !(dl && isnan(v));
    REQUIRE(off >= 1);
    u = (uint32_t)((int64_t)u + off + (right ? 1 : 0));
  }
}

std::vector<float> inputs(std::mt19937_64 &rng, int F, const std::vector<float> &pool,
                          bool nans) {
  std::vector<float> x((size_t)F);
  std::uniform_real_distribution<float> u(-2.5f, 2.5f);
  for (int f = 0; f < F; ++f) {
    const uint64_t r = rng() % 20;
    x[(size_t)f] = r < 6    ? pool[rng() % pool.size()]  // ties with thresholds
                   : r < 8  ? (nans ? NAN : 0.0f)
                   : r == 8 ? -0.0f
                   : r == 9 ? (rng() & 1 ? INFINITY : -INFINITY)
                            : u(rng);
  }
  return x;
}

struct Case {
  const char *name;
  int trees, F, max_depth, min_splits, max_splits;
  bool chain;
};

bool run_perfect(const Case &c, uint64_t seed, bool corrupt) {
  std::mt19937_64 rng(seed);
  std::vector<float> pool;
  for (int i = 0; i < 64; ++i) pool.push_back(std::uniform_real_distribution<float>(-2, 2)(rng));
  pool.push_back(0.0f);
  pool.push_back(-0.0f);
  std::vector<Tree> trees;
  int D = 1;
  for (int t = 0; t < c.trees; ++t) {
    const int s = c.min_splits + (int)(rng() % (uint64_t)(c.max_splits - c.min_splits + 1));
    trees.push_back(random_tree(rng, s, c.max_depth, c.F, c.chain, pool));
    if (trees.back().depth > D) D = trees.back().depth;
  }
  const size_t rb = ml2::record_bytes(D);
  const int tpad = (c.trees + ml2::kTreePad - 1) / ml2::kTreePad * ml2::kTreePad;
  std::vector<char> bytes((size_t)tpad * rb, 0);
  for (int t = 0; t < tpad; ++t) {
    if (t < c.trees)
      ml2::pad_tree(trees[(size_t)t].view(), D, bytes.data() + (size_t)t * rb);
    else
      ml2::pad_identity_tree(D, bytes.data() + (size_t)t * rb);
  }
  if (corrupt) {  // a node's feature index beyond F, then a walk that reaches it
    const uint32_t bad = (uint32_t)c.F + 3u;
    memcpy(bytes.data() + 8, &bad, 4);  // tree 0, node 1 (the root)
  }
  for (int r = 0; r < 200; ++r) {
    const std::vector<float> x = inputs(rng, c.F, pool, false);
    for (int t = 0; t < tpad; ++t) {
      float got;
      if (!walk_perfect(bytes.data() + (size_t)t * rb, D, c.F, x.data(), &got)) return false;
      const float want = t < c.trees ? walk_tree(trees[(size_t)t], x.data(), false) : -0.0f;
      if (!same_bits(got, want)) {
        snprintf(why, sizeof why, "tree %d: leaf %a, unpacked tree %a", t, got, want);
        return false;
      }
    }
  }
  return true;
}

bool run_ragged(const Case &c, uint64_t seed, bool corrupt) {
  std::mt19937_64 rng(seed);
  std::vector<float> pool;
  for (int i = 0; i < 64; ++i) pool.push_back(std::uniform_real_distribution<float>(-2, 2)(rng));
  pool.push_back(0.0f);
  pool.push_back(-0.0f);
  std::vector<Tree> trees;
  std::vector<TreeView> views;
  std::vector<int> depths;
  for (int t = 0; t < c.trees; ++t) {
    const int s = c.min_splits + (int)(rng() % (uint64_t)(c.max_splits - c.min_splits + 1));
    trees.push_back(random_tree(rng, s, c.max_depth, c.F, c.chain, pool));
  }
  for (const Tree &t : trees) {
    views.push_back(t.view());
    depths.push_back(t.depth);
  }
  ml2::RaggedPack pk;
  ml2::pack_ragged(views, depths, &pk);
  constexpr size_t CAP = ml2::kRaggedChunkBytes;
  if ((size_t)pk.slots * CAP != pk.bytes.size()) {
    snprintf(why, sizeof why, "%d slots in %zu bytes", pk.slots, pk.bytes.size());
    return false;
  }
  if (corrupt) {  // the first tree's root: a split's left-child offset past
                  // its tree, or a leaf's next-root offset one node on
    char *slot = pk.bytes.data();
    const uint32_t root = word(slot, 16);
    uint32_t w0 = word(slot, 8u * root);
    w0 = (w0 >> 16) == 0x7FFFu ? w0 + 8u : (w0 & 0x8000FFFFu) | (0x3000u << 16);
    memcpy(slot + 8u * root, &w0, 4);
  }
  // header fields: trees per slot (whole groups), global index of the first
  size_t t = 0;
  int32_t index = 0;
  std::vector<std::pair<size_t, size_t>> place;  // slot, position of each real tree
  for (int32_t s = 0; s < pk.slots; ++s) {
    const char *slot = pk.bytes.data() + (size_t)s * CAP;
    const uint32_t ntr = word(slot, 0), first = word(slot, 12);
    if (ntr == 0 || ntr % ml2::kRaggedGroup != 0 || (int32_t)first != index) {
      snprintf(why, sizeof why, "slot %d header {%u trees, first %u}", s, ntr, first);
      return false;
    }
    index += (int32_t)ntr;
  }
  if (index != pk.trees) {
    snprintf(why, sizeof why, "%d trees in the slots, %d reported", index, pk.trees);
    return false;
  }
  // real trees in order, each slot's before its padding (a padding tree is
  // one node, so real trees of three or more nodes are told apart by span)
  for (int32_t s = 0; s < pk.slots && t < trees.size(); ++s) {
    const char *slot = pk.bytes.data() + (size_t)s * CAP;
    const uint32_t ntr = word(slot, 0);
    uint32_t i = 0;
    uint32_t maxd = 0;
    while (i < ntr && t < trees.size()) {
      const uint32_t root = word(slot, 16 + 4 * i), next = word(slot, 16 + 4 * (i + 1));
      if ((int64_t)(next - root) != (int64_t)trees[t].left.size()) break;
      place.emplace_back((size_t)s, (size_t)i);
      if ((uint32_t)trees[t].depth > maxd) maxd = (uint32_t)trees[t].depth;
      ++i;
      ++t;
    }
    for (uint32_t j = i; j < ntr; ++j) {  // padding trees: single -0.0 leaves
      const uint32_t root = word(slot, 16 + 4 * j), next = word(slot, 16 + 4 * (j + 1));
      if (next != root + 1u || word(slot, 8u * root + 4u) != 0x80000000u) {
        snprintf(why, sizeof why, "slot %d position %u: expected a padding leaf", s, j);
        return false;
      }
    }
    if (word(slot, 4) != maxd) {
      snprintf(why, sizeof why, "slot %d: depth %u, deepest tree %u", s, word(slot, 4), maxd);
      return false;
    }
  }
  if (t != trees.size()) {
    snprintf(why, sizeof why, "%zu of %zu trees found in the slots", t, trees.size());
    return false;
  }
  for (int r = 0; r < 100; ++r) {
    const std::vector<float> x = inputs(rng, c.F, pool, true);
    for (size_t k = 0; k < trees.size(); ++k) {
      float got;
      const char *slot = pk.bytes.data() + place[k].first * CAP;
      if (!walk_ragged(slot, place[k].second, c.F, x.data(), &got)) return false;
      const float want = walk_tree(trees[k], x.data(), true);
      if (!same_bits(got, want)) {
        snprintf(why, sizeof why, "tree %zu: leaf %a, unpacked tree %a", k, got, want);
        return false;
      }
    }
  }
  return true;
}

}  // namespace

int main(int argc, char **argv) {
  const bool corrupt = argc > 1 && std::string(argv[1]) == "corrupt";
  // name, trees, F, max depth, splits (min, max), chain
  const Case perfect[] = {
      {"perfect stumps", 5, 1, 1, 0, 1, false},
      {"perfect depth 6, F 40", 70, 40, 6, 1, 40, false},
      {"perfect depth 10, F 64", 9, 64, 10, 200, 600, false},
      {"perfect depth 12, F 256", 3, 256, 12, 1000, 3000, false},
      {"perfect chains depth 12", 4, 7, 12, 12, 12, true},
  };
  const Case ragged[] = {
      {"ragged single leaves", 9, 3, 14, 0, 0, false},
      {"ragged ~100 nodes depth 14, F 64", 300, 64, 14, 30, 70, false},
      {"ragged chains depth 32", 40, 5, 32, 32, 32, true},
      {"ragged largest trees (3062 nodes)", 3, 256, 32, 1530, 1530, false},
      {"ragged mixed sizes, F 256", 120, 256, 20, 1, 400, false},
  };
  int failed = 0;
  uint64_t seed = 1;
  for (const Case &c : perfect) {
    why[0] = 0;
    const bool ok = run_perfect(c, seed++, corrupt);
    printf("%s %s%s%s\n", ok ? "ok" : "FAIL", c.name, ok ? "" : ": ", ok ? "" : why);
    failed += ok == corrupt;
  }
  for (const Case &c : ragged) {
    why[0] = 0;
    const bool ok = run_ragged(c, seed++, corrupt);
    printf("%s %s%s%s\n", ok ? "ok" : "FAIL", c.name, ok ? "" : ": ", ok ? "" : why);
    failed += ok == corrupt;
  }
  if (corrupt) printf("%s\n", failed ? "corruption NOT detected" : "corruption detected in every case");
  return failed ? 1 : 0;
}
