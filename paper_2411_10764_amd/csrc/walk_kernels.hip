// Tree-ensemble walks on gfx950: the validity filter (model V) and the
// performance prediction over accepted candidates (model P) of ML2Tuner's
// configuration explorer (Section 2, "ML Model P" / "ML Model V").
//
// Mapping (one workgroup = W waves, persistent over the pool):
//   * Each wave owns a tile of 64/S candidates whose features sit in LDS
//     transposed: feature f of candidate c at f * (256/S) + 4c, so the
//     per-level feature reads of a wave hit distinct banks whatever features
//     the lanes' current nodes test.
//   * S = 1: lane = candidate.  S = 2: lanes c and c+32 hold candidate c; the
//     lower half-wave walks the first G trees of every group of 2G, the upper
//     half the next G, and the lower half folds both (the upper half's leaves
//     cross over with one v_permlane32_swap per tree).  Splitting halves the
//     tile of a wave, so twice as many waves fit the LDS and every SIMD runs
//     two: one wave's VALU work issues while the other's LDS reads do.
//   * All lanes of a half-wave walk the same trees in lockstep (the trees are
//     perfect), so at level l a tree is touched only at its 2^l
//     breadth-ordered nodes of that level.
//   * The ensemble streams through one LDS buffer in chunks of whole trees.
//     The next chunks are fetched into registers while the current one is
//     walked, then written to LDS between two barriers.  An ensemble that
//     fits one chunk stays resident, and with S = 2 the staging registers
//     then carry the next round's rows instead.
//   * Rows are fetched for the next round while the current one is walked
//     (aligned rows of at most 128 features), one candidate per lane, so
//     that each lane writes its own column of the transposed tile.
//   * Each lane walks G trees at once, as two halves offset by half a level:
//     while one half waits for its node (or feature) reads, the other half
//     issues its own.  Leaves are added to the running margin in tree-index
//     order, so the float32 left fold is exactly the defined one.
//   * Per level a walk costs two LDS reads (node, feature value) and four
//     VALU instructions (node address, feature address, compare, and one
//     add-with-carry that moves to child 2u + [x < t]).
//   * The performance pass compacts the accepted candidates of the pool into
//     an LDS queue (wave ballots + a workgroup prefix) and only ever walks
//     full tiles of accepted candidates; rejected ones get -inf directly.
#include <math.h>
#include <stdlib.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "ml2_internal.h"

namespace ml2 {
namespace {

constexpr int kLanes = 64;
constexpr int kMaxWaves = 8;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Tile geometry for S lanes per candidate.
template <int S>
struct Geo {
  static constexpr int kCand = kLanes / S;            // candidates per wave
  static constexpr uint32_t kRowBytes = 4u * kCand;   // one feature of a tile
  static constexpr int kRowShift = S == 1 ? 8 : 7;    // log2(kRowBytes)
};

// 16-byte registers per thread that stage one chunk: 6 / S, and 8 with one
// lane per candidate for trees of depth 10 or more (12 KiB records), so that
// six waves stage a chunk of four of them; such kernels keep two chunks in
// registers instead of three (the register file holds no more).
constexpr int stage_regs(int D, int S) { return (S == 1 && D >= 10) ? 8 : 6 / S; }
constexpr int stage_sets(int D, int S, int sets) { return (S == 1 && D >= 10) ? 2 : sets; }

struct WalkArgs {
  const float *X;
  int64_t n;            // entries: pool rows, or list entries
  int64_t n_pool;       // rows of X
  int64_t ld;
  const char *trees;
  int32_t ntrees;       // padded tree count
  int32_t chunk_trees;
  int32_t nchunks;
  int32_t F;
  int32_t vec4;         // rows are 16-byte aligned (X aligned, ld % 4 == 0)
  int32_t nbuf;         // LDS chunk buffers: 2 (asynchronous refill) or 1
  int32_t regstage;     // one buffer: the next chunk is fetched into registers
  int32_t rowpf;        // 1: rows load in line batches (vec4, F % 4 == 0, F <= 128)
  int32_t nthreads;     // threads per workgroup (== blockDim.x).  Read from the
                        // kernel arguments, which stay in scalar registers;
                        // blockDim.x is a vector load from the dispatch packet
                        // that the compiler re-issues under register pressure,
                        // and each re-issue waits for every load in flight.
  float base;
  uint8_t *valid_out;   // validity
  float *margin_out;
  const uint8_t *valid_in;  // perf
  float *score_out;         // perf; the fold of a row list
  const int32_t *rows_in;   // row list: entry i is pool row rows_in[i]
  float *leaves_out;        // leaf walk of a row list: [fold_trees][n]
  int32_t fold_trees;       // trees (with padding trees) the fold adds up
  const char *trees2;       // one pass over the pool: model P's records
  int32_t ntrees2;          // its trees (V's are the first fold_trees of the list)
  float base2;              // its margin bias
};

// Row `row` of X into the tile of its candidate (dst = tile + 4*candidate),
// whole, by one lane.  Pool rows are read with plain loads: a line whose
// 16-byte pieces arrive in separate instructions is fetched from HBM once,
// where with the non-temporal hint it was measured to be fetched twice.
template <int S>
__device__ __forceinline__ void load_row(const WalkArgs &a, int64_t row, char *dst) {
  constexpr uint32_t RW = Geo<S>::kRowBytes;
  const float *src = a.X + row * a.ld;
  int q = 0;
  if (a.vec4) {
    for (; q + 4 <= a.F; q += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(src + q);
      *reinterpret_cast<float *>(dst + (q + 0) * RW) = v.x;
      *reinterpret_cast<float *>(dst + (q + 1) * RW) = v.y;
      *reinterpret_cast<float *>(dst + (q + 2) * RW) = v.z;
      *reinterpret_cast<float *>(dst + (q + 3) * RW) = v.w;
    }
  }
  for (; q < a.F; ++q) *reinterpret_cast<float *>(dst + q * RW) = src[q];
}

// Rows of pools with at most kRowVecs*4 features and 16-byte aligned rows
// load in batches of 8 vectors per lane.  A batch is one 128-byte line of
// the row, lane half h taking lines h, h+S, ...; or, in the validity walk
// with two lanes per candidate (P), a batch spans two lines of which lane
// half h takes the vectors of parity h, so that one wave instruction
// requests 32 lines (both halves' pieces of each line) instead of 64 (3 %
// faster validity walk on the 16M pool; the perf walk, whose rows are
// scattered over the pool, ran 0.4 % slower with it).  A wave never has
// requests for many lines of one row in flight at once, which was measured
// to fetch lines again and evict the ensemble from L2.  The first batch of
// the next round's rows is fetched while the current round is walked.
// Loads are unconditional (a missing row reads row 0, a short row repeats
// its last vector), so the compiler knows how many are in flight.
constexpr int kRowVecs = 32;
constexpr int kRowBatch = 8;

__device__ __forceinline__ const f32x4 *row_src(const WalkArgs &a, int64_t row) {
  const int64_t rr = (row >= 0 && row < a.n_pool) ? row : 0;
  return reinterpret_cast<const f32x4 *>(a.X + rr * a.ld);
}

// Vector index (within the row) of element k of line-batch b (whole lines),
// or, with P, of lane half h's batch b (two lines shared by the halves).
template <bool P>
__device__ __forceinline__ int batch_vec(int b, int k, int h) {
  if constexpr (P)
    return (2 * b + (k >> 2)) * kRowBatch + 2 * (k & 3) + h;
  else
    return b * kRowBatch + k;
}

template <bool P>
__device__ __forceinline__ void row_batch_load(const WalkArgs &a, int64_t row, int b, int h,
                                               f32x4 (&v)[kRowBatch]) {
  const f32x4 *src = row_src(a, row);
  const int last = a.F / 4 - 1;
#pragma unroll
  for (int k = 0; k < kRowBatch; ++k) v[k] = src[min(batch_vec<P>(b, k, h), last)];
}

template <int S, bool P>
__device__ __forceinline__ void row_batch_store(const WalkArgs &a, int b, int h,
                                                const f32x4 (&v)[kRowBatch], char *dst) {
  constexpr uint32_t RW = Geo<S>::kRowBytes;
  const int nv = a.F / 4;
#pragma unroll
  for (int k = 0; k < kRowBatch; ++k) {
    const int q = batch_vec<P>(b, k, h);
    if (q < nv) {
      *reinterpret_cast<float *>(dst + (4 * q + 0) * RW) = v[k].x;
      *reinterpret_cast<float *>(dst + (4 * q + 1) * RW) = v[k].y;
      *reinterpret_cast<float *>(dst + (4 * q + 2) * RW) = v[k].z;
      *reinterpret_cast<float *>(dst + (4 * q + 3) * RW) = v[k].w;
    }
  }
}

// Tree chunks.  Chunk c holds trees [c*chunk_trees, min((c+1)*chunk_trees,
// ntrees)) and is walked cyclically.  With two LDS buffers the next chunk is
// copied by direct global->LDS loads (global_load_lds_dwordx4, no registers)
// while the current one is walked; completion is awaited with
// s_waitcnt vmcnt(0) and a workgroup barrier.  With one buffer the copy goes
// through registers (loaded chunks ahead) or is synchronous between two
// barriers.
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ uint32_t chunk_bytes_of(const WalkArgs &a, uint32_t rb, int c) {
  if (c >= a.nchunks) return 0u;  // padding chunk of the register-staged sequence
  const int nt = min(a.chunk_trees, a.ntrees - c * a.chunk_trees);
  return (uint32_t)nt * rb;
}

__device__ __forceinline__ const char *chunk_src(const WalkArgs &a, uint32_t rb, int c) {
  return a.trees + (size_t)c * a.chunk_trees * rb;
}

// Asynchronous copy of chunk c into dst: every wave takes 1 KiB segments.
__device__ __forceinline__ void stage_async(const WalkArgs &a, uint32_t rb, int c, char *dst) {
  const char *src = chunk_src(a, rb, c);
  const uint32_t bytes = chunk_bytes_of(a, rb, c);
  const uint32_t lane = threadIdx.x & (kLanes - 1);
  const uint32_t nw = a.nthreads / kLanes;
  for (uint32_t seg = (threadIdx.x / kLanes) * 1024u; seg < bytes; seg += nw * 1024u) {
    const uint32_t off = seg + lane * 16u;
    if (off < bytes)
      __builtin_amdgcn_global_load_lds((const void *)(src + off), (lds_void *)(dst + seg), 16, 0,
                                       0);
  }
}

// Synchronous copy of chunk c into dst; caller synchronises.
__device__ __forceinline__ void stage_copy(const WalkArgs &a, uint32_t rb, int c, char *dst) {
  const uint4 *src = reinterpret_cast<const uint4 *>(chunk_src(a, rb, c));
  uint4 *d = reinterpret_cast<uint4 *>(dst);
  const uint32_t nv = chunk_bytes_of(a, rb, c) / 16u;
  for (uint32_t i = threadIdx.x; i < nv; i += a.nthreads) d[i] = src[i];
}

// Chunks in flight in registers (2..4; four spill at the widest groups).
// The validity walks keep two: the 16M pool's walk then needs no padding
// chunk (ten chunks of 32 trees) and no spilled register (1.6 % faster; the
// perf walk ran 0.4 % slower with two).
constexpr int kValiditySets = 2;
constexpr int kPerfSets = 3;

// One chunk in R registers per thread.  Loads are unconditional (the table
// has kTreeSlack readable bytes after it), so the compiler knows how many are
// in flight: writing one register set to LDS waits only for that set's
// loads, not for those of the sets loaded after it.
template <int R>
__device__ __forceinline__ void stage_regs_load(const WalkArgs &a, uint32_t rb, int c,
                                                u32x4 (&r)[R]) {
  const u32x4 *src = reinterpret_cast<const u32x4 *>(chunk_src(a, rb, c < a.nchunks ? c : 0));
#pragma unroll
  for (int k = 0; k < R; ++k) r[k] = src[threadIdx.x + (uint32_t)k * a.nthreads];
}

template <int R>
__device__ __forceinline__ void stage_regs_store(const WalkArgs &a, uint32_t rb, int c,
                                                 const u32x4 (&r)[R], char *dst) {
  const uint32_t nv = chunk_bytes_of(a, rb, c) / 16u;
  u32x4 *d = reinterpret_cast<u32x4 *>(dst);
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const uint32_t i = threadIdx.x + (uint32_t)k * a.nthreads;
    if (i < nv) d[i] = r[k];
  }
}

__device__ __forceinline__ void wait_dma_and_barrier() {
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0): the direct-to-LDS copies have landed
  __syncthreads();
}

// A wave's own tile, written by its lanes and then read by them: the LDS
// performs one wave's operations in issue order, so only the compiler must
// keep the accesses on their side of this point (no instruction, no wait
// for the other waves).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Lanes 0..31 receive the value of lanes 32..63 (v_permlane32_swap: the
// second result holds the first operand's upper half in its lower half).
__device__ __forceinline__ float from_upper_half(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(r[1]);
}

// H walks of one half: heap positions u (1-based; children 2u, 2u+1),
// current node {feature index, threshold}, feature value and final leaf.
template <int D, int H, int S>
struct Walks {
  static constexpr uint32_t RB = record_bytes(D);
  static constexpr uint32_t L = 1u << D;
  uint32_t u[H];
  uint2 nd[H];
  float x[H];
  float leaf[H];

  __device__ __forceinline__ void start() {
#pragma unroll
    for (int g = 0; g < H; ++g) u[g] = 1u;
  }
  __device__ __forceinline__ void read_nodes(const char *rec) {
#pragma unroll
    for (int g = 0; g < H; ++g) nd[g] = *reinterpret_cast<const uint2 *>(rec + g * RB + 8u * u[g]);
  }
  __device__ __forceinline__ void read_features(const char *tile_lane) {
#pragma unroll
    for (int g = 0; g < H; ++g)
      x[g] = *reinterpret_cast<const float *>(tile_lane + (nd[g].x << Geo<S>::kRowShift));
  }
  // u <- 2u + [x < threshold]: one compare into a lane mask and one
  // add-with-carry per walk.  All compares precede all adds, so each mask is
  // H-1 instructions old when read (s_nop covers H < 3).
  __device__ __forceinline__ void descend() {
    uint64_t lt[H];
#pragma unroll
    for (int g = 0; g < H; ++g)
      asm volatile("v_cmp_lt_f32_e64 %0, %1, %2"
                   : "=s"(lt[g])
                   : "v"(x[g]), "v"(__uint_as_float(nd[g].y)));
    if (H < 3) asm volatile("s_nop 1");
#pragma unroll
    for (int g = 0; g < H; ++g)
      asm volatile("v_addc_co_u32_e64 %0, vcc, %0, %0, %1" : "+v"(u[g]) : "s"(lt[g]) : "vcc");
  }
  __device__ __forceinline__ void read_leaves(const char *rec) {
#pragma unroll
    for (int g = 0; g < H; ++g)
      leaf[g] = *reinterpret_cast<const float *>(rec + g * RB + 4u * L + 4u * u[g]);
  }
  // Fold this half's leaves (lower lanes' own), in tree order.
  __device__ __forceinline__ float fold(float m) const {
#pragma unroll
    for (int g = 0; g < H; ++g) m = m + leaf[g];
    return m;
  }
  // Fold the upper half-wave's leaves into the lower half's margins.
  __device__ __forceinline__ float fold_upper(float m) const {
#pragma unroll
    for (int g = 0; g < H; ++g) m = m + from_upper_half(leaf[g]);
    return m;
  }
};

// H walks of one half over a ragged chunk slot: u is the index of the
// current 8-byte node in the slot.  One step: x < t goes left, a missing x
// goes left where the node's default is left, else right; the right child
// follows the left one (u <- u + offset + [right]), and a leaf (offset -1)
// goes right, onto itself.  A leaf's second word is its value.
template <int H, int S>
struct RWalks {
  uint32_t u[H];
  uint2 nd[H];
  float x[H];
  float leaf[H];

  __device__ __forceinline__ void read_nodes(const char *slot) {
#pragma unroll
    for (int g = 0; g < H; ++g) nd[g] = *reinterpret_cast<const uint2 *>(slot + 8u * u[g]);
  }
  __device__ __forceinline__ void read_features(const char *tile_lane) {
#pragma unroll
    for (int g = 0; g < H; ++g) {
      // bits 15..0 of word 0: the feature's offset in 256-byte tile rows
      const uint32_t off = S == 1 ? (nd[g].x & 0xFFFFu) : (nd[g].x & 0xFFFFu) >> 1;
      x[g] = *reinterpret_cast<const float *>(tile_lane + off);
    }
  }
  __device__ __forceinline__ void descend() {
#pragma unroll
    for (int g = 0; g < H; ++g) {
      const float t = __uint_as_float(nd[g].y);
      const bool missing_left = (int32_t)nd[g].x < 0 && __builtin_isnan(x[g]);
      const bool right = is_leaf(nd[g].x) || (!(x[g] < t) && !missing_left);
      const int32_t off = (int32_t)(nd[g].x << 1) >> 17;  // bits 30..16, signed
      u[g] = u[g] + (uint32_t)off + (right ? 1u : 0u);
    }
  }
  // Once every walk is on a leaf, the nodes last read are the leaves.
  __device__ __forceinline__ void take_leaves() {
#pragma unroll
    for (int g = 0; g < H; ++g) leaf[g] = __uint_as_float(nd[g].y);
  }
  // Every walk of this lane is on a leaf.
  __device__ __forceinline__ bool at_leaves() const {
    bool all = true;
#pragma unroll
    for (int g = 0; g < H; ++g) all = all && is_leaf(nd[g].x);
    return all;
  }
  __device__ __forceinline__ float fold(float m) const {
#pragma unroll
    for (int g = 0; g < H; ++g) m = m + leaf[g];
    return m;
  }
  __device__ __forceinline__ float fold_upper(float m) const {
#pragma unroll
    for (int g = 0; g < H; ++g) m = m + from_upper_half(leaf[g]);
    return m;
  }
  // a leaf's first word: offset -1 in bits 31..16 (no split has it)
  __device__ __forceinline__ static bool is_leaf(uint32_t w0) { return (w0 >> 16) == 0x7FFFu; }
};

// Ragged chunk slot header (layout.h), read from LDS into scalars.
struct SlotHead {
  int ntrees;
  int depth;
  uint32_t sentinel;  // node index of the slot's sentinel leaf
  int tree0;
};

__device__ __forceinline__ SlotHead slot_head(const char *slot) {
  const uint4 h = *reinterpret_cast<const uint4 *>(slot);
  return {__builtin_amdgcn_readfirstlane((int)h.x), __builtin_amdgcn_readfirstlane((int)h.y),
          (uint32_t)__builtin_amdgcn_readfirstlane((int)h.z),
          __builtin_amdgcn_readfirstlane((int)h.w)};
}

// One group of a ragged slot: the G trees whose root offsets start at
// `roots` (in LDS), walked until every lane of the wave is on leaves, at
// most `depth` steps (the slot's deepest path).  Leaves step onto
// themselves, so stopping at any point past that gives the same leaves.
template <int G, int S, typename Done>
__device__ __forceinline__ void walk_group_ragged(const char *slot, const uint32_t *roots,
                                                  int depth, const char *tile_lane,
                                                  Done done) {
  // Loops whose only exit is at the bottom (an early exit made the compiler
  // wait for every LDS read in flight at the top of each step): a step whose
  // walks are all on leaves is still taken, as leaves step onto themselves.
  if constexpr (G == 1) {
    RWalks<1, S> A;
    A.u[0] = roots[0];
    A.read_nodes(slot);
    int l = 0;
    bool go = depth > 0;
    while (go) {
      A.read_features(tile_lane);
      const bool all = __all(A.at_leaves());
      A.descend();
      A.read_nodes(slot);
      go = !all && ++l < depth;
    }
    A.take_leaves();
    done(A, A);
  } else {
    constexpr int H = G / 2;
    RWalks<H, S> A, B;
#pragma unroll
    for (int g = 0; g < H; ++g) {
      A.u[g] = roots[g];
      B.u[g] = roots[H + g];
    }
    A.read_nodes(slot);
    B.read_nodes(slot);
    __builtin_amdgcn_sched_barrier(0);
    int l = 0;
    bool go = depth > 0;
    while (go) {
      // the exit test follows the feature reads, so that it does not hold
      // them back until every node read has landed
      A.read_features(tile_lane);
      __builtin_amdgcn_sched_barrier(0);
      B.read_features(tile_lane);
      __builtin_amdgcn_sched_barrier(0);
      const bool all = __all(A.at_leaves() && B.at_leaves());
      A.descend();
      A.read_nodes(slot);
      __builtin_amdgcn_sched_barrier(0);
      B.descend();
      B.read_nodes(slot);
      __builtin_amdgcn_sched_barrier(0);
      go = !all && ++l < depth;
    }
    A.take_leaves();
    B.take_leaves();
    done(A, B);
  }
}

// All groups of a ragged slot with one lane per candidate, each lane on its
// own group: a lane whose G walks are all on leaves folds their values (the
// leaves' second words, in tree order) and moves on to its next group while
// the other lanes keep descending, so the wave waits for the lane with the
// longest sum of group lengths instead of, group by group, for the longest
// path of any lane.  The roots of a lane's next group are read at every
// step, so a move never waits for LDS.  Every lane is done after at most
// (groups) x (depth + 1) steps; the loop stops a little past that at the
// latest.
template <int G>
__device__ __forceinline__ float walk_slot_lanes(const char *slot, int ntr, int depth,
                                                 const char *tile_lane, float m) {
  constexpr int H = G == 1 ? 1 : G / 2;
  using RootVec = std::conditional_t<G == 4, uint4, std::conditional_t<G == 2, uint2, uint32_t>>;
  const uint32_t *roots = reinterpret_cast<const uint32_t *>(slot + 16);
  auto load_roots = [&](int t, uint32_t (&r)[G]) {  // t: a multiple of G, at most ntr + G
    const RootVec v = *reinterpret_cast<const RootVec *>(roots + t);
    if constexpr (G == 4) {
      r[0] = v.x;
      r[1] = v.y;
      r[2] = v.z;
      r[3] = v.w;
    } else if constexpr (G == 2) {
      r[0] = v.x;
      r[1] = v.y;
    } else {
      r[0] = v;
    }
  };
  RWalks<H, 1> A, B;
  uint32_t nxt[G];
  load_roots(0, nxt);
#pragma unroll
  for (int g = 0; g < H; ++g) {
    A.u[g] = nxt[g];
    if constexpr (G > 1) B.u[g] = nxt[H + g];
  }
  A.read_nodes(slot);
  if constexpr (G > 1) B.read_nodes(slot);
  // t: the lane's next group (its current group is the one before; ntr + G
  // once every group is done).  Reading the roots of a group past the last
  // reads node words of the slot, which a finished lane never uses.
  int t = G;
  load_roots(t, nxt);
  __builtin_amdgcn_sched_barrier(0);
  // The only exit is at the bottom: an early exit made the compiler wait
  // for every LDS read in flight at the top of each step.
  const int cap = (ntr / G) * (depth + 2) + 2;
  int it = 0;
  bool go = true;
  while (go) {
    A.read_features(tile_lane);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (G > 1) B.read_features(tile_lane);
    __builtin_amdgcn_sched_barrier(0);
    const bool fin = t > ntr;
    bool leaves = A.at_leaves();
    if constexpr (G > 1) leaves = leaves && B.at_leaves();
    const bool sw = !fin && leaves;
    float fm = m;
#pragma unroll
    for (int g = 0; g < H; ++g) fm = fm + __uint_as_float(A.nd[g].y);
    if constexpr (G > 1) {
#pragma unroll
      for (int g = 0; g < H; ++g) fm = fm + __uint_as_float(B.nd[g].y);
    }
    m = sw ? fm : m;
    const bool mv = sw && t < ntr;
    t += sw ? G : 0;
    A.descend();
#pragma unroll
    for (int g = 0; g < H; ++g) A.u[g] = mv ? nxt[g] : A.u[g];
    A.read_nodes(slot);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (G > 1) {
      B.descend();
#pragma unroll
      for (int g = 0; g < H; ++g) B.u[g] = mv ? nxt[H + g] : B.u[g];
      B.read_nodes(slot);
    }
    load_roots(t, nxt);
    __builtin_amdgcn_sched_barrier(0);
    go = !__all(t > ntr) && ++it < cap;
  }
  return m;
}

// A ragged slot with one lane per candidate and one tree per lane: a walk on
// a leaf adds the leaf's value and, in the same step, moves on to the root
// of the lane's next tree, whose place the leaf holds, so no lane waits for
// another's path.  The last tree's leaves lead to the slot's sentinel (a
// leaf of value -0.0 that leads to itself), and adding -0.0 leaves every
// float unchanged, so a finished lane needs no test of its own.  The loop
// runs eight steps per trip (one exit test per trip: every lane on the
// sentinel).  Every lane is done after at most (trees) x (depth + 1) steps;
// the loop stops a little past that at the latest.
__device__ __forceinline__ float walk_slot_single(const char *slot, const SlotHead &hd,
                                                  const char *tile_lane, float m) {
  const uint32_t *roots = reinterpret_cast<const uint32_t *>(slot + 16);
  // a: byte offset of the lane's current node in the slot
  uint32_t a = 8u * roots[0];
  uint2 nd = *reinterpret_cast<const uint2 *>(slot + a);
  __builtin_amdgcn_sched_barrier(0);
  const uint32_t end = 8u * hd.sentinel;
  const int cap = hd.ntrees * (hd.depth + 2) + 8;
  int it = 0;
  bool go = true;
  while (go) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint32_t w0 = nd.x;
      // bits 15..0: the feature's byte offset in a 256-byte tile row (a
      // leaf: the next root's byte offset, read and ignored)
      const float x = *reinterpret_cast<const float *>(tile_lane + (w0 & 0xFFFFu));
      __builtin_amdgcn_sched_barrier(0);
      // both next addresses before the feature value is in: the left child
      // (the right one follows it), or a leaf's next root either way
      const bool leaf = RWalks<1, 1>::is_leaf(w0);
      const int32_t off = (int32_t)(w0 << 1) >> 17;  // bits 30..16, signed
      const uint32_t to_left = leaf ? (w0 & 0xFFFFu) : a + 8u * (uint32_t)off;
      const uint32_t to_right = leaf ? (w0 & 0xFFFFu) : to_left + 8u;
      m = m + (leaf ? __uint_as_float(nd.y) : -0.0f);
      // right: x >= t where a missing x goes left (default-left, bit 31),
      // not x < t otherwise (a missing x goes right); both candidates
      // follow from the feature in one compare each
      const float t = __uint_as_float(nd.y);
      const uint32_t by_ge = (x >= t) ? to_right : to_left;
      const uint32_t by_nlt = !(x < t) ? to_right : to_left;
      a = (int32_t)w0 < 0 ? by_ge : by_nlt;
      asm volatile("" : "+v"(a));  // computed by every lane: no branch
      nd = *reinterpret_cast<const uint2 *>(slot + a);
      __builtin_amdgcn_sched_barrier(0);
    }
    it += 8;
    go = !__all(a == end) && it < cap;
  }
  return m;
}

// One group: half-wave h walks the G trees of records starting at `rec`
// (two halves of H = G/2 offset by half a level), then `done(A, B)` gets the
// leaves (A: the first H trees, B: the next H; with G == 1 only A).
template <int D, int G, int S, typename Done>
__device__ __forceinline__ void walk_group(const char *rec, const char *tile_lane, Done done) {
  constexpr uint32_t RB = record_bytes(D);
  if constexpr (G == 1) {
    Walks<D, 1, S> A;
    A.start();
#pragma unroll
    for (int l = 0; l < D; ++l) {
      A.read_nodes(rec);
      A.read_features(tile_lane);
      A.descend();
    }
    A.read_leaves(rec);
    done(A, A);
  } else {
    constexpr int H = G / 2;
    const char *recA = rec;
    const char *recB = rec + H * RB;
    Walks<D, H, S> A, B;
    A.start();
    B.start();
    A.read_nodes(recA);
    B.read_nodes(recB);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int l = 0; l < D; ++l) {
      A.read_features(tile_lane);
      __builtin_amdgcn_sched_barrier(0);
      B.read_features(tile_lane);
      __builtin_amdgcn_sched_barrier(0);
      A.descend();
      if (l + 1 < D) A.read_nodes(recA); else A.read_leaves(recA);
      __builtin_amdgcn_sched_barrier(0);
      B.descend();
      if (l + 1 < D) B.read_nodes(recB); else B.read_leaves(recB);
      __builtin_amdgcn_sched_barrier(0);
    }
    done(A, B);
  }
}

// Calls of walk_chunk's `after` for a chunk of ntr records: one per group
// of perfect trees, one per ragged slot.
template <int D, int G, int S>
__device__ __forceinline__ int walk_groups(int ntr) {
  return D == 0 ? ntr : ntr / (G * S);
}

// Walk `ntr` trees (a multiple of S*G) of the chunk at `cb`, folding their
// leaves into m in tree order.  Half-wave h walks trees [t0 + h*G, t0 +
// (h+1)*G) of each group of S*G; with S = 2 only the lower half's m is the
// candidate's margin.
template <int D, int G, int S, typename After>
__device__ __forceinline__ float walk_chunk_after(const char *cb, int ntr, const char *tile_lane,
                                                  int h, float m, After after) {
  constexpr uint32_t RB = record_bytes(D);
  constexpr int GS = G * S;
  auto fold = [&](const auto &A, const auto &B) {
    if constexpr (G == 1) {
      m = A.fold(m);
      if constexpr (S == 2) m = A.fold_upper(m);
    } else {
      m = B.fold(A.fold(m));
      if constexpr (S == 2) m = B.fold_upper(A.fold_upper(m));
    }
  };
  if constexpr (D == 0) {  // ntr ragged slots
    for (int i = 0; i < ntr; ++i) {
      const char *slot = cb + (uint32_t)i * RB;
      const SlotHead hd = slot_head(slot);
      if constexpr (S == 1 && G == 1) {
        m = walk_slot_single(slot, hd, tile_lane, m);
      } else if constexpr (S == 1) {
        m = walk_slot_lanes<G>(slot, hd.ntrees, hd.depth, tile_lane, m);
      } else {
        const uint32_t *roots = reinterpret_cast<const uint32_t *>(slot + 16) + h * G;
        for (int t0 = 0; t0 < hd.ntrees; t0 += GS)
          walk_group_ragged<G, S>(slot, roots + t0, hd.depth, tile_lane, fold);
      }
      after(i);
    }
  } else {
    for (int t0 = 0; t0 < ntr; t0 += GS) {
      walk_group<D, G, S>(cb + (uint32_t)(t0 + h * G) * RB, tile_lane, fold);
      after(t0 / GS);
    }
  }
  return m;
}

// The same without a call between groups (the streamed chunks' walk).
template <int D, int G, int S>
__device__ __forceinline__ float walk_chunk(const char *cb, int ntr, const char *tile_lane,
                                            int h, float m) {
  constexpr uint32_t RB = record_bytes(D);
  constexpr int GS = G * S;
  auto fold = [&](const auto &A, const auto &B) {
    if constexpr (G == 1) {
      m = A.fold(m);
      if constexpr (S == 2) m = A.fold_upper(m);
    } else {
      m = B.fold(A.fold(m));
      if constexpr (S == 2) m = B.fold_upper(A.fold_upper(m));
    }
  };
  if constexpr (D == 0) {  // ntr ragged slots
    for (int i = 0; i < ntr; ++i) {
      const char *slot = cb + (uint32_t)i * RB;
      const SlotHead hd = slot_head(slot);
      if constexpr (S == 1 && G == 1) {
        m = walk_slot_single(slot, hd, tile_lane, m);
      } else if constexpr (S == 1) {
        m = walk_slot_lanes<G>(slot, hd.ntrees, hd.depth, tile_lane, m);
      } else {
        const uint32_t *roots = reinterpret_cast<const uint32_t *>(slot + 16) + h * G;
        for (int t0 = 0; t0 < hd.ntrees; t0 += GS)
          walk_group_ragged<G, S>(slot, roots + t0, hd.depth, tile_lane, fold);
      }
    }
  } else {
    for (int t0 = 0; t0 < ntr; t0 += GS)
      walk_group<D, G, S>(cb + (uint32_t)(t0 + h * G) * RB, tile_lane, fold);
  }
  return m;
}

// Staging state.  Invariant between walks: `cur` holds the chunk about to be
// walked; the following chunk is in flight to `other` (two buffers) or to
// the registers `r` (one buffer).
// K: chunks in flight in registers, R registers each.
template <int K, int R>
struct Stage {
  char *cur;    // holds the chunk about to be walked
  char *other;  // two buffers: the next chunk lands here (== cur with one)
  u32x4 r[K][R];  // registers: the next K chunks
};

// Row prefetch: batches h, h+S, ..., h+E*S of a row (the lane half's first
// E+1 batches) in registers.  With the whole ensemble in one chunk nothing is
// restaged, the staging registers are dead, and E extra batches take their
// place, so that the next round's rows are (for F <= 128 with S = 2: fully)
// in flight while the current round is walked.
template <int S, int K, int R>
constexpr int row_extra_batches() {
  return S == 2 ? (K * R) / kRowBatch : 0;  // one lane per candidate: no room
}

// Lines shared by four lanes (Q, S = 2): lanes (h, r, q) with h = lane bit
// 5, r = lane bit 4 and q = lane bits 3..0 hold candidates q + 16r.  The four
// lanes (h, r) of candidates q and q+16 load the four vectors 4j..4j+3 (one
// 64-byte half) of a line, first of row q, then of row q+16 (lane (h, r)
// takes vector 4j + 2r + h), so a wave instruction requests 16 half-lines;
// one v_permlane16_swap per word then gives every lane the vectors of
// parity h of its own row, as the paired layout expects (element k of a
// batch = vector 2(k&3) + h of line k/4).
__device__ __forceinline__ void quad_rows(int64_t row, int64_t &rx, int64_t &ry) {
  const uint32_t lo = (uint32_t)(uint64_t)row, hi = (uint32_t)((uint64_t)row >> 32);
  const auto l = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  const auto u = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
  rx = (int64_t)(((uint64_t)u[0] << 32) | l[0]);  // the row of candidate q
  ry = (int64_t)(((uint64_t)u[1] << 32) | l[1]);  // the row of candidate q + 16
}

__device__ __forceinline__ void row_batch_load_quad(const WalkArgs &a, int64_t rx, int64_t ry,
                                                    int b, int h, f32x4 (&v)[kRowBatch]) {
  const f32x4 *sx = row_src(a, rx);
  const f32x4 *sy = row_src(a, ry);
  const int last = a.F / 4 - 1;
  const int r = (threadIdx.x >> 4) & 1;
#pragma unroll
  for (int l = 0; l < 2; ++l) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int q = min((2 * b + l) * kRowBatch + 4 * j + 2 * r + h, last);
      v[4 * l + 2 * j] = sx[q];
      v[4 * l + 2 * j + 1] = sy[q];
    }
  }
}

__device__ __forceinline__ void swap_rows16(f32x4 &x, f32x4 &y) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(x[c]), __float_as_uint(y[c]),
                                                    false, false);
    x[c] = __uint_as_float(t[0]);
    y[c] = __uint_as_float(t[1]);
  }
}

__device__ __forceinline__ void quad_swap(f32x4 (&v)[kRowBatch]) {
#pragma unroll
  for (int l = 0; l < 2; ++l) {
#pragma unroll
    for (int j = 0; j < 2; ++j) swap_rows16(v[4 * l + 2 * j], v[4 * l + 2 * j + 1]);
  }
}

// P: the lane halves take their halves of the same lines (paired layout);
// Q: with P, the lines shared by four lanes (quad loads).
template <int S, int E, bool P, bool Q = P>
struct RowPrefetch {
  static_assert(P || !Q, "quad loads fill the paired layout");
  f32x4 v[E + 1][kRowBatch];

  // the batch index of prefetched batch e of lane half h
  __device__ __forceinline__ static int batch(int e, int h) { return P ? e : h + e * S; }

  __device__ __forceinline__ void load(const WalkArgs &a, int64_t row, int h) {
    if constexpr (Q) {
      int64_t rx, ry;
      quad_rows(row, rx, ry);
#pragma unroll
      for (int e = 0; e <= E; ++e) row_batch_load_quad(a, rx, ry, e, h, v[e]);
    } else {
#pragma unroll
      for (int e = 0; e <= E; ++e) row_batch_load<P>(a, row, batch(e, h), h, v[e]);
    }
  }
  template <int e>
  __device__ __forceinline__ void load_batch(const WalkArgs &a, int64_t row, int h) {
    if constexpr (Q) {
      int64_t rx, ry;
      quad_rows(row, rx, ry);
      row_batch_load_quad(a, rx, ry, e, h, v[e]);
    } else {
      row_batch_load<P>(a, row, batch(e, h), h, v[e]);
    }
  }
  // Batch 0 is loaded before a walk; after group g of the walk, batch g+1:
  // the loads of a round spread over the walk instead of reaching the memory
  // path at once (all at the start of the walk, or later than one group
  // ahead of the next round, measured slower).  load_rest() then loads the
  // batches of a walk with fewer groups than batches.
  __device__ __forceinline__ void load_after_group(const WalkArgs &a, int64_t row, int h, int g) {
    static_assert(E <= 2, "extra batches beyond two");
    if constexpr (E >= 1) {
      if (g == 0) load_batch<1>(a, row, h);
    }
    if constexpr (E >= 2) {
      if (g == 1) load_batch<2>(a, row, h);
    }
  }
  __device__ __forceinline__ void load_rest(const WalkArgs &a, int64_t row, int h, int groups) {
    if constexpr (E >= 1) {
      if (groups < 1) load_batch<1>(a, row, h);
    }
    if constexpr (E >= 2) {
      if (groups < 2) load_batch<2>(a, row, h);
    }
  }
  // Write the prefetched batches into the tile, then load and write the lane
  // half's remaining batches.
  __device__ __forceinline__ void commit(const WalkArgs &a, int64_t row, int h, char *dst) {
    const int lines = (a.F / 4 + kRowBatch - 1) / kRowBatch;
    if constexpr (Q) {
#pragma unroll
      for (int e = 0; e <= E; ++e) {
        quad_swap(v[e]);
        row_batch_store<S, P>(a, e, h, v[e], dst);
      }
      int64_t rx, ry;
      quad_rows(row, rx, ry);
      for (int b = E + 1; 2 * b < lines; ++b) {
        f32x4 w[kRowBatch];
        row_batch_load_quad(a, rx, ry, b, h, w);
        quad_swap(w);
        row_batch_store<S, P>(a, b, h, w, dst);
      }
    } else if constexpr (P) {
#pragma unroll
      for (int e = 0; e <= E; ++e) row_batch_store<S, P>(a, e, h, v[e], dst);
      for (int b = E + 1; 2 * b < lines; ++b) {
        f32x4 w[kRowBatch];
        row_batch_load<P>(a, row, b, h, w);
        row_batch_store<S, P>(a, b, h, w, dst);
      }
    } else {
#pragma unroll
      for (int e = 0; e <= E; ++e) row_batch_store<S, P>(a, batch(e, h), h, v[e], dst);
      for (int b = h + (E + 1) * S; b < lines; b += S) {
        f32x4 w[kRowBatch];
        row_batch_load<P>(a, row, b, h, w);
        row_batch_store<S, P>(a, b, h, w, dst);
      }
    }
  }
};

// Length of the cyclic chunk sequence: with register staging it is padded
// with empty chunks to a multiple of K, so that set j always holds a chunk
// whose index is j+1 modulo K and every set index is a compile-time constant.
template <int K>
__device__ __forceinline__ int seq_len(const WalkArgs &a) {
  return a.regstage ? (a.nchunks + K - 1) / K * K : a.nchunks;
}

__device__ __forceinline__ int cyc(int c, int nseq) {
  while (c >= nseq) c -= nseq;
  return c;
}

template <int K, int R>
__device__ __forceinline__ void stage_prime(const WalkArgs &a, uint32_t rb, Stage<K, R> &s) {
  stage_copy(a, rb, 0, s.cur);
  if (a.nchunks > 1) {
    if (a.nbuf == 2) {
      stage_async(a, rb, 1, s.other);
    } else if (a.regstage) {
      const int nseq = seq_len<K>(a);
#pragma unroll
      for (int j = 0; j < K; ++j) stage_regs_load<R>(a, rb, cyc(1 + j, nseq), s.r[j]);
    }
  }
  wait_dma_and_barrier();
}

// Register staging, after walking chunk c (c == J mod K): set J holds chunk
// c+1; write it to LDS and start loading chunk c+1+K.  The sets loaded after
// set J stay in flight.
// LATE: issue those loads after the second barrier instead of before it
// (one lane per candidate: its perf walk 3 % faster on the explorer
// workload; with two lanes per candidate 3.6 % slower on the 16M pool).
template <int J, int K, int R, bool LATE = false>
__device__ __forceinline__ void stage_advance_regs(const WalkArgs &a, uint32_t rb, int c,
                                                   int nseq, Stage<K, R> &s) {
  __syncthreads();  // every wave is done with the buffer
  stage_regs_store<R>(a, rb, cyc(c + 1, nseq), s.r[J], s.cur);
  if constexpr (!LATE) stage_regs_load<R>(a, rb, cyc(c + 1 + K, nseq), s.r[J]);
  __syncthreads();
  if constexpr (LATE) stage_regs_load<R>(a, rb, cyc(c + 1 + K, nseq), s.r[J]);
}

// Two buffers or a synchronous copy, after walking chunk c.
template <int K, int R>
__device__ __forceinline__ void stage_advance(const WalkArgs &a, uint32_t rb, int c,
                                              Stage<K, R> &s) {
  if (a.nchunks == 1) return;
  const int next = cyc(c + 1, a.nchunks);
  if (a.nbuf == 2) {
    wait_dma_and_barrier();  // chunk `next` landed; every wave is done with cur
    char *t = s.cur;
    s.cur = s.other;
    s.other = t;
    if (a.nchunks > 2) stage_async(a, rb, cyc(c + 2, a.nchunks), s.other);
  } else {
    __syncthreads();
    stage_copy(a, rb, next, s.cur);
    __syncthreads();
  }
}

// Every chunk of the ensemble for the candidates in the tiles; leaves the
// staging invariant in place for the next round.
template <int D, int G, int S, int K, int R>
__device__ __forceinline__ float walk_all(const WalkArgs &a, Stage<K, R> &s,
                                          const char *tile_lane, int h) {
  constexpr uint32_t RB = record_bytes(D);
  constexpr bool LT = S == 1;  // chunk loads after the second barrier
  float m = a.base;
  if (a.nchunks == 1) return walk_chunk<D, G, S>(s.cur, a.ntrees, tile_lane, h, m);
  if (a.regstage) {
    const int nseq = seq_len<K>(a);
    for (int c = 0; c < nseq; c += K) {
#pragma unroll
      for (int j = 0; j < K; ++j) {
        m = walk_chunk<D, G, S>(s.cur, (int)(chunk_bytes_of(a, RB, c + j) / RB), tile_lane, h,
                                m);
        switch (j) {  // compile-time set index
          case 0: stage_advance_regs<0, K, R, LT>(a, RB, c + j, nseq, s); break;
          case 1: stage_advance_regs<1, K, R, LT>(a, RB, c + j, nseq, s); break;
          case 2: if constexpr (K > 2) stage_advance_regs<2, K, R, LT>(a, RB, c + j, nseq, s); break;
          default: if constexpr (K > 3) stage_advance_regs<3, K, R, LT>(a, RB, c + j, nseq, s); break;
        }
      }
    }
  } else {
    for (int c = 0; c < a.nchunks; ++c) {
      m = walk_chunk<D, G, S>(s.cur, (int)(chunk_bytes_of(a, RB, c) / RB), tile_lane, h, m);
      stage_advance(a, RB, c, s);
    }
  }
  return m;
}

// walk_all, calling after() once the first chunk is walked (streamed
// ensembles, register staging: the streamed validity walk loads its second
// row batch for the next round there).
template <int D, int G, int S, int K, int R, typename After>
__device__ __forceinline__ float walk_all_after(const WalkArgs &a, Stage<K, R> &s,
                                                const char *tile_lane, int h, After after) {
  constexpr uint32_t RB = record_bytes(D);
  if (!a.regstage || a.nchunks == 1) {  // not the case the launcher sends here
    const float m = walk_all<D, G, S>(a, s, tile_lane, h);
    after();
    return m;
  }
  constexpr bool LT = S == 1;  // chunk loads after the second barrier
  float m = a.base;
  const int nseq = seq_len<K>(a);
  for (int c = 0; c < nseq; c += K) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
      m = walk_chunk<D, G, S>(s.cur, (int)(chunk_bytes_of(a, RB, c + j) / RB), tile_lane, h, m);
      if (j == 0 && c == 0) after();
      switch (j) {  // compile-time set index
        case 0: stage_advance_regs<0, K, R, LT>(a, RB, c + j, nseq, s); break;
        case 1: stage_advance_regs<1, K, R, LT>(a, RB, c + j, nseq, s); break;
        case 2: if constexpr (K > 2) stage_advance_regs<2, K, R, LT>(a, RB, c + j, nseq, s); break;
        default: if constexpr (K > 3) stage_advance_regs<3, K, R, LT>(a, RB, c + j, nseq, s); break;
      }
    }
  }
  return m;
}

// The round loop of a walk kernel, by regime.  kAny decides row prefetch and
// staging at run time.  With S = 2 the kernels run a separate loop for
// prefetched rows with a streamed ensemble and one with a resident ensemble
// (one chunk), so that no loop merges register values from another: where a
// loop did, the compiler copied the prefetched rows at the merge and, to do
// so, waited for every load in flight before each walk.  With S = 1 the
// kernels are near their register limit and keep the single loop.
// Resident ensembles with prefetched rows launch a kernel of their own
// (RES), whose loop spreads the next round's row loads over the walk.  The
// streamed kernel keeps its own resident loop (kResidentInline, not reached
// from the launcher): built without it, the compiler laid out the streamed
// loop so that the 16M-pool perf walk ran 2 % slower (measured three times).
constexpr int kAny = 0;
constexpr int kStreamed = 1;
constexpr int kResident = 2;        // the resident kernel: loads spread over the walk
constexpr int kResidentInline = 3;  // the same regime inside the streamed kernel

template <int S, bool RES, typename Rounds>
__device__ __forceinline__ void dispatch_rounds(const WalkArgs &a, Rounds &rounds) {
  if constexpr (RES) {
    rounds(std::integral_constant<int, kResident>{});
  } else if constexpr (S == 2) {
    if (!a.rowpf)
      rounds(std::integral_constant<int, kAny>{});
    else if (a.nchunks == 1)
      rounds(std::integral_constant<int, kResidentInline>{});
    else
      rounds(std::integral_constant<int, kStreamed>{});
  } else {
    rounds(std::integral_constant<int, kAny>{});
  }
}

// Launch the resident kernel (RES): S = 2, one chunk, rows prefetched.
constexpr bool resident_launch(int S, const WalkArgs &a) {
  return S == 2 && a.nchunks == 1 && a.rowpf;
}

// With S = 2 a kernel must leave room for two waves per SIMD (256 VGPRs).
template <int D, int G, int S, bool RES>
__global__ void __launch_bounds__(kLanes *kMaxWaves) __attribute__((amdgpu_waves_per_eu(S, S)))
validity_kernel(WalkArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr uint32_t RB = record_bytes(D);
  constexpr int CPW = Geo<S>::kCand;
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int h = lane / CPW;  // half-wave (0 with S = 1)
  const int cl = lane % CPW;
  const int W = a.nthreads / kLanes;
  const size_t tile_bytes = (size_t)a.F * Geo<S>::kRowBytes;
  const uint32_t chunk_bytes = (uint32_t)a.chunk_trees * RB;
  constexpr int K = stage_sets(D, S, kValiditySets);
  Stage<K, stage_regs(D, S)> st;
  st.cur = smem + W * tile_bytes;
  st.other = st.cur + (a.nbuf == 2 ? chunk_bytes : 0u);
  char *tile_lane = smem + wave * tile_bytes + 4 * cl;
  const int64_t ntiles = (a.n + CPW - 1) / CPW;
  stage_prime(a, RB, st);
  auto rounds = [&](auto mode) {
    constexpr int M = decltype(mode)::value;
    // streamed ensembles (register staging): a second batch, loaded after
    // the first chunk
    constexpr int E = M >= kResident ? row_extra_batches<S, K, stage_regs(D, S)>()
                      : (M == kStreamed && S == 2) ? 1
                                                   : 0;
    // lines shared by four lanes in the streamed kernel only (validity
    // 8.56 -> 8.31 ms on the 16M pool; the resident kernel of the HBM-bound
    // diagnostic ran 8 % slower with them)
    RowPrefetch<S, E, S == 2, S == 2 && !RES> pf;
    const bool pfr = M != kAny || a.rowpf;  // rows prefetched
    if (pfr) pf.load(a, ((int64_t)blockIdx.x * W + wave) * CPW + cl, h);
    for (int64_t tg = blockIdx.x; tg * W < ntiles; tg += gridDim.x) {
      const int64_t row = (tg * W + wave) * CPW + cl;
      const bool active = row < a.n;
      const int64_t rn = ((tg + gridDim.x) * W + wave) * CPW + cl;
      constexpr bool split_loads = M == kResident || (M == kStreamed && E >= 1);
      if (pfr) {
        pf.commit(a, row, h, tile_lane);
        if constexpr (split_loads)
          pf.template load_batch<0>(a, rn, h);
        else
          pf.load(a, rn, h);
      } else if (active && h == 0) {
        load_row<S>(a, row, tile_lane);
      }
      // a wave reads only its own tile, and every round finds chunk 0
      // complete in the buffer: staged once (stage_prime ends with a
      // barrier), or restaged by the previous round's last advance, which
      // ends with one
      wave_sync();
      float m;
      if constexpr (M == kResident) {
        m = walk_chunk_after<D, G, S>(st.cur, a.ntrees, tile_lane, h, a.base,
                                      [&](int g) { pf.load_after_group(a, rn, h, g); });
        pf.load_rest(a, rn, h, walk_groups<D, G, S>(a.ntrees));
      } else if constexpr (M == kStreamed && E >= 1) {
        // kStreamed runs with register staging and more than one chunk
        m = walk_all_after<D, G, S>(a, st, tile_lane, h,
                                    [&]() { pf.template load_batch<1>(a, rn, h); });
      } else if constexpr (M == kResidentInline) {
        m = walk_chunk<D, G, S>(st.cur, a.ntrees, tile_lane, h, a.base);
      } else {
        m = walk_all<D, G, S>(a, st, tile_lane, h);
      }
      if (active && h == 0) {
        __builtin_nontemporal_store((uint8_t)((m > 0.0f) ? 1 : 0), a.valid_out + row);
        if (a.margin_out) __builtin_nontemporal_store(m, a.margin_out + row);
      }
    }
  };
  dispatch_rounds<S, RES>(a, rounds);
}

template <int D, int G, int S, bool RES>
__global__ void __launch_bounds__(kLanes *kMaxWaves) __attribute__((amdgpu_waves_per_eu(S, S)))
perf_kernel(WalkArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int wave_count[kMaxWaves];
  constexpr uint32_t RB = record_bytes(D);
  constexpr int CPW = Geo<S>::kCand;
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int h = lane / CPW;
  const int cl = lane % CPW;
  const int NT = a.nthreads;  // mask entries scanned per step
  const int W = NT / kLanes;
  const int C = W * CPW;      // candidates walked per round
  const int cand = wave * CPW + cl;
  const size_t tile_bytes = (size_t)a.F * Geo<S>::kRowBytes;
  const uint32_t chunk_bytes = (uint32_t)a.chunk_trees * RB;
  constexpr int K = stage_sets(D, S, kPerfSets);
  Stage<K, stage_regs(D, S)> st;
  st.cur = smem + W * tile_bytes;
  st.other = st.cur + (a.nbuf == 2 ? chunk_bytes : 0u);
  int32_t *queue = reinterpret_cast<int32_t *>(st.other + chunk_bytes);  // C + NT entries
  char *tile_lane = smem + wave * tile_bytes + 4 * cl;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t nsteps = (a.n + NT - 1) / NT;
  int64_t step = blockIdx.x;
  int qn = 0;    // identical in every thread
  int took = 0;  // rows the last next_rows() took (identical in every thread)
  stage_prime(a, RB, st);
  // Scan the mask NT entries at a time until C candidates are queued (or the
  // pool is exhausted), then take up to C rows off the queue.  The queue
  // never holds more than C - 1 + NT entries.
  auto next_rows = [&]() -> int32_t {
    while (qn < C && step < nsteps) {
      const int64_t i = step * NT + threadIdx.x;
      const bool in = i < a.n;
      const bool v = in && (a.valid_in == nullptr || a.valid_in[i] != 0);
      if (in && !v) __builtin_nontemporal_store(-INFINITY, a.score_out + i);
      const uint64_t bal = __ballot(v);
      if (lane == 0) wave_count[wave] = __popcll(bal);
      __syncthreads();
      int off = 0, tot = 0;
      for (int w = 0; w < W; ++w) {
        const int c = wave_count[w];
        off += (w < wave) ? c : 0;
        tot += c;
      }
      if (v) queue[qn + off + __popcll(bal & below)] = (int32_t)i;
      qn += tot;
      step += gridDim.x;
      __syncthreads();
    }
    const int take = min(qn, C);
    took = __builtin_amdgcn_readfirstlane(take);
    const int32_t r = (cand < take) ? queue[cand] : -1;
    const int rem = qn - take;  // < NT
    const int32_t carry = (threadIdx.x < rem) ? queue[take + threadIdx.x] : 0;
    __syncthreads();
    if (threadIdx.x < rem) queue[threadIdx.x] = carry;
    qn = rem;
    __syncthreads();
    return r;
  };
  auto rounds = [&](auto mode) {  // see validity_kernel
    constexpr int M = decltype(mode)::value;
    constexpr int E = M >= kResident ? row_extra_batches<S, K, stage_regs(D, S)>() : 0;
    // lines shared by the halves in the resident kernel only (10 % faster
    // there; the streamed walk ran 0.4 % slower with it)
    RowPrefetch<S, E, RES && S == 2> pf;
    const bool pfr = M != kAny || a.rowpf;  // rows prefetched
    int32_t row = next_rows();
    int cur = took;  // rows of this round: the loop ends where there are none
    if (pfr) pf.load(a, row, h);
    for (;;) {
      if (cur == 0) break;
      if (pfr)
        pf.commit(a, row, h, tile_lane);
      else if (row >= 0 && h == 0)
        load_row<S>(a, row, tile_lane);
      const int32_t nrow = next_rows();  // ends with a barrier: the tiles are complete
      const int ntook = took;
      if (pfr) {
        if constexpr (M == kResident)
          pf.template load_batch<0>(a, nrow, h);
        else
          pf.load(a, nrow, h);
      }
      float m;
      if constexpr (M == kResident) {
        m = walk_chunk_after<D, G, S>(st.cur, a.ntrees, tile_lane, h, a.base,
                                      [&](int g) { pf.load_after_group(a, nrow, h, g); });
        pf.load_rest(a, nrow, h, walk_groups<D, G, S>(a.ntrees));
      } else if constexpr (M == kResidentInline) {
        m = walk_chunk<D, G, S>(st.cur, a.ntrees, tile_lane, h, a.base);
      } else {
        m = walk_all<D, G, S>(a, st, tile_lane, h);
      }
      if (row >= 0 && h == 0) __builtin_nontemporal_store(m, a.score_out + row);
      row = nrow;
      cur = ntook;
    }
  };
  dispatch_rounds<S, RES>(a, rounds);
}

// Validity and performance in one pass over the pool (both ensembles
// resident in LDS, perfect trees of one depth): each round loads the rows of
// its tiles once and walks model V's trees followed by model P's on them as
// one list of trees, in groups of G*S; each leaf is added to V's margin or
// P's by its place in the list (V's trees first, in order, then P's), so
// both folds keep tree order.  It writes the mask, the margin and the score
// (-inf where V rejects; P is walked on every row, as the rows are on chip).
// Rows are prefetched a round ahead as in the resident walks (the next
// round's first batch before the walk, the second after the first group).
// LDS: W tiles, then V's nv records, P's first trees, and -0.0 trees up to a
// whole number of groups (ntrees records in all).
template <int D, int G, int S, typename After>
__device__ __forceinline__ float2 walk_split(const char *cb, int ntr, int nv,
                                             const char *tile_lane, int h, float mv, float mp,
                                             After after) {
  constexpr uint32_t RB = record_bytes(D);
  constexpr int GS = G * S;
  constexpr int H = G == 1 ? 1 : G / 2;
  auto add = [&](int t, float leaf) {
    const bool to_v = t < nv;
    mv = to_v ? mv + leaf : mv;
    mp = to_v ? mp : mp + leaf;
  };
  for (int t0 = 0; t0 < ntr; t0 += GS) {
    walk_group<D, G, S>(cb + (uint32_t)(t0 + h * G) * RB, tile_lane,
                        [&](const auto &A, const auto &B) {
      // this half's G trees t0 + h*G ..; the lower half adds its own, then
      // the upper half's (they cross over by one lane swap per tree)
      if constexpr (G == 1) {
        add(t0, A.leaf[0]);
        if constexpr (S == 2) add(t0 + 1, from_upper_half(A.leaf[0]));
      } else {
#pragma unroll
        for (int g = 0; g < H; ++g) add(t0 + g, A.leaf[g]);
#pragma unroll
        for (int g = 0; g < H; ++g) add(t0 + H + g, B.leaf[g]);
        if constexpr (S == 2) {
#pragma unroll
          for (int g = 0; g < H; ++g) add(t0 + G + g, from_upper_half(A.leaf[g]));
#pragma unroll
          for (int g = 0; g < H; ++g) add(t0 + G + H + g, from_upper_half(B.leaf[g]));
        }
      }
    });
    after(t0 / GS);
  }
  return make_float2(mv, mp);
}

template <int D, int G, int S>
__global__ void __launch_bounds__(kLanes *kMaxWaves) __attribute__((amdgpu_waves_per_eu(S, S)))
fused_kernel(WalkArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr uint32_t RB = record_bytes(D);
  constexpr uint32_t L = 1u << D;
  constexpr int CPW = Geo<S>::kCand;
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int h = lane / CPW;
  const int cl = lane % CPW;
  const int W = a.nthreads / kLanes;
  const size_t tile_bytes = (size_t)a.F * Geo<S>::kRowBytes;
  char *trees = smem + W * tile_bytes;
  char *tile_lane = smem + wave * tile_bytes + 4 * cl;
  {
    // V's nv records, P's np records after them, then records of -0.0
    // leaves (x + (-0.0) == x) up to ntrees
    const int nv = a.fold_trees, np = a.ntrees2;
    const uint32_t wv = (uint32_t)nv * (RB / 16u), wp = (uint32_t)np * (RB / 16u);
    const uint32_t wall = (uint32_t)a.ntrees * (RB / 16u);
    const u32x4 *sv = reinterpret_cast<const u32x4 *>(a.trees);
    const u32x4 *sp = reinterpret_cast<const u32x4 *>(a.trees2);
    u32x4 *d = reinterpret_cast<u32x4 *>(trees);
    for (uint32_t i = threadIdx.x; i < wall; i += a.nthreads) {
      u32x4 v;
      if (i < wv) {
        v = sv[i];
      } else if (i < wv + wp) {
        v = sp[i - wv];
      } else {  // leaf j (L <= j < 2L) at byte 4L + 4j: bytes 8L .. 12L of the record
        const uint32_t off = (i % (RB / 16u)) * 16u;
        const uint32_t z = (off >= 8u * L && off < 12u * L) ? 0x80000000u : 0u;
        v = u32x4{z, z, z, z};
      }
      d[i] = v;
    }
  }
  constexpr int E = S == 2 ? 1 : 0;
  RowPrefetch<S, E, S == 2, false> pf;
  const int64_t ntiles = (a.n + CPW - 1) / CPW;
  pf.load(a, ((int64_t)blockIdx.x * W + wave) * CPW + cl, h);
  __syncthreads();
  for (int64_t tg = blockIdx.x; tg * W < ntiles; tg += gridDim.x) {
    const int64_t row = (tg * W + wave) * CPW + cl;
    const bool active = row < a.n;
    const int64_t rn = ((tg + gridDim.x) * W + wave) * CPW + cl;
    pf.commit(a, row, h, tile_lane);
    pf.template load_batch<0>(a, rn, h);
    wave_sync();  // the ensembles are staged; a wave reads only its own tile
    const float2 m = walk_split<D, G, S>(trees, a.ntrees, a.fold_trees, tile_lane, h, a.base,
                                         a.base2,
                                         [&](int g) { pf.load_after_group(a, rn, h, g); });
    pf.load_rest(a, rn, h, (a.ntrees + G * S - 1) / (G * S));
    if (active && h == 0) {
      const bool ok = m.x > 0.0f;
      __builtin_nontemporal_store((uint8_t)(ok ? 1 : 0), a.valid_out + row);
      if (a.margin_out) __builtin_nontemporal_store(m.x, a.margin_out + row);
      __builtin_nontemporal_store(ok ? m.y : -INFINITY, a.score_out + row);
    }
  }
}

// Tree-parallel walk of a short row list (the second level): workgroup
// (c, r) stages tree chunk c once, loads list entries [r*64W, (r+1)*64W)
// (lane = entry) and writes the leaf each of its trees gives each entry to
// leaves_out[t * n + entry].  fold_kernel then adds them up in tree order, so
// a list of a few rows still spreads over the whole GPU.
template <int D, int G>
__global__ void __launch_bounds__(kLanes * 4) leaves_kernel(WalkArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr uint32_t RB = record_bytes(D);
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int W = a.nthreads / kLanes;
  const size_t tile_bytes = (size_t)a.F * Geo<1>::kRowBytes;
  char *chunk = smem + W * tile_bytes;
  const int r0 = blockIdx.x * a.chunk_trees;         // first record
  const int nr = min(a.chunk_trees, a.ntrees - r0);  // records (a multiple of G if perfect)
  const u32x4 *src = reinterpret_cast<const u32x4 *>(a.trees + (size_t)r0 * RB);
  for (uint32_t i = threadIdx.x; i < (uint32_t)nr * (RB / 16u); i += a.nthreads)
    reinterpret_cast<u32x4 *>(chunk)[i] = src[i];
  const int64_t pos = ((int64_t)blockIdx.y * W + wave) * kLanes + lane;
  int64_t row = -1;
  if (pos < a.n) {
    const int32_t r = a.rows_in[pos];
    if (r >= 0 && r < a.n_pool) row = r;
  }
  char *tile_lane = smem + wave * tile_bytes + 4 * lane;
  if (row >= 0) load_row<1>(a, row, tile_lane);
  __syncthreads();
  // the leaves of trees t .. t+G-1 of the ensemble
  auto store = [&](int t, const auto &A, const auto &B) {
    if (row < 0) return;
    float *out = a.leaves_out + (size_t)t * a.n + pos;
    constexpr int H = G == 1 ? 1 : G / 2;
#pragma unroll
    for (int g = 0; g < H; ++g) out[(size_t)g * a.n] = A.leaf[g];
    if constexpr (G > 1) {
#pragma unroll
      for (int g = 0; g < H; ++g) out[(size_t)(H + g) * a.n] = B.leaf[g];
    }
  };
  if constexpr (D == 0) {
    for (int i = 0; i < nr; ++i) {
      const char *slot = chunk + (uint32_t)i * RB;
      const SlotHead hd = slot_head(slot);
      const uint32_t *roots = reinterpret_cast<const uint32_t *>(slot + 16);
      for (int g0 = 0; g0 < hd.ntrees; g0 += G)
        walk_group_ragged<G, 1>(slot, roots + g0, hd.depth, tile_lane,
                                [&](const auto &A, const auto &B) { store(hd.tree0 + g0, A, B); });
    }
  } else {
    for (int g0 = 0; g0 < nr; g0 += G)
      walk_group<D, G, 1>(chunk + (uint32_t)g0 * RB, tile_lane,
                          [&](const auto &A, const auto &B) { store(r0 + g0, A, B); });
  }
}

// score_out[i] = base + leaf_0 + leaf_1 + ... (float32, tree order) for list
// entries whose row is in the pool, -inf for the others.
__global__ void __launch_bounds__(256) fold_kernel(WalkArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int32_t r = a.rows_in[i];
  if (r < 0 || r >= a.n_pool) {
    a.score_out[i] = -INFINITY;
    return;
  }
  float m = a.base;
  for (int t = 0; t < a.fold_trees; ++t) m = m + a.leaves_out[(size_t)t * a.n + i];
  a.score_out[i] = m;
}

// Trees walked concurrently per lane that a depth allows.  S = 1: a chunk
// must hold at least G whole trees.  S = 2: a 24 KiB register-staged chunk
// must hold the 2G trees of a group.
constexpr bool group_allowed(int d, int g, int s) {
  if (d == 0) return kRaggedGroup % (g * s) == 0 && g <= 4;  // ragged slots
  if (s == 2)
    return d <= 7 ? (g == 4 || g == 8)
         : d == 8 ? (g == 2 || g == 4)
         : d == 9 ? (g == 1 || g == 2)
         : d == 10 ? (g == 1)
                   : false;
  return d <= 9 ? (g == 4 || g == 8)
       : d == 10 ? (g == 2 || g == 4)
                 : (g == 1 || g == 2);
}

// ---- visit probe -----------------------------------------------------------

// 32-bit integer hash: the xorshift-multiply "lowbias32" constants found by
// C. Wellons' hash-prospector search (2018).
__device__ __forceinline__ uint32_t probe_hash(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}
__device__ __forceinline__ float probe_unit(uint32_t i) {  // in [0, 1)
  return (float)(probe_hash(i) >> 8) * (1.0f / 16777216.0f);
}

// The walks' inner loop alone: each workgroup fills its LDS with W candidate
// tiles of F pseudo-random features in [0, 1) and one chunk of G*S perfect
// trees of depth D (random split features below F, thresholds in [0, 1),
// random leaves), then walks that chunk `iters` times with walk_chunk: the
// node and feature reads, the child steps and the fold, without row loads,
// restaging or barriers.  Every address stays in the tiles and the chunk.
template <int D, int G, int S>
__global__ void __launch_bounds__(kLanes *kMaxWaves) __attribute__((amdgpu_waves_per_eu(S, S)))
visit_probe_kernel(float *out, int iters, int F, int W) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr uint32_t RB = record_bytes(D);
  constexpr uint32_t L = 1u << D;
  constexpr int CPW = Geo<S>::kCand;
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int h = lane / CPW;
  const int cl = lane % CPW;
  const uint32_t nthreads = (uint32_t)W * kLanes;
  const uint32_t tile_bytes = (uint32_t)F * Geo<S>::kRowBytes;
  char *chunk = smem + (uint32_t)W * tile_bytes;
  float *tiles = reinterpret_cast<float *>(smem);
  for (uint32_t i = threadIdx.x; i < (uint32_t)W * tile_bytes / 4u; i += nthreads)
    tiles[i] = probe_unit(i + 0x51ED27u * blockIdx.x);
  for (uint32_t i = threadIdx.x; i < (uint32_t)(G * S) * L; i += nthreads) {
    const uint32_t t = i / L, j = i % L;
    char *rec = chunk + t * RB;
    if (j >= 1)
      reinterpret_cast<uint2 *>(rec)[j] =
          make_uint2(probe_hash(i ^ 0xA5A5A5u) % (uint32_t)F, __float_as_uint(probe_unit(i * 3u)));
    reinterpret_cast<float *>(rec + 4u * L)[L + j] = probe_unit(i * 5u + 1u) - 0.5f;
  }
  __syncthreads();
  const char *tile_lane = smem + (uint32_t)wave * tile_bytes + 4u * (uint32_t)cl;
  float m = 0.0f;
  for (int it = 0; it < iters; ++it) m = walk_chunk<D, G, S>(chunk, G * S, tile_lane, h, m);
  if (h == 0) out[((size_t)blockIdx.x * W + wave) * CPW + cl] = m;
}

template <int D, int G, int S, bool RES>
hipError_t launch_kernel(bool perf, const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  const void *fn = perf ? reinterpret_cast<const void *>(&perf_kernel<D, G, S, RES>)
                        : reinterpret_cast<const void *>(&validity_kernel<D, G, S, RES>);
  hipError_t e = ensure_dynamic_lds(fn, p.lds_bytes);
  if (e != hipSuccess) return e;
  dim3 grid(p.grid), block(p.waves * kLanes);
  if (perf)
    hipLaunchKernelGGL((perf_kernel<D, G, S, RES>), grid, block, p.lds_bytes, s, a);
  else
    hipLaunchKernelGGL((validity_kernel<D, G, S, RES>), grid, block, p.lds_bytes, s, a);
  return hipGetLastError();
}

template <int D, int G, int S>
hipError_t launch_dgs(bool perf, const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  // Chunks hold whole groups: every chunk's tree count, including the last
  // one's, is a multiple of the padding and hence of the group.
  static_assert((D == 0 ? kRaggedGroup : kTreePad) % (G * S) == 0,
                "a walk group must divide the tree padding");
  if constexpr (S == 2) {
    if (resident_launch(S, a)) return launch_kernel<D, G, S, true>(perf, p, a, s);
  }
  return launch_kernel<D, G, S, false>(perf, p, a, s);
}

template <int D, int S>
hipError_t launch_ds(bool perf, const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  switch (p.group) {
    case 1: if constexpr (group_allowed(D, 1, S)) return launch_dgs<D, 1, S>(perf, p, a, s); break;
    case 2: if constexpr (group_allowed(D, 2, S)) return launch_dgs<D, 2, S>(perf, p, a, s); break;
    case 4: if constexpr (group_allowed(D, 4, S)) return launch_dgs<D, 4, S>(perf, p, a, s); break;
    case 8: if constexpr (group_allowed(D, 8, S)) return launch_dgs<D, 8, S>(perf, p, a, s); break;
    case 16: if constexpr (group_allowed(D, 16, S)) return launch_dgs<D, 16, S>(perf, p, a, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_depth(bool perf, const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  if (p.split == 2) {
    if constexpr (D <= 10) return launch_ds<D, 2>(perf, p, a, s);  // D == 0: ragged
    return hipErrorInvalidValue;
  }
  return launch_ds<D, 1>(perf, p, a, s);
}

hipError_t launch_walk(bool perf, const Forest &f, const WalkPlan &p, const WalkArgs &a,
                       hipStream_t s) {
  if (f.ragged) return launch_depth<0>(perf, p, a, s);
  switch (f.depth) {
    case 1: return launch_depth<1>(perf, p, a, s);
    case 2: return launch_depth<2>(perf, p, a, s);
    case 3: return launch_depth<3>(perf, p, a, s);
    case 4: return launch_depth<4>(perf, p, a, s);
    case 5: return launch_depth<5>(perf, p, a, s);
    case 6: return launch_depth<6>(perf, p, a, s);
    case 7: return launch_depth<7>(perf, p, a, s);
    case 8: return launch_depth<8>(perf, p, a, s);
    case 9: return launch_depth<9>(perf, p, a, s);
    case 10: return launch_depth<10>(perf, p, a, s);
    case 11: return launch_depth<11>(perf, p, a, s);
    case 12: return launch_depth<12>(perf, p, a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int D, int G>
hipError_t launch_leaves_dg(const WalkArgs &a, int W, size_t lds, int row_tiles, hipStream_t s) {
  const void *fn = reinterpret_cast<const void *>(&leaves_kernel<D, G>);
  hipError_t e = ensure_dynamic_lds(fn, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((leaves_kernel<D, G>), dim3((unsigned)a.nchunks, (unsigned)row_tiles),
                     dim3(W * kLanes), lds, s, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_leaves_depth(const WalkArgs &a, int G, int W, size_t lds, int row_tiles,
                               hipStream_t s) {
  switch (G) {
    case 1: if constexpr (group_allowed(D, 1, 1)) return launch_leaves_dg<D, 1>(a, W, lds, row_tiles, s); break;
    case 2: if constexpr (group_allowed(D, 2, 1)) return launch_leaves_dg<D, 2>(a, W, lds, row_tiles, s); break;
    case 4: if constexpr (group_allowed(D, 4, 1)) return launch_leaves_dg<D, 4>(a, W, lds, row_tiles, s); break;
    case 8: if constexpr (group_allowed(D, 8, 1)) return launch_leaves_dg<D, 8>(a, W, lds, row_tiles, s); break;
    case 16: if constexpr (group_allowed(D, 16, 1)) return launch_leaves_dg<D, 16>(a, W, lds, row_tiles, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

hipError_t launch_leaves(int depth, const WalkArgs &a, int G, int W, size_t lds, int row_tiles,
                         hipStream_t s) {
  switch (depth) {
    case 0: return launch_leaves_depth<0>(a, G, W, lds, row_tiles, s);
    case 1: return launch_leaves_depth<1>(a, G, W, lds, row_tiles, s);
    case 2: return launch_leaves_depth<2>(a, G, W, lds, row_tiles, s);
    case 3: return launch_leaves_depth<3>(a, G, W, lds, row_tiles, s);
    case 4: return launch_leaves_depth<4>(a, G, W, lds, row_tiles, s);
    case 5: return launch_leaves_depth<5>(a, G, W, lds, row_tiles, s);
    case 6: return launch_leaves_depth<6>(a, G, W, lds, row_tiles, s);
    case 7: return launch_leaves_depth<7>(a, G, W, lds, row_tiles, s);
    case 8: return launch_leaves_depth<8>(a, G, W, lds, row_tiles, s);
    case 9: return launch_leaves_depth<9>(a, G, W, lds, row_tiles, s);
    case 10: return launch_leaves_depth<10>(a, G, W, lds, row_tiles, s);
    case 11: return launch_leaves_depth<11>(a, G, W, lds, row_tiles, s);
    case 12: return launch_leaves_depth<12>(a, G, W, lds, row_tiles, s);
    default: return hipErrorInvalidValue;
  }
}

std::atomic<int> g_tune[kTuneFields];

size_t stage_reg_bytes(const WalkPlan &p, int depth) {
  return (size_t)stage_regs(depth, p.split) * 16 * kLanes * p.waves;
}

WalkArgs make_args(const Forest &f, const WalkPlan &p, const float *X, int64_t n, int64_t ld) {
  WalkArgs a{};
  a.X = X;
  a.n = n;
  a.n_pool = n;
  a.ld = ld;
  a.trees = static_cast<const char *>(f.d_trees);
  a.ntrees = f.records;  // staged records: perfect trees or ragged slots
  a.chunk_trees = p.chunk_trees;
  a.nchunks = (f.records + p.chunk_trees - 1) / p.chunk_trees;
  a.F = f.num_features;
  a.vec4 = ((reinterpret_cast<uintptr_t>(X) & 15u) == 0 && (ld & 3) == 0) ? 1 : 0;
  a.nbuf = p.nbuf;
  a.regstage = (p.nbuf == 1 &&
                 (size_t)p.chunk_trees * f.rec_bytes <= stage_reg_bytes(p, f.ragged ? 0 : f.depth))
                    ? 1
                    : 0;
  a.rowpf = (a.vec4 && (f.num_features % 4) == 0 && f.num_features <= 4 * kRowVecs) ? 1 : 0;
  a.nthreads = p.waves * kLanes;
  a.base = f.base;
  return a;
}

// One candidate plan: S lanes per candidate, W waves, staging mode (0: one
// buffer refilled from registers, 1: two buffers, 2: one buffer copied
// synchronously), G trees per lane.  Returns false if it does not fit.
bool try_plan(const Forest &f, int64_t n_work, int cu_count, int S, int W, int mode, int G,
              int want_c, WalkPlan *p) {
  const int D = f.ragged ? 0 : f.depth;
  if (!group_allowed(D, G, S) || W < 1 || W > kMaxWaves) return false;
  // two lanes per candidate: register staging only (two buffers filled by
  // direct global-to-LDS copies were 12 to 75 % slower where they fit)
  if (S == 2 && mode != 0) return false;
  const size_t rb = f.rec_bytes;
  const int cpw = kLanes / S;
  const size_t tile = (size_t)f.num_features * 4 * cpw;
  // tiles + the perf queue (C + NT entries, C = W * cpw, NT = 64 W)
  const size_t fixed = (size_t)W * (tile + (size_t)(cpw + kLanes) * sizeof(int32_t));
  const int nbuf = mode == 1 ? 2 : 1;
  const int gs = f.ragged ? 1 : G * S;  // records per group (a ragged slot holds whole groups)
  if (fixed + (size_t)nbuf * gs * rb > kLdsBudget) return false;
  const size_t room = (kLdsBudget - fixed) / nbuf;
  const int tpad = (f.records + gs - 1) / gs * gs;
  int chunk_trees = (int)(room / rb) / gs * gs;
  WalkPlan q{};
  q.split = S;
  q.waves = W;
  if (mode == 0) {  // the chunk must fit the staging registers
    const int reg_trees = (int)(stage_reg_bytes(q, D) / rb) / gs * gs;
    if (reg_trees < gs) return false;
    if (chunk_trees > reg_trees) chunk_trees = reg_trees;
  }
  if (want_c > 0 && want_c % gs == 0 && want_c <= chunk_trees) chunk_trees = want_c;
  if (chunk_trees > tpad) chunk_trees = tpad;
  q.group = G;
  q.chunk_trees = chunk_trees;
  q.nbuf = nbuf;
  q.lds_bytes = fixed + (size_t)nbuf * chunk_trees * rb;
  int per_cu = (int)(kLdsBudget / q.lds_bytes);
  if (per_cu < 1) per_cu = 1;
  if (per_cu > 8) per_cu = 8;
  const int64_t tiles = (n_work + cpw - 1) / cpw;
  const int64_t wgs = (tiles + W - 1) / W;
  int64_t grid = (int64_t)cu_count * per_cu;
  if (wgs < grid) grid = wgs;
  if (grid < 1) grid = 1;
  q.grid = (int)grid;
  *p = q;
  return true;
}

// One pass over the pool: depths 1..8, (G, S) with G*S dividing the tree
// padding.
template <int D, int G, int S>
hipError_t launch_fused_dgs(const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  static_assert(kTreePad % (G * S) == 0, "a walk group must divide the tree padding");
  const void *fn = reinterpret_cast<const void *>(&fused_kernel<D, G, S>);
  hipError_t e = ensure_dynamic_lds(fn, p.lds_bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((fused_kernel<D, G, S>), dim3(p.grid), dim3(p.waves * kLanes), p.lds_bytes,
                     s, a);
  return hipGetLastError();
}

template <int D, int S>
hipError_t launch_fused_ds(const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  switch (p.group) {
    case 1: if constexpr (group_allowed(D, 1, S)) return launch_fused_dgs<D, 1, S>(p, a, s); break;
    case 2: if constexpr (group_allowed(D, 2, S)) return launch_fused_dgs<D, 2, S>(p, a, s); break;
    case 4: if constexpr (group_allowed(D, 4, S)) return launch_fused_dgs<D, 4, S>(p, a, s); break;
    case 8: if constexpr (group_allowed(D, 8, S) && 8 * S <= kTreePad) return launch_fused_dgs<D, 8, S>(p, a, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_fused_d(const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  return p.split == 2 ? launch_fused_ds<D, 2>(p, a, s) : launch_fused_ds<D, 1>(p, a, s);
}

}  // namespace

// One pass over the pool for V and P: both perfect, of one depth (at most
// kMaxFusedDepth), rows prefetchable (16-byte aligned, F a multiple of 4,
// at most 128 features), and the W candidate tiles plus both ensembles'
// trees (their sum rounded up to a whole number of groups) within one
// workgroup's LDS.  Shapes tried: eight waves with one lane per candidate,
// eight with two, then four of each (a pool of less than one eight-wave
// round per CU: four waves with two lanes first); larger groups first.  The
// tuning overrides of the split and the waves apply here too.  *nv: V's trees,
// *np: P's trees staged (all of them).
bool plan_fused(const Forest &v, const Forest &p, int64_t n, int64_t ld, const float *X,
                int cu_count, WalkPlan *plan, int *nv, int *np) {
  if (v.ragged || p.ragged || v.depth != p.depth || v.depth > kMaxFusedDepth) return false;
  const int F = v.num_features > p.num_features ? v.num_features : p.num_features;
  const bool vec4 = (reinterpret_cast<uintptr_t>(X) & 15u) == 0 && (ld & 3) == 0;
  if (!vec4 || F % 4 != 0 || F > 4 * kRowVecs) return false;
  const int D = v.depth;
  const size_t rb = v.rec_bytes;
  struct Shape { int s, w; };
  const Shape shapes[] = {{1, 8}, {2, 8}, {1, 4}, {2, 4}};
  // A pool of less than one eight-wave round per CU leaves most CUs idle:
  // four-wave workgroups with two lanes per candidate spread it over more
  // CUs and halve each lane's chain of trees (Tiny: 0.025 -> 0.019 ms).
  const Shape small[] = {{2, 4}, {2, 8}, {1, 8}, {1, 4}};
  const bool few = n <= (int64_t)kLanes * 8 * cu_count;
  // the tuning overrides force the split and the waves where they fit
  const int want_s = get_tune(kTuneSplit), want_w = get_tune(kTuneWaves);
  const Shape forced = {want_s ? want_s : 1, want_w};
  const bool force = want_w > 0;
  const Shape *list = force ? &forced : few ? small : shapes;
  const int nshapes = force ? 1 : 4;
  for (int si = 0; si < nshapes; ++si) {
    const Shape &sh = list[si];
    for (int G : {8, 4, 2, 1}) {
      const int gs = G * sh.s;
      if (!group_allowed(D, G, sh.s) || kTreePad % gs != 0) continue;
      const int all = (v.num_trees + p.num_trees + gs - 1) / gs * gs;
      const size_t tile = (size_t)F * 4 * (kLanes / sh.s);
      const size_t lds = (size_t)sh.w * tile + (size_t)all * rb;
      if (lds > kLdsBudget) continue;
      WalkPlan q{};
      q.split = sh.s;
      q.waves = sh.w;
      q.group = G;
      q.chunk_trees = all;
      q.nbuf = 1;
      q.lds_bytes = lds;
      int per_cu = (int)(kLdsBudget / lds);
      if (per_cu < 1) per_cu = 1;
      if (per_cu > 8) per_cu = 8;
      const int64_t tiles = (n + kLanes / sh.s - 1) / (kLanes / sh.s);
      int64_t grid = (tiles + sh.w - 1) / sh.w;
      if (grid > (int64_t)cu_count * per_cu) grid = (int64_t)cu_count * per_cu;
      if (grid < 1) grid = 1;
      q.grid = (int)grid;
      *plan = q;
      *nv = v.num_trees;
      *np = p.num_trees;
      return true;
    }
  }
  return false;
}

hipError_t launch_fused(const Forest &v, const Forest &p, const WalkPlan &pl, int nv, int np,
                        const float *X, int64_t n, int64_t ld, uint8_t *valid_out,
                        float *margin_out, float *score_out, hipStream_t s) {
  WalkArgs a{};
  a.X = X;
  a.n = n;
  a.n_pool = n;
  a.ld = ld;
  a.trees = static_cast<const char *>(v.d_trees);
  a.fold_trees = nv;  // V's trees: the first nv of the list
  a.trees2 = static_cast<const char *>(p.d_trees);
  a.ntrees2 = np;
  a.ntrees = pl.chunk_trees;  // the list, padded to whole groups
  a.chunk_trees = pl.chunk_trees;
  a.nchunks = 1;
  a.F = v.num_features > p.num_features ? v.num_features : p.num_features;
  a.vec4 = 1;
  a.nbuf = 1;
  a.rowpf = 1;
  a.nthreads = pl.waves * kLanes;
  a.base = v.base;
  a.base2 = p.base;
  a.valid_out = valid_out;
  a.margin_out = margin_out;
  a.score_out = score_out;
  switch (v.depth) {
    case 1: return launch_fused_d<1>(pl, a, s);
    case 2: return launch_fused_d<2>(pl, a, s);
    case 3: return launch_fused_d<3>(pl, a, s);
    case 4: return launch_fused_d<4>(pl, a, s);
    case 5: return launch_fused_d<5>(pl, a, s);
    case 6: return launch_fused_d<6>(pl, a, s);
    case 7: return launch_fused_d<7>(pl, a, s);
    case 8: return launch_fused_d<8>(pl, a, s);
    default: return hipErrorInvalidValue;
  }
}

void set_tune(int field, int value) { g_tune[field].store(value, std::memory_order_relaxed); }
int get_tune(int field) { return g_tune[field].load(std::memory_order_relaxed); }

// LDS of one workgroup = W candidate tiles (F * 256 / S bytes each, plus the
// compaction queue share) + nbuf chunk buffers of chunk_trees whole trees
// (a multiple of S*G, as large as the LDS allows).  Preference: eight waves
// (two per SIMD), with one lane per candidate where eight full tiles fit
// (twice the candidates per pass over the ensemble), else two; then one lane
// per candidate with four waves in the order register staging, two buffers,
// synchronous copy; then fewer waves.  Larger G first within each (ragged
// trees with one lane per candidate: smaller G first).  Deep perfect trees
// with one lane per candidate take six waves of four trees per lane over
// eight waves of fewer.  A walk over the survivors of a small pool (at most
// four one-lane rounds per workgroup were every row accepted) takes two
// lanes per candidate instead: a workgroup's survivors fill its last round
// only in part, and rounds of half the candidates halve that idle part
// (Medium's perf walk 0.096 -> 0.082 ms).  The tuning overrides
// (ml2_tune_walk_plan) replace the choice where they fit; overrides that do
// not fit are ignored.
bool plan_walk(const Forest &f, int64_t n_work, int cu_count, WalkPlan *p, const char **why,
               bool survivors) {
  const int want_s = get_tune(kTuneSplit);
  const int want_g = get_tune(kTuneGroup);
  const int want_w = get_tune(kTuneWaves);
  const int want_b = get_tune(kTuneNbuf);
  const int want_c = get_tune(kTuneChunk);
  const int groups[5] = {16, 8, 4, 2, 1};
  // ragged trees with one lane per candidate: one tree per lane first (each
  // lane then moves to its next tree as soon as its walk is on a leaf, and
  // no walk waits for a longer one of its lane)
  const int ragged_groups[5] = {1, 2, 4, 0, 0};
  struct Shape { int s, w; };
  const Shape shapes[] = {{1, 8}, {2, 8}, {1, 4}, {2, 4}, {1, 2}, {1, 1}};
  const bool forced = want_s || want_g || want_w || want_b || want_c;
  for (int pass = 0; pass < 2; ++pass) {  // pass 0 honours the overrides
    for (const Shape &sh : shapes) {
      int S = sh.s, W = sh.w;
      if (pass == 0) {
        if (want_s && want_s != S) continue;
        if (want_w > 0) W = want_w;
      }
      for (int mode = 0; mode < 3; ++mode) {
        if (pass == 0 && want_b && want_b != (mode == 1 ? 2 : 1)) continue;
        for (int G : (f.ragged && S == 1) ? ragged_groups : groups) {
          if (G == 0) break;
          if (pass == 0 && want_g && group_allowed(f.ragged ? 0 : f.depth, want_g, S) &&
              G != want_g)
            continue;
          if (!try_plan(f, n_work, cu_count, S, W, mode, G, pass == 0 ? want_c : 0, p)) continue;
          // Deep perfect trees (12 KiB and more) with one lane per candidate:
          // where eight tiles leave room for fewer than four trees per lane,
          // six waves with four (a chunk twice as long, half the restaging
          // per visit) are faster.
          WalkPlan q;
          if (!forced && !f.ragged && S == 1 && W == 8 && mode == 0 && G < 4 &&
              try_plan(f, n_work, cu_count, 1, 6, 0, 4, 0, &q))
            *p = q;
          else if (!forced && survivors && !f.ragged && f.depth < 10 && S == 1 && W == 8 &&
                   n_work <= (int64_t)4 * W * Geo<1>::kCand * cu_count) {
            for (int G2 : groups) {
              if (try_plan(f, n_work, cu_count, 2, 8, 0, G2, 0, &q)) {
                *p = q;
                break;
              }
            }
          }
          return true;
        }
      }
    }
  }
  *why = "ensemble depth and feature count exceed the LDS of one workgroup";
  return false;
}

hipError_t launch_validity(const Forest &f, const WalkPlan &p, const float *X, int64_t n,
                           int64_t ld, uint8_t *valid_out, float *margin_out, hipStream_t s) {
  WalkArgs a = make_args(f, p, X, n, ld);
  a.valid_out = valid_out;
  a.margin_out = margin_out;
  return launch_walk(false, f, p, a, s);
}

hipError_t launch_perf(const Forest &f, const WalkPlan &p, const float *X, int64_t n,
                       int64_t ld, const uint8_t *valid, float *score_out, hipStream_t s) {
  WalkArgs a = make_args(f, p, X, n, ld);
  a.valid_in = valid;
  a.score_out = score_out;
  return launch_walk(true, f, p, a, s);
}

size_t rows_workspace_bytes(const Forest &f, int32_t m) {
  const size_t b = (size_t)f.num_trees_padded * (size_t)(m > 0 ? m : 1) * sizeof(float);
  return (b + 255) & ~(size_t)255;
}

// Tree-parallel walk of m listed rows: W waves of 64 entries per workgroup
// (as many as the list needs, at most four, fewer if the tiles and G trees
// do not fit), chunks of whole trees sized so the grid holds about two
// workgroups per CU, then the ordered fold.
hipError_t launch_rows(const Forest &f, const float *X, int64_t n, int64_t ld, const int32_t *rows,
                       int32_t m, float *score_out, void *ws, int cu_count, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  const size_t rb = f.rec_bytes;
  const int D = f.ragged ? 0 : f.depth;
  const size_t tile = (size_t)f.num_features * Geo<1>::kRowBytes;
  int W = (int)std::min<int64_t>(4, (m + kLanes - 1) / kLanes);
  int G = 0;
  for (; W >= 1; --W) {
    for (int g : {16, 8, 4, 2, 1}) {
      const size_t recs = f.ragged ? 1 : (size_t)g;  // records one group needs
      if (group_allowed(D, g, 1) && W * tile + recs * rb <= kLdsBudget) {
        G = g;
        break;
      }
    }
    if (G) break;
  }
  if (!G) return hipErrorInvalidValue;  // excluded by the loader's limits
  const int row_tiles = (int)((m + (int64_t)W * kLanes - 1) / ((int64_t)W * kLanes));
  const int tpad = f.records;  // perfect: a multiple of kTreePad, hence of G
  const int gr = f.ragged ? 1 : G;  // records per group
  int ct = (int)((kLdsBudget - W * tile) / rb) / gr * gr;
  const int64_t want = 2 * (int64_t)cu_count;  // workgroups wanted in flight
  const int64_t chunks_wanted = (want + row_tiles - 1) / row_tiles;
  const int cap = (int)std::max<int64_t>(gr, (tpad / std::max<int64_t>(chunks_wanted, 1)) / gr * gr);
  ct = std::min(std::min(ct, cap), tpad);
  WalkArgs a{};
  a.X = X;
  a.n = m;
  a.n_pool = n;
  a.ld = ld;
  a.trees = static_cast<const char *>(f.d_trees);
  a.ntrees = tpad;  // records
  a.chunk_trees = ct;
  a.nchunks = (tpad + ct - 1) / ct;
  a.F = f.num_features;
  a.vec4 = ((reinterpret_cast<uintptr_t>(X) & 15u) == 0 && (ld & 3) == 0) ? 1 : 0;
  a.nthreads = W * kLanes;
  a.base = f.base;
  a.rows_in = rows;
  a.score_out = score_out;
  a.leaves_out = static_cast<float *>(ws);
  a.fold_trees = f.num_trees_padded;
  const size_t lds = W * tile + (size_t)ct * rb;
  hipError_t e = launch_leaves(D, a, G, W, lds, row_tiles, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(fold_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int D, int G, int S>
hipError_t launch_visit_probe_dgs(int waves, int features, int iters, int blocks, float *out,
                                  double *visits, hipStream_t s) {
  const void *fn = reinterpret_cast<const void *>(&visit_probe_kernel<D, G, S>);
  const size_t lds =
      (size_t)waves * features * Geo<S>::kRowBytes + (size_t)G * S * record_bytes(D);
  if (lds > kLdsBudget) return hipErrorInvalidValue;
  hipError_t e = ensure_dynamic_lds(fn, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((visit_probe_kernel<D, G, S>), dim3(blocks), dim3(waves * kLanes), lds, s,
                     out, iters, features, waves);
  // candidates x trees x levels
  *visits = (double)blocks * waves * Geo<S>::kCand * (double)iters * G * S * D;
  return hipGetLastError();
}

template <int D>
hipError_t launch_visit_probe_d(int G, int S, int waves, int features, int iters, int blocks,
                                float *out, double *visits, hipStream_t s) {
  if (S == 1) {
    switch (G) {
      case 1: return launch_visit_probe_dgs<D, 1, 1>(waves, features, iters, blocks, out, visits, s);
      case 2: return launch_visit_probe_dgs<D, 2, 1>(waves, features, iters, blocks, out, visits, s);
      case 4: return launch_visit_probe_dgs<D, 4, 1>(waves, features, iters, blocks, out, visits, s);
      case 8: return launch_visit_probe_dgs<D, 8, 1>(waves, features, iters, blocks, out, visits, s);
      default: break;
    }
  } else if (S == 2) {
    switch (G) {
      case 1: return launch_visit_probe_dgs<D, 1, 2>(waves, features, iters, blocks, out, visits, s);
      case 2: return launch_visit_probe_dgs<D, 2, 2>(waves, features, iters, blocks, out, visits, s);
      case 4: return launch_visit_probe_dgs<D, 4, 2>(waves, features, iters, blocks, out, visits, s);
      case 8: return launch_visit_probe_dgs<D, 8, 2>(waves, features, iters, blocks, out, visits, s);
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

// The visit probe: depth 6, 8 or 10; G in {1, 2, 4, 8}, S in {1, 2}; 1 to 8
// waves; 64 or 128 features; the tiles and the chunk must fit the LDS of one
// workgroup.  out: blocks * 512 floats.
hipError_t launch_visit_probe(int depth, int G, int S, int waves, int features, int iters,
                              int blocks, float *out, double *visits, hipStream_t s) {
  if (waves < 1 || waves > kMaxWaves || (features != 64 && features != 128))
    return hipErrorInvalidValue;
  if (depth == 6)
    return launch_visit_probe_d<6>(G, S, waves, features, iters, blocks, out, visits, s);
  if (depth == 8)
    return launch_visit_probe_d<8>(G, S, waves, features, iters, blocks, out, visits, s);
  if (depth == 10)
    return launch_visit_probe_d<10>(G, S, waves, features, iters, blocks, out, visits, s);
  return hipErrorInvalidValue;
}

}  // namespace ml2
