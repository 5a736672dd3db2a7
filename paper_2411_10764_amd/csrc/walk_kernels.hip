// Tree-ensemble walks on gfx950: the validity filter (model V) and the
// performance prediction over accepted candidates (model P) of ML2Tuner's
// configuration explorer (Section 2, "ML Model P" / "ML Model V").
//
// Mapping (one workgroup = W waves, persistent over the pool):
//   * lane = candidate.  Each wave owns a tile of 64 candidates whose
//     features sit in LDS transposed, feature f of lane l at f*256 + 4*l, so
//     the per-level feature reads of a wave hit 64 distinct banks whatever
//     features the lanes' current nodes test.
//   * All lanes of a wave walk the same trees in lockstep (the trees are
//     perfect), so at level l the wave touches only the 2^l breadth-ordered
//     nodes of that level: reads are broadcast or conflict-free.
//   * The ensemble streams through LDS in chunks of whole trees, double
//     buffered with direct global->LDS loads (global_load_lds_dwordx4); the
//     next chunk is in flight while the current one is walked.
//   * Each lane walks `G` trees at once (independent dependency chains) and
//     adds their leaves to its running margin in tree-index order, so the
//     float32 left fold is exactly the one the definition prescribes.
//   * The performance pass compacts the accepted candidates of the pool into
//     an LDS queue (wave ballots + a workgroup prefix) and only ever walks
//     full tiles of accepted candidates; rejected ones get -inf directly.
#include <math.h>

#include "ml2_internal.h"

namespace ml2 {
namespace {

constexpr int kLanes = 64;
constexpr int kTileStride = kLanes * 4;  // bytes per feature row of a wave tile
constexpr size_t kLdsBudget = 160 * 1024 - 256;  // headroom for static LDS
constexpr int kMaxWaves = 8;

struct WalkArgs {
  const float *X;
  int64_t n;
  int64_t ld;
  const char *trees;
  int32_t ntrees;       // padded tree count
  int32_t chunk_trees;
  int32_t nchunks;
  int32_t F;
  int32_t vec4;         // rows are 16-byte aligned (X aligned, ld % 4 == 0)
  int32_t nbuf;         // 2: double-buffered chunks; 1: one buffer (deep trees, wide F)
  float base;
  uint8_t *valid_out;   // validity
  float *margin_out;
  const uint8_t *valid_in;  // perf
  float *score_out;
};

typedef __attribute__((address_space(3))) void lds_void;

// Issue the asynchronous copy of `bytes` (multiple of 16) from global src to
// LDS dst; every wave takes 1 KiB segments round-robin.  Completion is
// awaited with s_waitcnt vmcnt(0) followed by a workgroup barrier.
__device__ __forceinline__ void stage_async(const char *src, char *dst, uint32_t bytes,
                                            int wave, int nwaves, int lane) {
  for (uint32_t seg = (uint32_t)wave * 1024u; seg < bytes; seg += (uint32_t)nwaves * 1024u) {
    const uint32_t off = seg + (uint32_t)lane * 16u;
    if (off < bytes)
      __builtin_amdgcn_global_load_lds((const void *)(src + off), (lds_void *)(dst + seg), 16, 0, 0);
  }
}

__device__ __forceinline__ void wait_all_and_barrier() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Row `row` of X into the wave tile, transposed (dst = tile + 4*lane).
__device__ __forceinline__ void load_row(const WalkArgs &a, int64_t row, char *dst) {
  const float *src = a.X + row * a.ld;
  int q = 0;
  if (a.vec4) {
    for (; q + 4 <= a.F; q += 4) {
      const float4 v = *reinterpret_cast<const float4 *>(src + q);
      *reinterpret_cast<float *>(dst + (q + 0) * kTileStride) = v.x;
      *reinterpret_cast<float *>(dst + (q + 1) * kTileStride) = v.y;
      *reinterpret_cast<float *>(dst + (q + 2) * kTileStride) = v.z;
      *reinterpret_cast<float *>(dst + (q + 3) * kTileStride) = v.w;
    }
  }
  for (; q < a.F; ++q) *reinterpret_cast<float *>(dst + q * kTileStride) = src[q];
}

// Walk `ntr` trees (a multiple of G) of the chunk at `cb`, folding their
// leaves into m in tree order.
template <int D, int G>
__device__ __forceinline__ float walk_chunk(const char *cb, int ntr, const char *tile_lane,
                                            float m) {
  constexpr uint32_t NI = (1u << D) - 1u;
  constexpr uint32_t RB = record_bytes(D);
  for (int t0 = 0; t0 < ntr; t0 += G) {
    const char *rec = cb + (uint32_t)t0 * RB;
    uint32_t u[G];
#pragma unroll
    for (int g = 0; g < G; ++g) u[g] = 0;
#pragma unroll
    for (int l = 0; l < D; ++l) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint2 nd = *reinterpret_cast<const uint2 *>(rec + g * RB + u[g] * 8u);
        const float x = *reinterpret_cast<const float *>(tile_lane + nd.x * (uint32_t)kTileStride);
        u[g] = 2u * u[g] + ((x < __uint_as_float(nd.y)) ? 1u : 2u);
      }
    }
    float leaf[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
      leaf[g] = *reinterpret_cast<const float *>(rec + g * RB + 4u * NI + 4u * u[g]);
#pragma unroll
    for (int g = 0; g < G; ++g) m = m + leaf[g];
  }
  return m;
}

// All chunks of the ensemble for the candidates whose features are in the
// tiles.  On entry chunk 0 has been issued into buf0 and the tiles written;
// on exit every wave has passed the final barrier.
template <int D, int G>
__device__ __forceinline__ float walk_all(const WalkArgs &a, char *buf0, char *buf1,
                                          uint32_t chunk_bytes, const char *tile_lane,
                                          int wave, int nwaves, int lane) {
  constexpr uint32_t RB = record_bytes(D);
  wait_all_and_barrier();
  float m = a.base;
  for (int c = 0; c < a.nchunks; ++c) {
    const bool more = c + 1 < a.nchunks;
    const int nt = more ? min(a.chunk_trees, a.ntrees - (c + 1) * a.chunk_trees) : 0;
    if (more && a.nbuf == 2)
      stage_async(a.trees + (size_t)(c + 1) * chunk_bytes, (c & 1) ? buf0 : buf1,
                  (uint32_t)nt * RB, wave, nwaves, lane);
    const int ntr = min(a.chunk_trees, a.ntrees - c * a.chunk_trees);
    m = walk_chunk<D, G>((c & 1) ? buf1 : buf0, ntr, tile_lane, m);
    wait_all_and_barrier();
    if (more && a.nbuf == 1) {  // buf1 aliases buf0: refill after everyone is done
      stage_async(a.trees + (size_t)(c + 1) * chunk_bytes, buf0, (uint32_t)nt * RB, wave,
                  nwaves, lane);
      wait_all_and_barrier();
    }
  }
  return m;
}

template <int D, int G>
__global__ void __launch_bounds__(kLanes *kMaxWaves) validity_kernel(WalkArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr uint32_t RB = record_bytes(D);
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int W = blockDim.x / kLanes;
  const size_t tile_bytes = (size_t)a.F * kTileStride;
  const uint32_t chunk_bytes = (uint32_t)a.chunk_trees * RB;
  char *buf0 = smem + W * tile_bytes;
  char *buf1 = buf0 + (a.nbuf == 2 ? chunk_bytes : 0u);
  char *tile_lane = smem + wave * tile_bytes + 4 * lane;
  const int64_t ntiles = (a.n + kLanes - 1) / kLanes;
  for (int64_t tg = blockIdx.x; tg * W < ntiles; tg += gridDim.x) {
    const int64_t row = (tg * W + wave) * kLanes + lane;
    const bool active = row < a.n;
    stage_async(a.trees, buf0, (uint32_t)min(a.chunk_trees, a.ntrees) * RB, wave, W, lane);
    if (active) load_row(a, row, tile_lane);
    const float m = walk_all<D, G>(a, buf0, buf1, chunk_bytes, tile_lane, wave, W, lane);
    if (active) {
      a.valid_out[row] = (m > 0.0f) ? 1 : 0;
      if (a.margin_out) a.margin_out[row] = m;
    }
  }
}

template <int D, int G>
__global__ void __launch_bounds__(kLanes *kMaxWaves) perf_kernel(WalkArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int wave_count[kMaxWaves];
  constexpr uint32_t RB = record_bytes(D);
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  const int B = blockDim.x;
  const int W = B / kLanes;
  const size_t tile_bytes = (size_t)a.F * kTileStride;
  const uint32_t chunk_bytes = (uint32_t)a.chunk_trees * RB;
  char *buf0 = smem + W * tile_bytes;
  char *buf1 = buf0 + (a.nbuf == 2 ? chunk_bytes : 0u);
  int32_t *queue = reinterpret_cast<int32_t *>(buf1 + chunk_bytes);  // 2*B entries
  char *tile_lane = smem + wave * tile_bytes + 4 * lane;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t nsteps = (a.n + B - 1) / B;
  int64_t step = blockIdx.x;
  int qn = 0;  // identical in every thread
  for (;;) {
    // Scan the mask B entries at a time until a full tile set is queued.
    while (qn < B && step < nsteps) {
      const int64_t i = step * B + threadIdx.x;
      const bool in = i < a.n;
      const bool v = in && (a.valid_in == nullptr || a.valid_in[i] != 0);
      if (in && !v) a.score_out[i] = -INFINITY;
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
    if (qn == 0) break;
    const int take = min(qn, B);
    const int slot = threadIdx.x;
    const int32_t row = (slot < take) ? queue[slot] : -1;
    stage_async(a.trees, buf0, (uint32_t)min(a.chunk_trees, a.ntrees) * RB, wave, W, lane);
    if (row >= 0) load_row(a, row, tile_lane);
    const float m = walk_all<D, G>(a, buf0, buf1, chunk_bytes, tile_lane, wave, W, lane);
    if (row >= 0) a.score_out[row] = m;
    const int rem = qn - take;
    const int32_t carry = (threadIdx.x < rem) ? queue[take + threadIdx.x] : 0;
    __syncthreads();
    if (threadIdx.x < rem) queue[threadIdx.x] = carry;
    qn = rem;
    __syncthreads();
  }
}

constexpr int group_for_depth(int d) { return d <= 6 ? 8 : d <= 9 ? 4 : d <= 10 ? 2 : 1; }

template <int D>
hipError_t launch_depth(bool perf, const WalkPlan &p, const WalkArgs &a, hipStream_t s) {
  constexpr int G = group_for_depth(D);
  if (p.group != G) return hipErrorInvalidValue;
  const void *fn = perf ? reinterpret_cast<const void *>(&perf_kernel<D, G>)
                        : reinterpret_cast<const void *>(&validity_kernel<D, G>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)p.lds_bytes);
  if (e != hipSuccess) return e;
  dim3 grid(p.grid), block(p.waves * kLanes);
  if (perf)
    hipLaunchKernelGGL((perf_kernel<D, G>), grid, block, p.lds_bytes, s, a);
  else
    hipLaunchKernelGGL((validity_kernel<D, G>), grid, block, p.lds_bytes, s, a);
  return hipGetLastError();
}

hipError_t launch_walk(bool perf, const Forest &f, const WalkPlan &p, const WalkArgs &a,
                       hipStream_t s) {
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

WalkArgs make_args(const Forest &f, const WalkPlan &p, const float *X, int64_t n, int64_t ld) {
  WalkArgs a{};
  a.X = X;
  a.n = n;
  a.ld = ld;
  a.trees = static_cast<const char *>(f.d_trees);
  a.ntrees = f.num_trees_padded;
  a.chunk_trees = p.chunk_trees;
  a.nchunks = (f.num_trees_padded + p.chunk_trees - 1) / p.chunk_trees;
  a.F = f.num_features;
  a.vec4 = ((reinterpret_cast<uintptr_t>(X) & 15u) == 0 && (ld & 3) == 0) ? 1 : 0;
  a.base = f.base;
  a.nbuf = p.nbuf;
  return a;
}

}  // namespace

bool plan_walk(const Forest &f, int64_t n_work, int cu_count, WalkPlan *p, const char **why) {
  const int G = group_for_depth(f.depth);
  const size_t rb = f.rec_bytes;
  int per = (int)(16384 / ((size_t)G * rb));
  if (per < 1) per = 1;
  int chunk_trees = G * per;
  if (chunk_trees > f.num_trees_padded) chunk_trees = f.num_trees_padded;  // multiple of G
  const size_t chunk_bytes = (size_t)chunk_trees * rb;
  const size_t tile = (size_t)f.num_features * kTileStride;
  const size_t per_wave = tile + 2 * kLanes * sizeof(int32_t);  // tile + queue share
  int nbuf = 2;
  if (2 * chunk_bytes + per_wave > kLdsBudget) nbuf = 1;
  if (nbuf * chunk_bytes + per_wave > kLdsBudget) {
    *why = "ensemble depth and feature count exceed the LDS of one workgroup";
    return false;
  }
  int W = (int)((kLdsBudget - nbuf * chunk_bytes) / per_wave);
  if (W > 4) W = 4;
  const size_t lds = (size_t)W * per_wave + nbuf * chunk_bytes;
  int per_cu = (int)(kLdsBudget / lds);
  if (per_cu < 1) per_cu = 1;
  if (per_cu > 8) per_cu = 8;
  const int64_t tiles = (n_work + kLanes - 1) / kLanes;
  int64_t groups = (tiles + W - 1) / W;
  int64_t grid = (int64_t)cu_count * per_cu;
  if (groups < grid) grid = groups;
  if (grid < 1) grid = 1;
  p->waves = W;
  p->group = G;
  p->chunk_trees = chunk_trees;
  p->lds_bytes = lds;
  p->nbuf = nbuf;
  p->grid = (int)grid;
  return true;
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

}  // namespace ml2
