// Internal declarations shared by the host entry points and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "layout.h"
#include "ml2.h"

namespace ml2 {

constexpr size_t kLdsBudget = 160 * 1024 - 256;  // LDS of a walk workgroup (static LDS headroom)
constexpr size_t kTreeSlack = 128 * 1024;  // readable zero bytes after the tree table

// hipFuncSetAttribute(MaxDynamicSharedMemorySize) for kernel fn on the current
// device, called only when `bytes` exceeds what was set there before (the
// launchers call it before every launch; the attribute call itself then runs
// once per kernel, device and size increase).
hipError_t ensure_dynamic_lds(const void *fn, size_t bytes);

struct Forest {
  int device;
  int32_t num_trees;        // trees in the descriptor
  int32_t num_trees_padded; // with the padding trees (perfect: a multiple of kTreePad)
  int32_t num_features;
  int32_t depth;            // deepest path (perfect: the padded depth, >= 1)
  int32_t ragged;           // 1: ragged layout
  int32_t records;          // staged records: perfect trees, or ragged chunk slots
  float base;
  uint32_t rec_bytes;       // record_bytes(depth), or record_bytes(0) when ragged
  void *d_trees;            // records * rec_bytes bytes (+ kTreeSlack zero bytes)
};

// Launch parameters of a walk (chosen on the host from D and F).
struct WalkPlan {
  int split;        // lanes per candidate: 1, or 2 (the two half-waves walk
                    // alternate halves of every tree group)
  int waves;        // waves per workgroup; each wave owns 64 / split candidates
  int group;        // trees walked concurrently per lane (ILP)
  int chunk_trees;  // trees per LDS chunk (multiple of group)
  int nbuf;         // LDS chunk buffers: 2 (asynchronous refill) or 1
  size_t lds_bytes; // dynamic LDS per workgroup
  int grid;         // workgroups
};

// Returns false (and sets *why) if no plan fits the LDS of one workgroup.
// survivors: the walk covers the rows a mask accepts out of n_work.
bool plan_walk(const Forest &f, int64_t n_work, int cu_count, WalkPlan *plan, const char **why,
               bool survivors = false);

// Validity and performance in one pass over the pool (fused_kernel): false
// where the two ensembles or the pool do not allow it.  nv, np: records of V
// and P walked.
constexpr int kMaxFusedDepth = 8;
bool plan_fused(const Forest &v, const Forest &p, int64_t n, int64_t ld, const float *X,
                int cu_count, WalkPlan *plan, int *nv, int *np);
hipError_t launch_fused(const Forest &v, const Forest &p, const WalkPlan &pl, int nv, int np,
                        const float *X, int64_t n, int64_t ld, uint8_t *valid_out,
                        float *margin_out, float *score_out, hipStream_t s);

// Tuning overrides (ml2_tune_walk_plan / ml2_tune_layout): process-wide,
// zero = the planner's or loader's choice.
enum TuneField { kTuneSplit, kTuneGroup, kTuneWaves, kTuneNbuf, kTuneChunk, kTuneLayout,
                 kTuneFields };
void set_tune(int field, int value);
int get_tune(int field);

hipError_t launch_validity(const Forest &f, const WalkPlan &p, const float *X, int64_t n,
                           int64_t ld, uint8_t *valid_out, float *margin_out, hipStream_t s);
hipError_t launch_perf(const Forest &f, const WalkPlan &p, const float *X, int64_t n,
                       int64_t ld, const uint8_t *valid, float *score_out, hipStream_t s);

// Walk of a list of pool rows: score_out[i] = margin of row rows[i], or -inf
// where rows[i] lies outside [0, n).  ws: rows_workspace_bytes(f, m) bytes
// of device memory (the per-tree leaves).
size_t rows_workspace_bytes(const Forest &f, int32_t m);
hipError_t launch_rows(const Forest &f, const float *X, int64_t n, int64_t ld, const int32_t *rows,
                       int32_t m, float *score_out, void *ws, int cu_count, hipStream_t s);

size_t topk_workspace_bytes(int64_t n, int32_t k);
// Device address of the selection's static scratch on `device` (which must
// be current), looked up once per device; its size covers any k up to
// ML2_MAX_TOPK.
size_t static_scratch_bytes();
hipError_t static_scratch(int device, void **ptr);
hipError_t launch_topk(const uint8_t *valid, const float *scores, int64_t n, int32_t k,
                       int32_t *idx, float *score, int32_t *num, void *ws, int cu_count,
                       hipStream_t s);

// mask[rows[j]] = 0 for the listed rows inside [0, n).
hipError_t launch_exclude(uint8_t *mask, int64_t n, const int32_t *rows, int32_t m,
                          hipStream_t s);

// Streamed explorer: proposed rows leave a chunk's mask (rows row0 ..
// row0+m-1); the held count is reset; the held set absorbs a chunk's
// selection (k best by (P desc, row asc), each row once; merge_held_lds(k)
// bytes of LDS, k <= 4096).
hipError_t launch_exclude_range(uint8_t *mask, int64_t row0, int64_t m, const int32_t *rows,
                                int32_t count, hipStream_t s);
hipError_t launch_held_reset(int32_t *held_id, float *held_p, float *held_a, int32_t *held_n,
                             int32_t k, hipStream_t s);
size_t merge_held_lds(int32_t k);
hipError_t launch_merge_held(const int32_t *h_id, const float *h_p, const float *h_a,
                             const int32_t *h_n, const int32_t *c_idx, const float *c_p,
                             const float *c_a, const int32_t *c_n, int64_t row0, int32_t k,
                             int32_t *o_id, float *o_p, float *o_a, int32_t *o_n, hipStream_t s);

// The `keep` best of m listed rows by (score desc, pool row asc); m <= ML2_MAX_TOPK.
hipError_t launch_rerank_select(const int32_t *rows, const float *scores, int32_t m, int64_t n,
                                int32_t keep, int32_t *idx, float *score, int32_t *num,
                                hipStream_t s);

// Microbenchmarks (measurement helpers behind the roofline figures).
// Visit probe: the walk of a resident chunk of random perfect trees of depth
// 6 or 8 over random feature tiles, iters times per lane, at the shape
// (trees per lane G, lanes per candidate S, waves, features); *visits: the
// node visits the launch makes.  hipErrorInvalidValue for a shape it does
// not build or whose tiles and chunk exceed the LDS.
hipError_t launch_visit_probe(int depth, int G, int S, int waves, int features, int iters,
                              int blocks, float *out, double *visits, hipStream_t s);
// LDS read probe (mode: 0..2 consecutive 4-, 8-, 16-byte reads per lane,
// 3..5 the same at random addresses) and a 32-bit integer add probe; *work:
// the bytes read or the lane operations of the launch.
hipError_t launch_lds_probe(int mode, int iters, int blocks, uint32_t *out, double *work,
                            hipStream_t s);
hipError_t launch_valu_probe(int iters, int blocks, uint32_t *out, double *work, hipStream_t s);

}  // namespace ml2
