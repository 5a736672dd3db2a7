/*
 * ml2_probe.h -- microbenchmarks behind the tree walks' roofline figures, and
 * the tuning overrides of the walks' launch plan and the ensembles' layout.
 *
 * Measurement and tuning helpers, not part of scoring: for the benchmark's
 * report of what the units a walk uses deliver on the current device, and
 * for sweeps and tests that force every launch shape the planner can choose.
 * The walk's unit of work is a node visit (a node read, a feature read, a
 * compare and a child step); the probe calls time the LDS reads, 32-bit adds
 * and the walk's inner loop in isolation.
 *
 * Each probe call runs on the HIP device current on the calling thread,
 * allocates its own output buffer, launches once untimed and once timed on
 * the null stream, synchronises, frees the buffer and returns.  ms and the
 * work output are HOST pointers.  Status codes as in ml2.h: INVALID_ARG for
 * an argument outside the stated range or a NULL output, OUT_OF_MEMORY, HIP.
 */
#ifndef ML2_PROBE_H
#define ML2_PROBE_H

#include <stdint.h>

#include "ml2.h"

#ifdef __cplusplus
extern "C" {
#endif

/* The walk's inner loop over a resident chunk: blocks workgroups of `waves`
 * waves, `lanes_per_candidate` lanes per candidate, `features` random
 * features per candidate, and a chunk of random perfect trees of depth
 * `depth` with `trees_per_lane` trees per lane, walked iters times (the
 * scoring walk's code without row loads or restaging).  *visits: node
 * visits made (candidates x trees x depth).  Built shapes: depth 6, 8 or
 * 10; trees_per_lane 1, 2, 4 or 8; lanes_per_candidate 1 or 2; waves 1 to
 * 8; features 64 or 128; the tiles and the chunk within one workgroup's
 * LDS.  1 <= iters <= 2^20; 1 <= blocks <= 65536.  The 16M
 * pool's walks: (6, 8, 2, 8, 128) and (8, 4, 2, 8, 128). */
ml2_status ml2_probe_visit(int32_t depth, int32_t trees_per_lane, int32_t lanes_per_candidate,
                           int32_t waves, int32_t features, int32_t iters, int32_t blocks,
                           double *ms, double *visits);

/* LDS reads: 256-thread workgroups, eight reads per lane and iteration of a
 * 64 KiB buffer.  mode 0, 1, 2: 4-, 8-, 16-byte reads at consecutive
 * addresses across the lanes; mode 3, 4, 5: the same widths at random
 * (hashed) addresses.  *bytes: bytes read.  1 <= iters <= 2^20;
 * 1 <= blocks <= 65536. */
ml2_status ml2_probe_lds(int32_t mode, int32_t iters, int32_t blocks, double *ms, double *bytes);

/* 32-bit integer adds: 256-thread workgroups, eight independent chains of
 * 16 adds per lane and iteration.  *lane_ops: lane additions made.
 * 1 <= iters <= 2^20; 1 <= blocks <= 65536. */
ml2_status ml2_probe_valu(int32_t iters, int32_t blocks, double *ms, double *lane_ops);

/* Launch-plan override of the walks (tuning sweeps, tests of every launch
 * shape).  Process-wide and sticky: every later ml2_score_validity,
 * ml2_score_perf and ml2_explorer_round call, on any thread, takes the
 * nonzero fields in place of the planner's choice where the forced shape
 * fits the ensemble and the LDS (a field that does not fit is ignored, as
 * is a zero field).  All zeros restore the planner.  The results of every
 * call are unchanged (bit for bit): only the launch shape differs.
 *   split: lanes per candidate (1 or 2)      group: trees per lane (1..16)
 *   waves: waves per workgroup (1..8)        nbuf: LDS chunk buffers (1 or 2)
 *   chunk: trees per staged chunk (a multiple of the group's trees)
 * Errors: INVALID_ARG for a negative field or one above those ranges. */
ml2_status ml2_tune_walk_plan(int32_t split, int32_t group, int32_t waves, int32_t nbuf,
                              int32_t chunk);

/* Layout override of later ml2_load_ensemble calls (process-wide, sticky):
 * 0 the loader's choice, 1 perfect padded trees and 2 ragged chunk slots,
 * each where it can represent the ensemble (else the loader's choice).
 * Errors: INVALID_ARG outside 0..2. */
ml2_status ml2_tune_layout(int32_t layout);

#ifdef __cplusplus
}
#endif

#endif /* ML2_PROBE_H */
