/*
 * ml2_probe.h -- microbenchmarks behind the tree walks' roofline figures.
 *
 * Measurement helpers, not part of scoring: for the benchmark's report of
 * what the units a walk uses deliver on the current device.  The walk's unit
 * of work is a node visit (a node read, a feature read, a compare and a child
 * step); these calls time the LDS reads, 32-bit adds and the walk's inner
 * loop in isolation.
 *
 * Each call runs on the HIP device current on the calling thread, allocates
 * its own output buffer, launches once untimed and once timed on the null
 * stream, synchronises, frees the buffer and returns.  ms and the work
 * output are HOST pointers.  Status codes as in ml2.h: INVALID_ARG for an
 * argument outside the stated range or a NULL output, OUT_OF_MEMORY, HIP.
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
 * visits made (candidates x trees x depth).  Built shapes: depth 6 or 8;
 * (trees_per_lane, lanes_per_candidate) (2, 2), (4, 2), (8, 2), (4, 1) or
 * (8, 1); waves 4 or 8; features 64 or 128; the tiles and the chunk within
 * one workgroup's LDS.  1 <= iters <= 2^20; 1 <= blocks <= 65536.  The 16M
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

#ifdef __cplusplus
}
#endif

#endif /* ML2_PROBE_H */
