/*
 * gemv_ar.h -- fused GEMV + AllReduce for AMD Instinct MI355X (gfx950).
 *
 * The scale-up operator of Sec. III-B of "Optimizing Distributed ML
 * Communication with Fused Computation-Collective Operations": R ranks hold
 * column blocks of a matrix (rank r: A_r, M x K_r) and the matching parts of
 * a vector (x_r, K_r elements), as in a tensor-parallel layer.  Each rank's
 * partial product A_r x_r is reduced across ranks with a two-phase direct
 * AllReduce (reduce-scatter, then all-gather) fused into the GEMV kernel:
 *
 *  - the M outputs are cut into tiles of tile_rows rows; tile i is owned by
 *    rank floor(i * R / n_tiles) (contiguous blocks of tiles);
 *  - P physical workgroups per rank; workgroup p of every rank computes the
 *    same tiles, i = p, p + P, p + 2P, ... (Sec. III-B);
 *  - a workgroup computes the tiles owned by other ranks first (remote tiles
 *    ahead of local ones, the communication-aware order of Sec. III-B),
 *    stores each partial tile straight into the owner's reduction slots
 *    (zero-copy stores) and, once all its tiles for one owner are stored,
 *    sets one ready flag for that owner;
 *  - the owner's workgroup p then waits for the flags of workgroup p of every
 *    other rank, sums the R partials of its tiles in rank order and stores the
 *    result into every rank's output vector (all-gather), then adds 1 to its
 *    output flag (reduce_mode 1).
 *
 * On one GPU the R ranks are logical and "peer memory" is a slot of a
 * plan-owned buffer.  reduce_mode 1 runs all ranks in one cooperative launch
 * (every workgroup resident at once, so the owners' waits always end).  The
 * default reduce_mode 0 replaces the waiting owner by an arrival counter per
 * (owner, workgroup): whichever rank's workgroup delivers last reduces and
 * broadcasts, so nothing waits and the kernel launches normally.
 *
 * Conventions: A[r] is row-major M x K[r] in the plan's storage type, row r
 * starting at byte i * K[r] * elt, 16-byte aligned, K[r] * elt a multiple of
 * 16; x[r] holds K[r] elements of the same type; y[r] is fp32 [M].  All
 * pointers are device pointers owned by the caller, passed as host arrays of
 * R pointers.  out_flags (optional) is uint32 [R * P]: flag r * P + p is
 * incremented (release at device scope) once workgroup p of owner r has
 * stored its reduced tiles into every rank's output; the caller zeroes it
 * once, and after n forwards every flag equals n.  Accumulation is fp32; the
 * reduction sums ranks in order 0 .. R-1, so fused and unfused results are
 * bitwise equal.
 *
 * Errors follow ebag_a2a.h (EBAG_OK / negative codes, checked before
 * anything is enqueued; ebag_a2a_last_error() holds the message).
 */
#ifndef GEMV_AR_H
#define GEMV_AR_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "ebag_a2a.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gemv_ar_plan* gemv_ar_t;

typedef struct gemv_ar_opts {
  int32_t tile_rows;           /* rows per output tile, 1..4096; 0 (default): 128, halved down to 64 while
                                  the R ranks have fewer than 2048 tiles in all */
  int32_t wgs_per_rank;        /* physical workgroups per rank P, at most the number of tiles; 0 (default):
                                  ceil(1024 / R), i.e. about 1024 workgroups in all, each taking one or more
                                  tiles (reduce_mode 0), or as many as can be resident at once for the
                                  whole grid (reduce_mode 1) */
  int32_t waves_per_wg;        /* wavefronts per workgroup, 1..16 (default 2) */
  int32_t comm_aware;          /* 1 (default): tiles owned by other ranks first; 0: tile order */
  int32_t debug_suppress_flag; /* >= 0: never set this peer flag ((owner * R + rank) * P + p), for
                                  failure-path tests; -1 (default) off */
  int32_t reduce_mode;         /* 0 (default): the last of the R ranks' workgroups p to store its partials
                                  for an owner reduces that owner's tiles (arrival counter, no waiting,
                                  normal launch; can be captured
                                  into a graph and replayed); 1: the owner's workgroup waits for the
                                  peer flags and reduces (the paper's scheme; cooperative launch, every
                                  workgroup resident; the flags carry a per-call epoch, so a forward on
                                  a stream under graph capture returns EBAG_EUNSUPPORTED) */
  int64_t timeout_us;          /* reduce_mode 1: an owner gives up waiting after this long (default 5 s) */
} gemv_ar_opts_t;

/* Fill *opts with the defaults listed above. */
int gemv_ar_default_opts(gemv_ar_opts_t* opts);

/*
 * Create a plan on the current HIP device for R ranks (1..16), M outputs and
 * K[r] columns per rank (host array of R values, each > 0 with K[r] * elt a
 * multiple of 16, K[r] * elt at most 64 KiB), storage type dtype (EBAG_F32,
 * EBAG_F16 or EBAG_BF16; anything else is EBAG_EINVAL).  The plan
 * owns the reduction slots (R * M floats), the peer flags, the arrival
 * counters and a status word.  One forward may be in flight per plan:
 * forwards on one stream are ordered, and a forward (fused or not) enqueued
 * on another stream while the plan's last forward has not completed returns
 * EBAG_EBUSY and enqueues nothing.  The check is an event recorded after each
 * forward and queried on the host, so it also refuses a second stream that
 * waits for the first; it is skipped under graph capture.  The forwards must
 * be called with the plan's device current (EBAG_EINVAL otherwise).
 */
int gemv_ar_create(gemv_ar_t* out, int32_t R, int64_t M, const int64_t* K, int32_t dtype,
                   const gemv_ar_opts_t* opts);

/* Fused forward: one launch (cooperative with reduce_mode 1) computing
 * y[r] = sum_s A_s x_s for every rank r.  A, x, y: host arrays of R device
 * pointers.  out_flags: NULL or device uint32 [R * P] (P from
 * gemv_ar_launch_info). */
int gemv_ar_forward(gemv_ar_t h, const void* const* A, const void* const* x, float* const* y,
                    uint32_t* out_flags, hipStream_t stream);

/* Bulk-synchronous baseline with the same contract and result: a GEMV
 * kernel writes every rank's partial vector, then an AllReduce kernel sums
 * them (rank order) into every rank's output, then the output flags are
 * incremented -- GEMV and collective at kernel boundaries (Sec. III-B,
 * Sec. IV-B). */
int gemv_ar_unfused_forward(gemv_ar_t h, const void* const* A, const void* const* x, float* const* y,
                            uint32_t* out_flags, hipStream_t stream);

/* Synchronise the plan's device and read the status: out[0] 1 if an owner
 * timed out, out[1] the lowest peer flag index it gave up on (-1 none).
 * Returns EBAG_OK or EBAG_ETIMEOUT.  This call and gemv_ar_reset make the
 * plan's device current for their duration and then restore the caller's. */
int gemv_ar_status(gemv_ar_t h, int32_t out[2]);

/* Clear the status word (after a timeout).  Synchronous. */
int gemv_ar_reset(gemv_ar_t h);

/* Launch shape: out[0] P (workgroups per rank), out[1] threads per
 * workgroup, out[2] number of tiles, out[3] workgroups the device can hold
 * resident at once for this kernel, out[4] rows per tile. */
int gemv_ar_launch_info(gemv_ar_t h, int32_t out[5]);

/* Release the plan's device memory.  NULL is ignored. */
void gemv_ar_destroy(gemv_ar_t h);

#ifdef __cplusplus
}
#endif

#endif /* GEMV_AR_H */
