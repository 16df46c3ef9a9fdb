/*
 * ebag_a2a.h -- fused embedding-bag pooling + All-to-All send layout for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (Sec. III-A of "Optimizing Distributed ML Communication with
 * Fused Computation-Collective Operations"): every pooled embedding vector is
 * produced by one logical workgroup of an EmbeddingBag kernel and stored
 * directly where the All-to-All must deliver it, i.e. in a destination-
 * partitioned send buffer of shape [R][B/R][sum_t D_t], and each slice is
 * announced with a ready flag as soon as its last contributor finishes, so a
 * consumer can move finished slices while pooling is still running.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  T tables; table t has rows_t rows of D_t elements of the plan's storage
 *  type, dense and row-major (row r starts at byte r * D_t * elt), 16-byte
 *  aligned.  D_t * elt must be a multiple of 16 bytes.
 *
 *  Bags are table-major CSR: bag (t, b) for sample b in [0, B) is
 *  indices[offsets[t*B + b] .. offsets[t*B + b + 1]); offsets has T*B + 1
 *  int64 entries, offsets[0] == 0, non-decreasing; indices are int32 in
 *  [0, rows_t).  An empty bag pools to a zero vector; repeated indices count
 *  with multiplicity.  weights (optional) are fp32, one per index: the bag
 *  value is sum_k w_k * row_k (plain sum when weights == NULL).  A plan
 *  created with pooling_mode = 1 pools the mean instead: the sum divided by
 *  the bag length (weights must then be NULL).
 *
 *  Destinations: the batch is split into R contiguous parts of S = B / R
 *  samples, the first to destination 0 (Sec. III-A, worked example).  Pooled
 *  vector (t, b) is written as fp32 to send_buf[r][s][off_t + j] with
 *  r = b / S, s = b % S, off_t = sum of D over tables before t -- the
 *  {local batch, numTables x D} shape handed to the next operator.  The
 *  memory order is identical to a [B][sum D] array.
 *
 *  Slices ("chunks"): slice (r, c) is the C samples r*S + c*C ..
 *  r*S + (c+1)*C - 1 of destination r for all T tables -- a contiguous block
 *  of C * sum(D) floats.  flags has R * (S / C) uint32 entries, slice (r, c)
 *  at r * (S / C) + c (equivalently the global slice g = b / C).  With
 *  slice_granule = 1 each slice is split per table: flag (g, t) covers the C
 *  pooled vectors of table t in slice g (columns off_t .. off_t + D_t of C
 *  consecutive rows), flags has T * (B / C) entries and (g, t) is at
 *  g * T + t.  "Flag index" below means this index.
 *
 *  Flags are epochs: the caller zeroes the flag array once; every completed
 *  forward adds exactly 1 to every flag of the batch with release semantics
 *  at device (agent) scope, after all of that slice's data is stored.  After
 *  n forwards every flag equals n.
 *
 *  Pointers named *_buf, tables, indices, offsets, weights and flags are
 *  device pointers owned by the caller; the library never frees them.
 *  indices must be non-null even when every bag is empty (nnz = 0): the
 *  library cannot read nnz on the host, and never reads past offsets.  All
 *  device work is enqueued on the given HIP stream; calls return as soon as
 *  the work is enqueued.  One forward (fused or unfused) may be in flight per
 *  plan at a time: the plan's slice counters and unfused scratch are shared.
 *  Forwards on one stream are ordered; a forward enqueued on another stream
 *  while the plan's last forward has not completed returns EBAG_EBUSY and
 *  enqueues nothing (checked on the host with an event, so also when that
 *  stream waits for the other one; not checked under graph capture).  Order a
 *  plan's forwards on one stream, or let the last one complete first.  The
 *  same holds, and is checked the same way, for the backward (the plan's
 *  table bases are shared) and for the delivery (its per-slice piece
 *  counters are shared): one of each may be in flight per plan, while a
 *  backward and a delivery are independent of each other.  Changed
 *  table pointers are uploaded by small kernels on the forward's stream: the
 *  call never waits for the device.
 *
 * Errors: every entry point returns EBAG_OK (0) or a negative code, checked
 * before anything is enqueued; ebag_a2a_last_error() returns a message for
 * the calling thread's most recent failure.  Preconditions that are not
 * checked on the host (index range, offset monotonicity) are checked in the
 * kernels when the plan was created with check_indices = 1: rows with an
 * out-of-range index are skipped, a bag whose offsets are invalid is pooled
 * as zeros, and the first such bag is reported by ebag_a2a_status_ex().
 */
#ifndef EBAG_A2A_H
#define EBAG_A2A_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ebag_a2a_plan* ebag_a2a_t;

/* Table storage types.  Entry points take them as int32_t, so that any
 * other value is an argument error (EBAG_EINVAL), never undefined behaviour. */
typedef enum { EBAG_F32 = 0, EBAG_F16 = 1, EBAG_BF16 = 2 } ebag_dtype_t;

enum {
  EBAG_OK = 0,
  EBAG_EINVAL = -1,       /* bad argument (null pointer, size, split, alignment) */
  EBAG_EUNSUPPORTED = -2, /* valid, but outside what the library supports */
  EBAG_EHIP = -3,         /* a HIP runtime call failed */
  EBAG_ETIMEOUT = -4,     /* reported by ebag_a2a_status() */
  EBAG_ENOMEM = -5,       /* device or host allocation failed */
  EBAG_EBUSY = -6         /* a forward was enqueued on another stream while this plan's last one still runs */
};

/* Tuning and debugging knobs; pass NULL to ebag_a2a_create for defaults, or
 * fill with ebag_a2a_default_opts() and change fields. */
typedef struct ebag_a2a_opts {
  int32_t waves_per_wg;        /* wavefronts (64 lanes) per pooling workgroup, 1..16 (default 4) */
  int32_t bags_per_run;        /* bags a workgroup pools before one slice-counter update (default 16;
                                  capped so that the run's pooled rows, bags x max D floats, fit a 16 KiB
                                  LDS tile, and at chunk_samples) */
  int32_t rows_in_flight;      /* 16-byte row loads each wave keeps in flight: 4, 8 or 16 (default 8) */
  int32_t persistent_wgs_per_cu; /* 0: one workgroup per run; >0: persistent grid of that many WGs per CU
                                    (-1: as many as fit), whose workgroups claim runs in production order
                                    from an atomic ticket (Sec. III-A task loop) */
  int32_t release_mode;        /* slice release: 1 (default) device-scope stores + completion wait, 0 agent-scope release fence per run */
  int32_t chunk_order;         /* 0: natural slice order; 1: slices of destination self_rank last */
  int32_t self_rank;           /* the destination whose slices stay local (chunk_order == 1) */
  int32_t trace;               /* 1: record a device timestamp at every slice release and drain */
  int32_t check_indices;       /* 1: kernels check offsets/indices, skip and report bad bags */
  int32_t debug_suppress_flag; /* >= 0: never publish the flag with this index (failure-path tests); -1 off */
  int32_t consumer_wgs;        /* single-wave workgroups of the consumer kernel (default 512) */
  int32_t stream_rows;         /* 1 (default): table rows are read with non-temporal loads (no reuse expected);
                                  0: cached loads (skewed index distributions with hot rows) */
  int64_t consume_timeout_us;  /* the consumer, and the backward waiting on gradient flags, give up after
                                  this long and report it through ebag_a2a_status (default 5,000,000 us) */
  int32_t pooling_mode;        /* 0 (default): sum (weighted sum when weights are given); 1: mean -- the
                                  bag's sum divided by its length L, zeros for an empty bag; takes no weights
                                  (the sum / mean modes of the original pooling kernel, Sec. III-A) */
  int32_t slice_granule;       /* 0 (default): a flag per (destination, C samples) for all T tables;
                                  1: a flag per (destination, C samples, table) -- the paper's per-table
                                  slice (Sec. III-A); see "Slices" above */
  int32_t backward_bags_per_run;  /* ebag_a2a_backward: bags per workgroup (default 4; capped so that the
                                     bags' gradient rows fit in 64 KiB of LDS) */
  int32_t backward_waves_per_wg;  /* ebag_a2a_backward: wavefronts per workgroup, 1..16 (default 16) */
  int32_t table_major;         /* 0 (default): runs slice by slice, tables fastest inside a slice; 1: table
                                  by table, slices in order inside each table, and (when T is a multiple
                                  of the XCD count) each XCD working through its own tables one at a time,
                                  so that a table's hot rows stay in that XCD's caches; 2: table by table
                                  for the whole device, so that one table's rows share the device-wide
                                  cache.  Meant for slice_granule = 1, whose per-table slices then still
                                  complete progressively; with whole slices every slice completes at the
                                  end.  The consumer, backward and delivery follow the same order. */
  int32_t consume_nontemporal; /* 1: the consumer reads and writes slice data non-temporally, so its
                                  stream does not displace the producer's cached table rows (pays off
                                  when rows are reused: Zipf indices, small tables); 0 (default): plain
                                  loads and stores, which may hit the freshly written slices in cache */
  int32_t deliver_wgs;         /* ebag_a2a_deliver: workgroups of the delivery stand-in, a copy that never
                                  waits (default 32) */
  int32_t deliver_waves_per_wg; /* ebag_a2a_deliver: wavefronts per delivery workgroup, 1..16 (default 8);
                                   each keeps eight 16-byte loads in flight per lane, so a few workgroups
                                   feed the backward while holding only a few CUs */
} ebag_a2a_opts_t;

/* Fill *opts with the defaults listed above.  Returns EBAG_OK or EBAG_EINVAL. */
int ebag_a2a_default_opts(ebag_a2a_opts_t* opts);

/*
 * Create a plan for T tables on the current HIP device.  Every later call on
 * the plan must be made with that device current (EBAG_EINVAL otherwise),
 * with buffers and a stream of that device.
 *   rows_per_table[T], dim_per_table[T]: host arrays; rows >= 0 (< 2^31), D > 0,
 *     D * elt % 16 == 0.
 *   table_dtype: storage type shared by all tables (EBAG_F32, EBAG_F16 or
 *     EBAG_BF16; anything else is EBAG_EINVAL); pooled output is fp32.
 *   chunk_samples (C): samples per slice, > 0; one slice (C * sum(D) fp32)
 *     must be below 2 GiB.
 *   max_batch: largest B any forward will use (sizes the slice counters and
 *     the unfused scratch of max_batch * sum(D) floats).
 *   max_ranks: largest R any forward will use.
 * Device memory owned by the plan: slice counters, unfused scratch, table
 * descriptors, status word, trace buffers; released by ebag_a2a_destroy.
 */
int ebag_a2a_create(ebag_a2a_t* out, int32_t num_tables, const int64_t* rows_per_table,
                    const int32_t* dim_per_table, int32_t table_dtype, int32_t chunk_samples,
                    int64_t max_batch, int32_t max_ranks, const ebag_a2a_opts_t* opts);

/*
 * Fused forward (Sec. III-A): pool every bag, store each pooled vector
 * straight into send_buf at its destination slot (zero-copy placement,
 * Sec. III-B / IV-B), and release each slice's flag (+1) when the last of
 * its C*T bags is stored.  Slices complete progressively in slice order.
 *   tables: HOST array of T device pointers (16-byte aligned).
 *   indices, offsets, weights: device arrays as described above.
 *   B > 0, R > 0, B % R == 0, (B / R) % C == 0, B <= max_batch, R <= max_ranks;
 *   weights == NULL when the plan pools means.
 *   send_buf: device fp32 [B * sum(D)], 16-byte aligned.  flags: device
 *   uint32 [B / C] ([T * B / C] with slice_granule = 1).
 */
int ebag_a2a_forward(ebag_a2a_t h, const void* const* tables, const int32_t* indices, const int64_t* offsets,
                     const float* weights, int64_t B, int32_t R, float* send_buf, uint32_t* flags,
                     hipStream_t stream);

/*
 * Fused forward without a plan, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same operation, result and flag contract as
 * ebag_a2a_forward on a plan created with the same tables, chunk_samples and
 * opts; the table shapes (as for ebag_a2a_create) come with every call.
 *
 * The device memory a plan would own -- table descriptors and pointers,
 * slice counters, status word, run ticket -- is instead one statically
 * allocated device array of EBAG_NOALLOC_SCRATCH_BYTES per GPU, which every
 * GPU the library runs on holds until the process ends.  Each call first
 * enqueues a small kernel (one per 64 tables) that writes the descriptors
 * into that array and clears the counters, ticket and status word, then the
 * pooling kernel; it calls no hipMalloc, hipFree or other allocating routine
 * (its host-side descriptors live on the calling thread's stack, about 52 KB).
 *   num_tables: 1 .. EBAG_NOALLOC_MAX_TABLES.
 *   opts: NULL for the defaults; trace = 1 and check_indices = 1 are refused
 *     with EBAG_EUNSUPPORTED (their results are read through a plan);
 *     consumer, backward and delivery options are ignored.
 *   B / chunk_samples flags (times num_tables with slice_granule = 1) must
 *     not exceed EBAG_NOALLOC_MAX_FLAGS (EBAG_EINVAL otherwise).
 *   Other arguments as for ebag_a2a_create and ebag_a2a_forward; every check
 *   is made before anything is enqueued.
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents: two calls that overlap on one GPU (on different streams, or from
 * different host threads without ordering) race on it and corrupt each
 * other's slice counters.  Order them on one stream.  The first call on a
 * device looks up the array's device address (hipGetSymbolAddress) with that
 * device current.
 */
#define EBAG_NOALLOC_MAX_TABLES 1024
#define EBAG_NOALLOC_MAX_FLAGS 65536
#define EBAG_NOALLOC_SCRATCH_BYTES (320 * 1024)
int ebag_a2a_forward_noalloc(int32_t num_tables, const int64_t* rows_per_table, const int32_t* dim_per_table,
                             int32_t table_dtype, int32_t chunk_samples, const ebag_a2a_opts_t* opts,
                             const void* const* tables, const int32_t* indices, const int64_t* offsets,
                             const float* weights, int64_t B, int32_t R, float* send_buf, uint32_t* flags,
                             hipStream_t stream);

/*
 * Bulk-synchronous baseline with the same contract and result: a pooling
 * kernel writes per-table outputs [T][B][D_t] to plan scratch, then a
 * repack kernel copies them into the send layout and releases each slice's
 * flag -- the pool -> repack -> collective sequence at kernel boundaries
 * that the fused operator replaces (Sec. II-B, IV-A).
 */
int ebag_a2a_unfused_forward(ebag_a2a_t h, const void* const* tables, const int32_t* indices,
                             const int64_t* offsets, const float* weights, int64_t B, int32_t R,
                             float* send_buf, uint32_t* flags, hipStream_t stream);

/*
 * Receiver side (Sec. III-A, "Book-keeping Flags"): each slice is split
 * into pieces of up to 32 KiB (with slice_granule = 1: one piece per
 * per-table slice, C rows of D_t floats); each consumer workgroup (one
 * wavefront) owns a distinct subset of pieces, polls the slice's flag until
 * it reaches expected_epoch, then copies the piece from send_buf to recv_buf
 * (same layout and size).  Meant to run on a second
 * stream concurrently with a forward.  Enqueue it after the forward it
 * waits for: streams may share a hardware queue, and a consumer queued ahead
 * of its producer on the same queue can only time out.  Polling is bounded
 * by the plan's consume_timeout_us; on timeout the kernel stops and records
 * the first missing slice for ebag_a2a_status().  expected_epoch is fixed
 * when the call is made, so a graph replay could not wait for its own
 * producer: on a stream under capture the call returns EBAG_EUNSUPPORTED
 * and enqueues nothing.
 */
int ebag_a2a_consume(ebag_a2a_t h, const float* send_buf, const uint32_t* flags, float* recv_buf, int64_t B,
                     int32_t R, uint32_t expected_epoch, hipStream_t stream);

/*
 * Embedding backward fused with the arrival of the gradient All-to-All (the
 * paper overlaps the backward embedding operations with their All-to-All as
 * well, Sec. IV-D).  The table owner receives the gradient of every pooled
 * vector of the batch in the send layout of the forward:
 *   grad_buf: device fp32 [B * sum(D)], pooled vector (t, b) at
 *     grad_buf[b * sum(D) + off_t ..] (the [R][B/R][sum D] order).
 *   grad_flags: NULL -- the gradient is complete (bulk-synchronous: launch
 *     after the collective); or the per-slice epoch flags of the gradient's
 *     arrival (same layout as the forward's flags for this plan's
 *     slice_granule): the runs of a slice start once its flag reaches
 *     expected_epoch (bounded by consume_timeout_us; a timeout is reported
 *     by ebag_a2a_status and leaves that run's rows unwritten).
 *   offsets, weights: the forward's bags (weights NULL for plain or mean
 *     pooling; the plan's pooling_mode applies).
 *   values: device fp32 output, one row per lookup: for each table t, in
 *     lookup order, nnz_t = offsets[(t+1)B] - offsets[tB] rows of D_t floats;
 *     table blocks follow each other in table order.  Lookup k of bag (t, b)
 *     gets w_k * grad (sum; w_k = 1 without weights) or grad / L (mean), each
 *     value rounded once to fp32 -- the values of the sparse gradient of an
 *     EmbeddingBag, whose indices are the forward's indices.
 * Launch shape: backward_bags_per_run bags per workgroup of
 * backward_waves_per_wg wavefronts.  With grad_flags, on a stream under
 * graph capture the call returns EBAG_EUNSUPPORTED (expected_epoch would be
 * fixed for every replay); without flags it can be captured and replayed.
 */
int ebag_a2a_backward(ebag_a2a_t h, const float* grad_buf, const uint32_t* grad_flags, uint32_t expected_epoch,
                      const int64_t* offsets, const float* weights, int64_t B, int32_t R, float* values,
                      hipStream_t stream);

/*
 * One-GPU stand-in for the arrival of an All-to-All: copies every slice of
 * src into dst (same layout, [B * sum(D)] fp32) in slice order and, once a
 * slice is stored (device-scope stores), adds 1 to its flag in flags (the
 * layout of the forward's flags for this plan).  Used to feed
 * ebag_a2a_backward from a second stream: on one GPU it plays the gradient
 * All-to-All whose arrival the backward overlaps (Sec. IV-D), the receiving
 * side of the flags of Sec. III-A.  Grid: the plan's deliver_wgs
 * workgroups of deliver_waves_per_wg wavefronts.  Errors: EBAG_EINVAL for a null plan, buffer
 * or flags, misaligned buffers or a bad B / R split, checked before anything
 * is enqueued.
 */
int ebag_a2a_deliver(ebag_a2a_t h, const float* src, float* dst, uint32_t* flags, int64_t B, int32_t R,
                     hipStream_t stream);

/*
 * Synchronise the plan's device and read the plan's status word.  This call,
 * ebag_a2a_status_ex, ebag_a2a_reset, ebag_a2a_trace and ebag_a2a_occupancy
 * make the plan's device current for their duration and then restore the
 * caller's current device.
 *   timed_out: 1 if a consumer gave up waiting, else 0.
 *   first_missing_flag: lowest flag index a consumer timed out on, else -1.
 * Returns EBAG_OK, or EBAG_ETIMEOUT when timed_out is set.
 */
int ebag_a2a_status(ebag_a2a_t h, int32_t* timed_out, int32_t* first_missing_flag);

/*
 * Extended status: out[0] timed_out, out[1] first missing flag index (-1
 * none), out[2] flags seen above the expected epoch (double publication),
 * out[3] first bad bag t*B+b found by check_indices (-1 none).
 */
int ebag_a2a_status_ex(ebag_a2a_t h, int32_t out[4]);

/* Zero the slice counters, the persistent-grid ticket, the delivery's piece
 * counters and the status word (after a timeout or an aborted sequence).
 * Synchronous. */
int ebag_a2a_reset(ebag_a2a_t h);

/*
 * Copy the per-slice timestamps of the most recent traced forward/consume
 * (plan created with trace = 1) to host arrays of n entries, one per flag
 * index (n at most the flag count of max_batch): release_ticks[f] when flag
 * f was released, drain_ticks[f] when a consumer finished copying its slice
 * (0 = not recorded).  Ticks are the device's
 * constant wall clock; *ticks_per_us receives its rate.  Synchronous.
 */
int ebag_a2a_trace(ebag_a2a_t h, uint64_t* release_ticks, uint64_t* drain_ticks, int64_t n,
                   double* ticks_per_us);

/*
 * Launch geometry of this plan's fused pooling kernel, for sizing persistent
 * grids (the occupancy study of Sec. IV-C: time versus the fraction of
 * resident workgroup slots in use, Fig. 13).  weighted selects the weighted-sum
 * kernel.  out[0]: workgroups of that kernel that fit on one CU at once
 * (registers and LDS, from the HIP occupancy query); out[1]: CUs of the
 * plan's device; out[2]: threads per workgroup; out[3]: bags per run (K).
 * Returns EBAG_OK, EBAG_EINVAL (null argument) or EBAG_EHIP.
 */
int ebag_a2a_occupancy(ebag_a2a_t h, int32_t weighted, int32_t out[4]);

/*
 * Create a HIP stream with a hardware queue of its own (a CU-masked stream
 * with every CU enabled), for running ebag_a2a_consume concurrently with a
 * forward: ordinary streams of a process share a few hardware queues, and
 * two kernels on one queue run one after the other.  Release it with
 * ebag_a2a_queue_stream_destroy (or hipStreamDestroy).
 */
int ebag_a2a_queue_stream_create(hipStream_t* out);

/* Wait for a stream from ebag_a2a_queue_stream_create to drain, then destroy
 * it (its hardware queue is released).  Returns EBAG_OK, EBAG_EINVAL (null
 * stream) or EBAG_EHIP. */
int ebag_a2a_queue_stream_destroy(hipStream_t stream);

/* Release the plan's device memory.  NULL is ignored. */
void ebag_a2a_destroy(ebag_a2a_t h);

/* Message for the calling thread's most recent failing call ("" if none). */
const char* ebag_a2a_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EBAG_A2A_H */
