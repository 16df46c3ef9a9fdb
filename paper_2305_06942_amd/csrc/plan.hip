// Host side of the C ABI declared in include/ebag_a2a.h: argument checks,
// plan-owned device memory, launch geometry and kernel dispatch.
#include <algorithm>
#include <climits>
#include <cstdlib>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "ebag_a2a.h"
#include "common.h"
#include "table_order.h"
#include "backward.h"
#include "consume.h"
#include "device_guard.h"

using namespace ebag;

namespace {

thread_local std::string g_err;

}  // namespace

// Record the calling thread's error message (shared by every entry point of
// the library, read back with ebag_a2a_last_error).
int ebag::fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

void ebag::clear_error() { g_err.clear(); }

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(EBAG_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(call, what)              \
  do {                                   \
    hipError_t e_ = (call);              \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int log2_exact(int v) {
  for (int s = 0; s <= 6; ++s)
    if ((1 << s) == v) return s;
  return -1;
}

}  // namespace

// MI355X: 8 XCDs of 32 CUs.
int ebag::xcd_count(int num_cus) { return (num_cus % 32 == 0 && num_cus >= 64) ? num_cus / 32 : 1; }

// Table-major runs: 1 -> one table group per XCD when the tables divide
// evenly (each XCD pools its own tables); 2 -> one table at a time for the
// whole device.
int32_t ebag::table_groups_for(const ebag_a2a_opts_t& o, int32_t T, int n_xcd) {
  return o.table_major == 2 ? 1 : o.table_major == 1 ? (T % n_xcd == 0 ? n_xcd : 1) : 0;
}

// One kind of call whose device state a plan shares between calls: the
// event recorded after the last one and the stream it was enqueued on.
struct InFlight {
  hipEvent_t done = nullptr;
  hipStream_t stream = nullptr;
  bool pending = false;
};

struct ebag_a2a_plan {
  int device = 0;
  int32_t T = 0;
  int dtype = 0;
  int elt = 4;
  int32_t C = 0;
  int64_t max_batch = 0;
  int32_t max_ranks = 0;
  int32_t sum_dim = 0;
  int num_cus = 0;
  int32_t table_groups = 0;  // SliceOrder::table_groups for this plan's options
  double ticks_per_us = 100.0;
  ebag_a2a_opts_t opts{};
  std::vector<TabMeta> meta;
  std::vector<const void*> host_tables;  // last table pointers uploaded
  bool tables_valid = false;
  // The last forward's, backward's and delivery's completion, for refusing
  // another of the same kind on another stream while it still runs (the
  // slice counters and scratch, the table bases and the piece counters are
  // shared).
  InFlight fwd, bwd, dlv;
  int64_t max_chunks = 0;
  int64_t max_flags = 0;   // max_chunks, times T with per-table slices
  // device memory
  TabMeta* d_meta = nullptr;
  int32_t* d_tperm = nullptr;
  const void** d_tables = nullptr;
  uint32_t* d_counters = nullptr;
  float* d_scratch = nullptr;
  int32_t* d_status = nullptr;
  uint32_t* d_ticket = nullptr;  // persistent-grid run ticket [2], self-resetting
  int64_t* d_value_base = nullptr;    // backward: first float of each table's block [T + 1]
  uint32_t* d_deliver_cnt = nullptr;  // deliver: pieces stored per slice [max_chunks], self-resetting
  uint64_t* d_trace_release = nullptr;
  uint64_t* d_trace_drain = nullptr;
};

namespace {

void free_plan(ebag_a2a_plan* h) {
  if (!h) return;
  for (InFlight* f : {&h->fwd, &h->bwd, &h->dlv})
    if (f->done) (void)hipEventDestroy(f->done);
  (void)hipFree(h->d_meta);
  (void)hipFree(h->d_tperm);
  (void)hipFree(h->d_tables);
  (void)hipFree(h->d_counters);
  (void)hipFree(h->d_scratch);
  (void)hipFree(h->d_status);
  (void)hipFree(h->d_ticket);
  (void)hipFree(h->d_value_base);
  (void)hipFree(h->d_deliver_cnt);
  (void)hipFree(h->d_trace_release);
  (void)hipFree(h->d_trace_drain);
  delete h;
}

}  // namespace

int ebag::check_opts(const ebag_a2a_opts_t& o) {
  if (o.waves_per_wg < 1 || o.waves_per_wg > 16) return fail(EBAG_EINVAL, "waves_per_wg must be in [1, 16]");
  if (o.bags_per_run < 1) return fail(EBAG_EINVAL, "bags_per_run must be >= 1");
  if (o.rows_in_flight != 4 && o.rows_in_flight != 8 && o.rows_in_flight != 16)
    return fail(EBAG_EINVAL, "rows_in_flight must be 4, 8 or 16");
  if (o.persistent_wgs_per_cu < -1) return fail(EBAG_EINVAL, "persistent_wgs_per_cu must be >= -1");
  if (o.release_mode < 0 || o.release_mode > 1) return fail(EBAG_EINVAL, "release_mode must be 0 or 1");
  if (o.chunk_order != 0 && o.chunk_order != 1) return fail(EBAG_EINVAL, "chunk_order must be 0 or 1");
  if (o.self_rank < 0) return fail(EBAG_EINVAL, "self_rank must be >= 0");
  if (o.stream_rows < 0 || o.stream_rows > 1) return fail(EBAG_EINVAL, "stream_rows must be 0 or 1");
  if (o.consumer_wgs < 1) return fail(EBAG_EINVAL, "consumer_wgs must be >= 1");
  if (o.consume_timeout_us < 1) return fail(EBAG_EINVAL, "consume_timeout_us must be >= 1");
  if (o.pooling_mode != 0 && o.pooling_mode != 1) return fail(EBAG_EINVAL, "pooling_mode must be 0 (sum) or 1 (mean)");
  if (o.slice_granule != 0 && o.slice_granule != 1) return fail(EBAG_EINVAL, "slice_granule must be 0 or 1");
  if (o.table_major < 0 || o.table_major > 2) return fail(EBAG_EINVAL, "table_major must be 0, 1 or 2");
  if (o.consume_nontemporal != 0 && o.consume_nontemporal != 1)
    return fail(EBAG_EINVAL, "consume_nontemporal must be 0 or 1");
  if (o.backward_bags_per_run < 1) return fail(EBAG_EINVAL, "backward_bags_per_run must be >= 1");
  if (o.backward_waves_per_wg < 1 || o.backward_waves_per_wg > 16)
    return fail(EBAG_EINVAL, "backward_waves_per_wg must be in [1, 16]");
  if (o.deliver_wgs < 1) return fail(EBAG_EINVAL, "deliver_wgs must be >= 1");
  if (o.deliver_waves_per_wg < 1 || o.deliver_waves_per_wg > 16)
    return fail(EBAG_EINVAL, "deliver_waves_per_wg must be in [1, 16]");
  return EBAG_OK;
}

namespace {

// B / R checks shared by every entry point that walks slices; fills the
// slice order.
int check_split(const ebag_a2a_plan* h, int64_t B, int32_t R, SliceOrder* so) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != h->device)
    return fail(EBAG_EINVAL, "the plan belongs to device %d, but device %d is current", h->device, dev);
  if (B <= 0 || R <= 0) return fail(EBAG_EINVAL, "B and R must be positive (B=%lld R=%d)", (long long)B, R);
  if (B > h->max_batch) return fail(EBAG_EINVAL, "B=%lld exceeds max_batch=%lld", (long long)B, (long long)h->max_batch);
  if (R > h->max_ranks) return fail(EBAG_EINVAL, "R=%d exceeds max_ranks=%d", R, h->max_ranks);
  if (B % R != 0) return fail(EBAG_EINVAL, "B=%lld is not a multiple of R=%d", (long long)B, R);
  if ((B / R) % h->C != 0)
    return fail(EBAG_EINVAL, "B/R=%lld is not a multiple of chunk_samples=%d", (long long)(B / R), h->C);
  if (h->opts.chunk_order == 1 && h->opts.self_rank >= R)
    return fail(EBAG_EINVAL, "self_rank=%d is not a destination (R=%d)", h->opts.self_rank, R);
  so->n_chunks = B / h->C;
  so->per_rank = (B / R) / h->C;
  so->self = h->opts.self_rank;
  so->order = h->opts.chunk_order;
  so->table_groups = h->table_groups;
  return EBAG_OK;
}

// Validation shared by both forwards; fills the slice order.
int check_forward(const ebag_a2a_plan* h, const void* const* tables, const int32_t* indices, const int64_t* offsets,
                  const float* weights, int64_t B, int32_t R, const float* send_buf, const uint32_t* flags,
                  SliceOrder* so) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  if (weights && h->opts.pooling_mode == 1) return fail(EBAG_EINVAL, "mean pooling takes no weights");
  if (!tables) return fail(EBAG_EINVAL, "null table pointer array");
  if (!offsets || !send_buf || !flags) return fail(EBAG_EINVAL, "null offsets, send_buf or flags");
  if (!indices) return fail(EBAG_EINVAL, "null indices");
  const int rc = check_split(h, B, R, so);
  if (rc) return rc;
  if (!aligned16(send_buf)) return fail(EBAG_EINVAL, "send_buf is not 16-byte aligned");
  for (int32_t t = 0; t < h->T; ++t) {
    if (!tables[t] && h->meta[t].rows > 0) return fail(EBAG_EINVAL, "null pointer for table %d", t);
    if (!aligned16(tables[t])) return fail(EBAG_EINVAL, "table %d is not 16-byte aligned", t);
  }
  return EBAG_OK;
}

constexpr int kPtrBatch = 64;
struct PtrBatch {
  const void** dst;
  int32_t n;
  int32_t pad;
  const void* p[kPtrBatch];
};

// Writes n table pointers carried in the kernel arguments.
__global__ __launch_bounds__(64) void put_pointers_kernel(const PtrBatch b) {
  if ((int)threadIdx.x < b.n) b.dst[threadIdx.x] = b.p[threadIdx.x];
}

// Upload table pointers when they differ from the last upload: small
// kernels ordered on `stream` that carry the pointers as arguments, so the
// host neither waits nor keeps the array (it may be reused at once).
int sync_tables(ebag_a2a_plan* h, const void* const* tables, hipStream_t stream) {
  if (h->tables_valid && std::memcmp(h->host_tables.data(), tables, sizeof(void*) * h->T) == 0) return EBAG_OK;
  h->tables_valid = false;  // stays false unless every upload is enqueued
  for (int32_t first = 0; first < h->T; first += kPtrBatch) {
    PtrBatch b;
    std::memset(&b, 0, sizeof b);
    b.dst = h->d_tables + first;
    b.n = h->T - first < kPtrBatch ? h->T - first : kPtrBatch;
    for (int32_t i = 0; i < b.n; ++i) b.p[i] = tables[first + i];
    hipLaunchKernelGGL(put_pointers_kernel, dim3(1), dim3(64), 0, stream, b);
    HIP_TRY(hipGetLastError(), "upload table pointers");
  }
  std::memcpy(h->host_tables.data(), tables, sizeof(void*) * h->T);
  h->tables_valid = true;
  return EBAG_OK;
}

// Whether `stream` is being captured into a graph.  Work that waits for a
// host-chosen epoch cannot be replayed from a graph: the epoch is fixed at
// capture, so a replay would not wait for the flags of its own producer.
bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  return hipStreamIsCapturing(stream, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone;
}

// One call of each kind in flight per plan: a call on another stream than
// the last one of its kind, while that one has not completed, would share its
// device state.
int check_busy(InFlight& f, hipStream_t stream, const char* what) {
  if (!f.pending || stream == f.stream || capturing(stream)) return EBAG_OK;
  const hipError_t e = hipEventQuery(f.done);
  if (e == hipErrorNotReady)
    return fail(EBAG_EBUSY, "a %s of this plan is still running on another stream (the plan's device state for it "
                            "is shared): order them on one stream or wait for it", what);
  if (e != hipSuccess) return hip_fail(e, "query the last call");
  f.pending = false;
  return EBAG_OK;
}

// Remember the call just enqueued on `stream` (not under graph capture).
int note_call(InFlight& f, hipStream_t stream) {
  if (capturing(stream)) {
    f.pending = false;
    return EBAG_OK;
  }
  HIP_TRY(hipEventRecord(f.done, stream), "record the call's completion");
  f.stream = stream;
  f.pending = true;
  return EBAG_OK;
}

}  // namespace

void ebag::fill_pool_args(const PoolSetup& s, const int32_t* indices, const int64_t* offsets, const float* weights,
                          int64_t B, const SliceOrder& so, float* out, uint32_t* flags, PoolArgs* a) {
  std::memset(a, 0, sizeof *a);
  const ebag_a2a_opts_t& o = *s.o;
  int32_t K = o.bags_per_run < s.C ? o.bags_per_run : s.C;
  // The fast kernels keep a run's pooled rows in LDS (K x max dim floats):
  // cap that buffer at 16 KiB.
  int32_t max_dim = 0;
  for (int32_t t = 0; t < s.T; ++t) max_dim = s.meta[t].dim > max_dim ? s.meta[t].dim : max_dim;
  const int32_t k_cap = 16384 / (4 * max_dim) > 1 ? 16384 / (4 * max_dim) : 1;
  if (K > k_cap) K = k_cap;
  a->tables = s.d_tables;
  a->meta = s.d_meta;
  a->tperm = s.d_tperm;
  a->indices = indices;
  a->offsets = offsets;
  a->weights = weights;
  a->out = out;
  a->counters = s.d_counters;
  a->flags = flags;
  a->status = s.d_status;
  a->trace_release = o.trace ? s.d_trace_release : nullptr;
  a->ticket = s.d_ticket;
  a->B = B;
  a->K = K;
  a->J = (s.C + K - 1) / K;
  a->T = s.T;
  a->C = s.C;
  a->nruns = so.n_chunks * (int64_t)s.T * a->J;
  a->suppress = o.debug_suppress_flag;
  a->so = so;
  a->sum_dim = s.sum_dim;
  a->check = o.check_indices;
  a->release_mode = o.release_mode;
  a->waves = o.waves_per_wg;
  a->out_floats = K * max_dim;
  a->stream_rows = o.stream_rows;
  a->mean = o.pooling_mode == 1;
  a->per_table = o.slice_granule == 1;
}

// The fast pooling kernels handle tables below 4 GiB (32-bit buffer offsets)
// whose rows are 2^k <= 64 sixteen-byte vectors, without index reporting;
// anything else uses the general kernels.
bool ebag::needs_safe(const PoolSetup& s) {
  if (s.o->check_indices) return true;
  for (int32_t t = 0; t < s.T; ++t) {
    const TabMeta& m = s.meta[t];
    if (m.vshift < 0 || m.rows * m.row_bytes > (int64_t)0xFFFFFFFFll) return true;
  }
  return false;
}

int ebag::pool_grid(const PoolSetup& s, int64_t nruns, bool fused, bool weighted, int block, int out_floats) {
  int64_t grid = nruns;
  if (s.o->persistent_wgs_per_cu != 0) {
    int per_cu = s.o->persistent_wgs_per_cu;
    if (per_cu < 0)
      per_cu = pool_max_wgs_per_cu(s.dtype, s.o->rows_in_flight, weighted, fused, needs_safe(s), block, out_floats);
    if (per_cu < 1) per_cu = 1;
    const int64_t pg = (int64_t)per_cu * s.num_cus;
    if (pg < grid) grid = pg;
  }
  if (grid > INT_MAX) grid = INT_MAX;
  return (int)grid;
}

namespace {

// The plan as a pooling launch sees it.
PoolSetup setup_of(const ebag_a2a_plan* h) {
  PoolSetup s;
  s.o = &h->opts;
  s.meta = h->meta.data();
  s.T = h->T;
  s.C = h->C;
  s.sum_dim = h->sum_dim;
  s.dtype = h->dtype;
  s.num_cus = h->num_cus;
  s.table_groups = h->table_groups;
  s.d_tables = h->d_tables;
  s.d_meta = h->d_meta;
  s.d_tperm = h->d_tperm;
  s.d_counters = h->d_counters;
  s.d_status = h->d_status;
  s.d_trace_release = h->d_trace_release;
  s.d_ticket = h->d_ticket;
  return s;
}

}  // namespace



extern "C" {

int ebag_a2a_default_opts(ebag_a2a_opts_t* o) {
  if (!o) return fail(EBAG_EINVAL, "null opts");
  std::memset(o, 0, sizeof *o);
  o->waves_per_wg = 4;
  o->bags_per_run = 16;
  o->rows_in_flight = 8;
  o->persistent_wgs_per_cu = 0;
  o->release_mode = 1;
  o->chunk_order = 0;
  o->self_rank = 0;
  o->trace = 0;
  o->check_indices = 0;
  o->debug_suppress_flag = -1;
  o->consumer_wgs = 512;
  o->stream_rows = 1;
  o->consume_timeout_us = 5000000;
  o->backward_bags_per_run = 4;
  o->backward_waves_per_wg = 16;
  o->deliver_wgs = 32;
  o->deliver_waves_per_wg = 8;
  return EBAG_OK;
}

int ebag_a2a_create(ebag_a2a_t* out, int32_t num_tables, const int64_t* rows_per_table,
                    const int32_t* dim_per_table, int32_t table_dtype, int32_t chunk_samples,
                    int64_t max_batch, int32_t max_ranks, const ebag_a2a_opts_t* opts) {
  if (!out) return fail(EBAG_EINVAL, "null output handle");
  *out = nullptr;
  if (num_tables <= 0) return fail(EBAG_EINVAL, "num_tables must be positive");
  if (!rows_per_table || !dim_per_table) return fail(EBAG_EINVAL, "null rows/dims array");
  if (table_dtype != EBAG_F32 && table_dtype != EBAG_F16 && table_dtype != EBAG_BF16)
    return fail(EBAG_EINVAL, "unknown table dtype %d", (int)table_dtype);
  if (chunk_samples <= 0) return fail(EBAG_EINVAL, "chunk_samples must be positive");
  if (max_batch <= 0 || max_ranks <= 0) return fail(EBAG_EINVAL, "max_batch and max_ranks must be positive");
  ebag_a2a_opts_t o;
  if (opts)
    o = *opts;
  else
    ebag_a2a_default_opts(&o);
  int rc = check_opts(o);
  if (rc) return rc;
  const int elt = table_dtype == EBAG_F32 ? 4 : 2;
  std::vector<TabMeta> meta(num_tables);
  int64_t sum_dim = 0;
  for (int32_t t = 0; t < num_tables; ++t) {
    const int64_t rows = rows_per_table[t];
    const int32_t D = dim_per_table[t];
    if (rows < 0 || rows > INT32_MAX) return fail(EBAG_EINVAL, "rows of table %d out of range", t);
    if (D <= 0) return fail(EBAG_EINVAL, "dim of table %d must be positive", t);
    if (((int64_t)D * elt) % 16 != 0)
      return fail(EBAG_EINVAL, "table %d: D*elt = %lld bytes is not a multiple of 16", t, (long long)D * elt);
    meta[t].rows = rows;
    meta[t].row_bytes = (int64_t)D * elt;
    meta[t].dim = D;
    meta[t].col_off = (int32_t)sum_dim;
    meta[t].vecs = (int32_t)(meta[t].row_bytes / 16);
    meta[t].vshift = log2_exact(meta[t].vecs);
    sum_dim += D;
  }
  if (sum_dim > INT32_MAX / 4) return fail(EBAG_EINVAL, "sum of dims too large");
  if ((int64_t)max_batch * sum_dim > (int64_t)1 << 40) return fail(EBAG_EINVAL, "max_batch * sum(D) too large");
  // A slice is one message: the per-table consumer and delivery address it
  // with 32-bit byte offsets.
  if ((int64_t)chunk_samples * sum_dim * 4 > INT32_MAX)
    return fail(EBAG_EINVAL, "a slice (chunk_samples x sum(D) fp32) must be below 2 GiB");

  ebag_a2a_plan* h = new (std::nothrow) ebag_a2a_plan();
  if (!h) return fail(EBAG_ENOMEM, "host allocation failed");
  h->T = num_tables;
  h->dtype = (int)table_dtype;
  h->elt = elt;
  h->C = chunk_samples;
  h->max_batch = max_batch;
  h->max_ranks = max_ranks;
  h->sum_dim = (int32_t)sum_dim;
  h->opts = o;
  h->meta = meta;
  h->host_tables.assign(num_tables, nullptr);
  h->max_chunks = (max_batch + chunk_samples - 1) / chunk_samples;
  h->max_flags = h->max_chunks * (o.slice_granule == 1 ? num_tables : 1);

#define CREATE_TRY(call, what)                                                             \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess) {                                                                \
      int r_ = e_ == hipErrorOutOfMemory ? fail(EBAG_ENOMEM, "%s: out of device memory", what) \
                                         : hip_fail(e_, what);                              \
      free_plan(h);                                                                        \
      return r_;                                                                           \
    }                                                                                      \
  } while (0)

  CREATE_TRY(hipGetDevice(&h->device), "hipGetDevice");
  CREATE_TRY(hipDeviceGetAttribute(&h->num_cus, hipDeviceAttributeMultiprocessorCount, h->device), "CU count");
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->device) == hipSuccess && khz > 0)
    h->ticks_per_us = khz / 1000.0;
  std::vector<int64_t> widths(num_tables);
  for (int32_t t = 0; t < num_tables; ++t) widths[t] = meta[t].row_bytes;
  const int n_xcd = xcd_count(h->num_cus);
  std::vector<int32_t> tperm(num_tables), order_work(num_tables);
  std::vector<int64_t> order_load(kMaxXcd);
  table_order(widths.data(), num_tables, n_xcd, tperm.data(), order_work.data(), order_load.data());
  h->table_groups = table_groups_for(o, num_tables, n_xcd);
  CREATE_TRY(hipMalloc((void**)&h->d_meta, sizeof(TabMeta) * num_tables), "alloc table meta");
  CREATE_TRY(hipMemcpy(h->d_meta, meta.data(), sizeof(TabMeta) * num_tables, hipMemcpyHostToDevice), "upload meta");
  CREATE_TRY(hipMalloc((void**)&h->d_tperm, sizeof(int32_t) * num_tables), "alloc table order");
  CREATE_TRY(hipMemcpy(h->d_tperm, tperm.data(), sizeof(int32_t) * num_tables, hipMemcpyHostToDevice), "upload order");
  CREATE_TRY(hipMalloc((void**)&h->d_tables, sizeof(void*) * num_tables), "alloc table pointers");
  CREATE_TRY(hipMalloc((void**)&h->d_counters, sizeof(uint32_t) * h->max_flags), "alloc slice counters");
  CREATE_TRY(hipMemset(h->d_counters, 0, sizeof(uint32_t) * h->max_flags), "zero slice counters");
  CREATE_TRY(hipMalloc((void**)&h->d_scratch, sizeof(float) * (size_t)max_batch * (size_t)sum_dim), "alloc scratch");
  CREATE_TRY(hipMalloc((void**)&h->d_value_base, sizeof(int64_t) * (num_tables + 1)), "alloc value bases");
  CREATE_TRY(hipMalloc((void**)&h->d_deliver_cnt, sizeof(uint32_t) * h->max_chunks), "alloc deliver counters");
  CREATE_TRY(hipMemset(h->d_deliver_cnt, 0, sizeof(uint32_t) * h->max_chunks), "zero deliver counters");
  CREATE_TRY(hipMalloc((void**)&h->d_ticket, 2 * sizeof(uint32_t)), "alloc run ticket");
  CREATE_TRY(hipMemset(h->d_ticket, 0, 2 * sizeof(uint32_t)), "zero run ticket");
  for (InFlight* f : {&h->fwd, &h->bwd, &h->dlv})
    CREATE_TRY(hipEventCreateWithFlags(&f->done, hipEventDisableTiming), "create completion event");
  CREATE_TRY(hipMalloc((void**)&h->d_status, sizeof(kStatusInit)), "alloc status");
  CREATE_TRY(hipMemcpy(h->d_status, kStatusInit, sizeof(kStatusInit), hipMemcpyHostToDevice), "init status");
  if (o.trace) {
    CREATE_TRY(hipMalloc((void**)&h->d_trace_release, sizeof(uint64_t) * h->max_flags), "alloc trace");
    CREATE_TRY(hipMalloc((void**)&h->d_trace_drain, sizeof(uint64_t) * h->max_flags), "alloc trace");
    CREATE_TRY(hipMemset(h->d_trace_release, 0, sizeof(uint64_t) * h->max_flags), "zero trace");
    CREATE_TRY(hipMemset(h->d_trace_drain, 0, sizeof(uint64_t) * h->max_flags), "zero trace");
  }
#undef CREATE_TRY
  *out = h;
  g_err.clear();
  return EBAG_OK;
}

int ebag_a2a_forward(ebag_a2a_t h, const void* const* tables, const int32_t* indices, const int64_t* offsets,
                     const float* weights, int64_t B, int32_t R, float* send_buf, uint32_t* flags,
                     hipStream_t stream) {
  SliceOrder so;
  int rc = check_forward(h, tables, indices, offsets, weights, B, R, send_buf, flags, &so);
  if (rc) return rc;
  rc = check_busy(h->fwd, stream, "forward");
  if (rc) return rc;
  PoolArgs a;
  fill_pool_args(setup_of(h), indices, offsets, weights, B, so, send_buf, flags, &a);
  const int block = 64 * h->opts.waves_per_wg;
  if (a.nruns >= INT_MAX) return fail(EBAG_EINVAL, "too many runs (%lld) for one launch", (long long)a.nruns);
  rc = sync_tables(h, tables, stream);
  if (rc) return rc;
  const int grid = pool_grid(setup_of(h), a.nruns, true, weights != nullptr, block, a.out_floats);
  hipError_t e = launch_pool(h->dtype, h->opts.rows_in_flight, weights != nullptr, true, needs_safe(setup_of(h)), a, grid,
                             block, stream);
  if (e != hipSuccess) return hip_fail(e, "launch fused pooling kernel");
  return note_call(h->fwd, stream);
}

int ebag_a2a_unfused_forward(ebag_a2a_t h, const void* const* tables, const int32_t* indices,
                             const int64_t* offsets, const float* weights, int64_t B, int32_t R,
                             float* send_buf, uint32_t* flags, hipStream_t stream) {
  SliceOrder so;
  int rc = check_forward(h, tables, indices, offsets, weights, B, R, send_buf, flags, &so);
  if (rc) return rc;
  rc = check_busy(h->fwd, stream, "forward");
  if (rc) return rc;
  PoolArgs a;
  fill_pool_args(setup_of(h), indices, offsets, weights, B, so, h->d_scratch, flags, &a);
  const int block = 64 * h->opts.waves_per_wg;
  if (a.nruns >= INT_MAX) return fail(EBAG_EINVAL, "too many runs (%lld) for one launch", (long long)a.nruns);
  if (so.n_chunks * h->T > INT_MAX) return fail(EBAG_EINVAL, "too many slices x tables for the repack grid");
  rc = sync_tables(h, tables, stream);
  if (rc) return rc;
  const int grid = pool_grid(setup_of(h), a.nruns, false, weights != nullptr, block, a.out_floats);
  hipError_t e = launch_pool(h->dtype, h->opts.rows_in_flight, weights != nullptr, false, needs_safe(setup_of(h)), a, grid,
                             block, stream);
  if (e != hipSuccess) return hip_fail(e, "launch pooling kernel");
  RepackArgs r;
  std::memset(&r, 0, sizeof r);
  r.scratch = h->d_scratch;
  r.send = send_buf;
  r.meta = h->d_meta;
  r.tperm = h->d_tperm;
  r.B = B;
  r.so = so;
  r.T = h->T;
  r.C = h->C;
  r.sum_dim = h->sum_dim;
  const int64_t rgrid = so.n_chunks * h->T;
  if (rgrid > INT_MAX) return fail(EBAG_EINVAL, "too many slices x tables for the repack grid");
  e = launch_repack(r, (int)rgrid, 256, stream);
  if (e != hipSuccess) return hip_fail(e, "launch repack kernel");
  PublishArgs pa;
  pa.flags = flags;
  pa.trace_release = h->opts.trace ? h->d_trace_release : nullptr;
  pa.n_flags = so.n_chunks * (h->opts.slice_granule == 1 ? h->T : 1);
  pa.suppress = h->opts.debug_suppress_flag;
  e = launch_publish(pa, stream);
  if (e != hipSuccess) return hip_fail(e, "launch flag publication kernel");
  return note_call(h->fwd, stream);
}

int ebag_a2a_consume(ebag_a2a_t h, const float* send_buf, const uint32_t* flags, float* recv_buf, int64_t B,
                     int32_t R, uint32_t expected_epoch, hipStream_t stream) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  if (!send_buf || !flags || !recv_buf) return fail(EBAG_EINVAL, "null send_buf, flags or recv_buf");
  if (!aligned16(send_buf) || !aligned16(recv_buf)) return fail(EBAG_EINVAL, "send/recv not 16-byte aligned");
  SliceOrder so;
  const int rc = check_split(h, B, R, &so);
  if (rc) return rc;
  if (capturing(stream))
    return fail(EBAG_EUNSUPPORTED, "consume waits for a fixed epoch; it cannot be captured into a graph");
  ConsumeArgs c;
  std::memset(&c, 0, sizeof c);
  c.send = send_buf;
  c.flags = flags;
  c.recv = recv_buf;
  c.status = h->d_status;
  c.trace_drain = h->opts.trace ? h->d_trace_drain : nullptr;
  c.chunk_floats = (int64_t)h->C * h->sum_dim;
  c.timeout_ticks = (uint64_t)((double)h->opts.consume_timeout_us * h->ticks_per_us);
  c.so = so;  // the producer's order, table-major included
  c.epoch = expected_epoch;
  c.coherent_loads = h->opts.release_mode == 1;
  c.nontemporal = h->opts.consume_nontemporal;
  c.per_table = h->opts.slice_granule == 1;
  c.meta = h->d_meta;
  c.tperm = h->d_tperm;
  c.T = h->T;
  c.C = h->C;
  c.sum_dim = h->sum_dim;
  // Work items: pieces of at most 32 KiB per slice, or one per (slice, table).
  const int64_t chunk_f4 = c.chunk_floats / 4;
  c.piece_f4 = chunk_f4 < 2048 ? chunk_f4 : 2048;
  c.pieces = (chunk_f4 + c.piece_f4 - 1) / c.piece_f4;
  const int64_t items = c.so.n_chunks * (c.per_table ? h->T : c.pieces);
  int64_t grid = h->opts.consumer_wgs;
  if (grid > items) grid = items;
  hipError_t e = launch_consume(c, (int)grid, 64, stream);
  if (e != hipSuccess) return hip_fail(e, "launch consumer kernel");
  return EBAG_OK;
}

int ebag_a2a_backward(ebag_a2a_t h, const float* grad_buf, const uint32_t* grad_flags, uint32_t expected_epoch,
                      const int64_t* offsets, const float* weights, int64_t B, int32_t R, float* values,
                      hipStream_t stream) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  if (!grad_buf || !offsets || !values) return fail(EBAG_EINVAL, "null grad_buf, offsets or values");
  if (!aligned16(grad_buf) || !aligned16(values)) return fail(EBAG_EINVAL, "grad_buf or values not 16-byte aligned");
  if (weights && h->opts.pooling_mode == 1) return fail(EBAG_EINVAL, "mean pooling takes no weights");
  if (grad_flags && capturing(stream))
    return fail(EBAG_EUNSUPPORTED, "backward with flags waits for a fixed epoch; it cannot be captured into a graph");
  SliceOrder so;
  int rc = check_split(h, B, R, &so);
  if (rc) return rc;
  int32_t max_dim = 0;
  for (const TabMeta& m : h->meta) max_dim = m.dim > max_dim ? m.dim : max_dim;
  const int block = 64 * h->opts.backward_waves_per_wg;
  // LDS holds the run's K gradient rows and K + 1 offsets: K is capped so
  // that they fit in 64 KiB.
  int32_t K = h->opts.backward_bags_per_run < h->C ? h->opts.backward_bags_per_run : h->C;
  const int32_t k_fit = (int32_t)(65536 / ((size_t)max_dim * sizeof(float) + sizeof(int64_t)) - 1);
  if (k_fit < 1) return fail(EBAG_EUNSUPPORTED, "backward: rows of %d floats do not fit in LDS", max_dim);
  if (K > k_fit) K = k_fit;
  if (K > block - 1) K = block - 1;
  const size_t lds = (size_t)K * max_dim * sizeof(float) + (size_t)(K + 1) * sizeof(int64_t);
  BackwardArgs a;
  std::memset(&a, 0, sizeof a);
  a.grad = grad_buf;
  a.flags = grad_flags;
  a.values = values;
  a.offsets = offsets;
  a.weights = weights;
  a.meta = h->d_meta;
  a.tperm = h->d_tperm;
  a.value_base = h->d_value_base;
  a.status = h->d_status;
  a.B = B;
  a.timeout_ticks = (uint64_t)((double)h->opts.consume_timeout_us * h->ticks_per_us);
  a.so = so;
  a.T = h->T;
  a.C = h->C;
  a.K = K;
  a.J = (h->C + a.K - 1) / a.K;
  a.nruns = so.n_chunks * (int64_t)h->T * a.J;
  if (a.nruns >= INT_MAX) return fail(EBAG_EINVAL, "too many runs (%lld) for one launch", (long long)a.nruns);
  a.sum_dim = h->sum_dim;
  a.max_dim = max_dim;
  a.per_table = h->opts.slice_granule == 1;
  a.mean = h->opts.pooling_mode == 1;
  a.epoch = expected_epoch;
  rc = check_busy(h->bwd, stream, "backward");
  if (rc) return rc;
  const hipError_t e = launch_backward(a, h->d_value_base, block, lds, stream);
  if (e != hipSuccess) return hip_fail(e, "launch backward kernels");
  return note_call(h->bwd, stream);
}

int ebag_a2a_deliver(ebag_a2a_t h, const float* src, float* dst, uint32_t* flags, int64_t B, int32_t R,
                     hipStream_t stream) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  if (!src || !dst || !flags) return fail(EBAG_EINVAL, "null src, dst or flags");
  if (!aligned16(src) || !aligned16(dst)) return fail(EBAG_EINVAL, "src or dst not 16-byte aligned");
  SliceOrder so;
  int rc = check_split(h, B, R, &so);
  if (rc) return rc;
  DeliverArgs d;
  std::memset(&d, 0, sizeof d);
  d.src = src;
  d.dst = dst;
  d.flags = flags;
  d.counters = h->d_deliver_cnt;
  d.meta = h->d_meta;
  d.tperm = h->d_tperm;
  d.chunk_floats = (int64_t)h->C * h->sum_dim;
  const int64_t chunk_f4 = d.chunk_floats / 4;
  d.piece_f4 = chunk_f4 < 2048 ? chunk_f4 : 2048;
  d.pieces = (chunk_f4 + d.piece_f4 - 1) / d.piece_f4;
  d.so = so;
  d.T = h->T;
  d.C = h->C;
  d.sum_dim = h->sum_dim;
  d.per_table = h->opts.slice_granule == 1;
  const int64_t items = so.n_chunks * (d.per_table ? h->T : d.pieces);
  const int waves = h->opts.deliver_waves_per_wg;
  int64_t grid = h->opts.deliver_wgs;
  if (grid > (items + waves - 1) / waves) grid = (items + waves - 1) / waves;
  if (grid > INT_MAX) grid = INT_MAX;
  rc = check_busy(h->dlv, stream, "delivery");
  if (rc) return rc;
  const hipError_t e = launch_deliver(d, (int)grid, 64 * waves, stream);
  if (e != hipSuccess) return hip_fail(e, "launch deliver kernel");
  return note_call(h->dlv, stream);
}

int ebag_a2a_status_ex(ebag_a2a_t h, int32_t out[4]) {
  if (!h || !out) return fail(EBAG_EINVAL, "null plan or output");
  const DeviceGuard dg(h->device);
  HIP_TRY(dg.error(), "make the plan's device current");
  HIP_TRY(hipDeviceSynchronize(), "synchronize");
  int32_t s[4];
  HIP_TRY(hipMemcpy(s, h->d_status, sizeof s, hipMemcpyDeviceToHost), "read status");
  out[0] = s[ST_TIMED_OUT];
  out[1] = s[ST_FIRST_MISSING] == INT_MAX ? -1 : s[ST_FIRST_MISSING];
  out[2] = s[ST_OVERSHOOT];
  out[3] = s[ST_FIRST_BAD_BAG] == INT_MAX ? -1 : s[ST_FIRST_BAD_BAG];
  return EBAG_OK;
}

int ebag_a2a_status(ebag_a2a_t h, int32_t* timed_out, int32_t* first_missing_flag) {
  int32_t s[4];
  int rc = ebag_a2a_status_ex(h, s);
  if (rc) return rc;
  if (timed_out) *timed_out = s[0];
  if (first_missing_flag) *first_missing_flag = s[1];
  return s[0] ? EBAG_ETIMEOUT : EBAG_OK;
}

int ebag_a2a_reset(ebag_a2a_t h) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  const DeviceGuard dg(h->device);
  HIP_TRY(dg.error(), "make the plan's device current");
  HIP_TRY(hipDeviceSynchronize(), "synchronize");
  HIP_TRY(hipMemset(h->d_counters, 0, sizeof(uint32_t) * h->max_flags), "zero counters");
  HIP_TRY(hipMemset(h->d_ticket, 0, 2 * sizeof(uint32_t)), "zero run ticket");
  HIP_TRY(hipMemset(h->d_deliver_cnt, 0, sizeof(uint32_t) * h->max_chunks), "zero deliver counters");
  HIP_TRY(hipMemcpy(h->d_status, kStatusInit, sizeof(kStatusInit), hipMemcpyHostToDevice), "reset status");
  if (h->d_trace_release) {
    HIP_TRY(hipMemset(h->d_trace_release, 0, sizeof(uint64_t) * h->max_flags), "zero trace");
    HIP_TRY(hipMemset(h->d_trace_drain, 0, sizeof(uint64_t) * h->max_flags), "zero trace");
  }
  HIP_TRY(hipDeviceSynchronize(), "synchronize");
  return EBAG_OK;
}

int ebag_a2a_trace(ebag_a2a_t h, uint64_t* release_ticks, uint64_t* drain_ticks, int64_t n, double* ticks_per_us) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  if (!h->d_trace_release) return fail(EBAG_EINVAL, "plan was created without trace = 1");
  if (n < 0 || n > h->max_flags) return fail(EBAG_EINVAL, "n=%lld outside [0, %lld]", (long long)n, (long long)h->max_flags);
  const DeviceGuard dg(h->device);
  HIP_TRY(dg.error(), "make the plan's device current");
  HIP_TRY(hipDeviceSynchronize(), "synchronize");
  if (release_ticks && n)
    HIP_TRY(hipMemcpy(release_ticks, h->d_trace_release, sizeof(uint64_t) * n, hipMemcpyDeviceToHost), "read trace");
  if (drain_ticks && n)
    HIP_TRY(hipMemcpy(drain_ticks, h->d_trace_drain, sizeof(uint64_t) * n, hipMemcpyDeviceToHost), "read trace");
  if (ticks_per_us) *ticks_per_us = h->ticks_per_us;
  return EBAG_OK;
}

int ebag_a2a_occupancy(ebag_a2a_t h, int32_t weighted, int32_t out[4]) {
  if (!h || !out) return fail(EBAG_EINVAL, "null plan or output");
  const DeviceGuard dg(h->device);
  HIP_TRY(dg.error(), "make the plan's device current");
  // Same launch shape as a forward: the LDS tile does not depend on B.
  PoolArgs a;
  SliceOrder so;
  std::memset(&so, 0, sizeof so);
  fill_pool_args(setup_of(h), nullptr, nullptr, nullptr, 0, so, nullptr, nullptr, &a);
  const int block = 64 * h->opts.waves_per_wg;
  const int n = pool_max_wgs_per_cu(h->dtype, h->opts.rows_in_flight, weighted != 0, true, needs_safe(setup_of(h)), block,
                                    a.out_floats);
  if (n <= 0) return fail(EBAG_EHIP, "occupancy query failed");
  out[0] = n;
  out[1] = h->num_cus;
  out[2] = block;
  out[3] = a.K;
  clear_error();
  return EBAG_OK;
}

int ebag_a2a_queue_stream_create(hipStream_t* out) {
  if (!out) return fail(EBAG_EINVAL, "null output stream");
  int dev = 0, cus = 0;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "CU count");
  // Every CU enabled: the mask only serves to get a hardware queue of the
  // stream's own.
  std::vector<uint32_t> mask((cus + 31) / 32, 0u);
  for (int i = 0; i < cus; ++i) mask[i / 32] |= 1u << (i % 32);
  HIP_TRY(hipExtStreamCreateWithCUMask(out, (uint32_t)mask.size(), mask.data()), "create stream");
  return EBAG_OK;
}

int ebag_a2a_queue_stream_destroy(hipStream_t stream) {
  if (!stream) return fail(EBAG_EINVAL, "null stream");
  HIP_TRY(hipStreamSynchronize(stream), "synchronize stream");
  HIP_TRY(hipStreamDestroy(stream), "destroy stream");
  return EBAG_OK;
}

void ebag_a2a_destroy(ebag_a2a_t h) { free_plan(h); }

const char* ebag_a2a_last_error(void) { return g_err.c_str(); }

}  // extern "C"
