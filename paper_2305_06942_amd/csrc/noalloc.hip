// Plan-free fused forward that allocates nothing (ebag_a2a_forward_noalloc).
//
// The device memory a plan owns for a forward -- table descriptors, table
// order and pointers, slice counters, status word, persistent-grid ticket --
// lives here in one statically allocated device array, `scratch`, of which
// every GPU the library runs on holds its own copy until the process ends.
// Each call refills the part it uses with a small install kernel (descriptors
// passed by value as kernel arguments, counters, ticket and status cleared),
// then launches the same fused pooling kernel as ebag_a2a_forward.
//
// In host code `scratch` names only the host-side shadow of the array, never
// a device address.  Its address on each device is looked up once, with that
// device current, by hipGetSymbolAddress, and that pointer is what the
// kernels receive.
#include <climits>
#include <cstring>
#include <mutex>

#include "common.h"

namespace ebag {
namespace {

constexpr int kInstallTables = 64;  // table descriptors one install launch carries
constexpr int kMaxDevices = 64;

struct NoallocScratch {
  TabMeta meta[EBAG_NOALLOC_MAX_TABLES];
  const void* tables[EBAG_NOALLOC_MAX_TABLES];
  int32_t tperm[EBAG_NOALLOC_MAX_TABLES];
  int32_t status[4];
  uint32_t ticket[2];
  uint32_t pad[2];
  uint32_t counters[EBAG_NOALLOC_MAX_FLAGS];
};
static_assert(sizeof(NoallocScratch) <= EBAG_NOALLOC_SCRATCH_BYTES, "scratch array too small");

}  // namespace
}  // namespace ebag

static __device__ __align__(256) unsigned char scratch[EBAG_NOALLOC_SCRATCH_BYTES];

namespace ebag {
namespace {

struct InstallArgs {
  NoallocScratch* s;   // the device's scratch array
  int32_t first;       // first table position this launch writes
  int32_t n;           // table positions this launch writes (<= kInstallTables)
  int32_t clear;       // 1: also zero counters [0, n_counters), the ticket and the status word
  int32_t n_counters;
  TabMeta meta[kInstallTables];
  const void* tables[kInstallTables];
  int32_t tperm[kInstallTables];
};

// Writes the descriptors of table positions [first, first + n) and, on the
// call's first launch, clears what the pooling kernel expects at zero.
__global__ __launch_bounds__(256) void install_kernel(const InstallArgs a) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i0 < a.n) {
    a.s->meta[a.first + i0] = a.meta[i0];
    a.s->tables[a.first + i0] = a.tables[i0];
    a.s->tperm[a.first + i0] = a.tperm[i0];
  }
  if (a.clear) {
    for (int64_t k = i0; k < a.n_counters; k += stride) a.s->counters[k] = 0u;
    if (i0 < 4) a.s->status[i0] = (i0 & 1) ? 0x7fffffff : 0;
    if (i0 < 2) a.s->ticket[i0] = 0u;
  }
}

std::mutex g_mu;
NoallocScratch* g_scratch[kMaxDevices];  // device address of `scratch`, per device
int g_cus[kMaxDevices];

// The calling device's scratch address and CU count, looked up on the first
// call made with that device current.
int device_scratch(int dev, NoallocScratch** out, int* cus) {
  if (dev < 0 || dev >= kMaxDevices) return fail(EBAG_EUNSUPPORTED, "device %d beyond the supported %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(EBAG_EHIP, "look up the scratch array on device %d: %s", dev, hipGetErrorString(e));
    // The host-side shadow is never a device address.
    if (p == static_cast<void*>(scratch))
      return fail(EBAG_EHIP, "scratch lookup on device %d returned the host shadow", dev);
    int n = 0;
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return fail(EBAG_EHIP, "CU count of device %d: %s", dev, hipGetErrorString(e));
    g_cus[dev] = n;
    g_scratch[dev] = static_cast<NoallocScratch*>(p);
  }
  *out = g_scratch[dev];
  *cus = g_cus[dev];
  return EBAG_OK;
}

int log2_vecs(int v) {
  for (int s = 0; s <= 6; ++s)
    if ((1 << s) == v) return s;
  return -1;
}

}  // namespace
}  // namespace ebag

using namespace ebag;

extern "C" int ebag_a2a_forward_noalloc(int32_t num_tables, const int64_t* rows_per_table,
                                        const int32_t* dim_per_table, int32_t table_dtype,
                                        int32_t chunk_samples, const ebag_a2a_opts_t* opts,
                                        const void* const* tables, const int32_t* indices, const int64_t* offsets,
                                        const float* weights, int64_t B, int32_t R, float* send_buf,
                                        uint32_t* flags, hipStream_t stream) {
  // Every argument is checked before the device is touched.
  if (num_tables <= 0 || num_tables > EBAG_NOALLOC_MAX_TABLES)
    return fail(EBAG_EINVAL, "num_tables=%d outside [1, %d]", num_tables, EBAG_NOALLOC_MAX_TABLES);
  if (!rows_per_table || !dim_per_table) return fail(EBAG_EINVAL, "null rows/dims array");
  if (table_dtype != EBAG_F32 && table_dtype != EBAG_F16 && table_dtype != EBAG_BF16)
    return fail(EBAG_EINVAL, "unknown table dtype %d", (int)table_dtype);
  if (chunk_samples <= 0) return fail(EBAG_EINVAL, "chunk_samples must be positive");
  ebag_a2a_opts_t o;
  if (opts)
    o = *opts;
  else
    ebag_a2a_default_opts(&o);
  int rc = check_opts(o);
  if (rc) return rc;
  if (o.trace || o.check_indices)
    return fail(EBAG_EUNSUPPORTED, "trace and check_indices need a plan (their results are read through it)");
  if (weights && o.pooling_mode == 1) return fail(EBAG_EINVAL, "mean pooling takes no weights");
  if (!tables) return fail(EBAG_EINVAL, "null table pointer array");
  if (!indices || !offsets || !send_buf || !flags) return fail(EBAG_EINVAL, "null indices, offsets, send_buf or flags");
  if (B <= 0 || R <= 0) return fail(EBAG_EINVAL, "B and R must be positive (B=%lld R=%d)", (long long)B, R);
  if (B % R != 0) return fail(EBAG_EINVAL, "B=%lld is not a multiple of R=%d", (long long)B, R);
  if ((B / R) % chunk_samples != 0)
    return fail(EBAG_EINVAL, "B/R=%lld is not a multiple of chunk_samples=%d", (long long)(B / R), chunk_samples);
  if (o.chunk_order == 1 && o.self_rank >= R)
    return fail(EBAG_EINVAL, "self_rank=%d is not a destination (R=%d)", o.self_rank, R);
  const int64_t n_chunks = B / chunk_samples;
  const int64_t n_flags = n_chunks * (o.slice_granule == 1 ? num_tables : 1);
  if (n_flags > EBAG_NOALLOC_MAX_FLAGS)
    return fail(EBAG_EINVAL, "%lld flags exceed the scratch array's %d slice counters", (long long)n_flags,
                EBAG_NOALLOC_MAX_FLAGS);
  if ((reinterpret_cast<uintptr_t>(send_buf) & 15u) != 0) return fail(EBAG_EINVAL, "send_buf is not 16-byte aligned");
  const int elt = table_dtype == EBAG_F32 ? 4 : 2;
  TabMeta meta[EBAG_NOALLOC_MAX_TABLES];
  int64_t widths[EBAG_NOALLOC_MAX_TABLES];
  int64_t sum_dim = 0;
  for (int32_t t = 0; t < num_tables; ++t) {
    const int64_t rows = rows_per_table[t];
    const int32_t D = dim_per_table[t];
    if (rows < 0 || rows > INT32_MAX) return fail(EBAG_EINVAL, "rows of table %d out of range", t);
    if (D <= 0) return fail(EBAG_EINVAL, "dim of table %d must be positive", t);
    if (((int64_t)D * elt) % 16 != 0)
      return fail(EBAG_EINVAL, "table %d: D*elt = %lld bytes is not a multiple of 16", t, (long long)D * elt);
    if (!tables[t] && rows > 0) return fail(EBAG_EINVAL, "null pointer for table %d", t);
    if ((reinterpret_cast<uintptr_t>(tables[t]) & 15u) != 0) return fail(EBAG_EINVAL, "table %d is not 16-byte aligned", t);
    meta[t].rows = rows;
    meta[t].row_bytes = (int64_t)D * elt;
    meta[t].dim = D;
    meta[t].col_off = (int32_t)sum_dim;
    meta[t].vecs = (int32_t)(meta[t].row_bytes / 16);
    meta[t].vshift = log2_vecs(meta[t].vecs);
    widths[t] = meta[t].row_bytes;
    sum_dim += D;
    if (sum_dim > INT32_MAX / 4) return fail(EBAG_EINVAL, "sum of dims too large");
  }

  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(EBAG_EHIP, "hipGetDevice failed");
  NoallocScratch* s = nullptr;
  int num_cus = 0;
  rc = device_scratch(dev, &s, &num_cus);
  if (rc) return rc;

  const int n_xcd = xcd_count(num_cus);
  int32_t tperm[EBAG_NOALLOC_MAX_TABLES], order_work[EBAG_NOALLOC_MAX_TABLES];
  int64_t order_load[kMaxXcd];
  table_order(widths, num_tables, n_xcd, tperm, order_work, order_load);

  PoolSetup ps;
  ps.o = &o;
  ps.meta = meta;
  ps.T = num_tables;
  ps.C = chunk_samples;
  ps.sum_dim = (int32_t)sum_dim;
  ps.dtype = (int32_t)table_dtype;
  ps.num_cus = num_cus;
  ps.table_groups = table_groups_for(o, num_tables, n_xcd);
  ps.d_tables = s->tables;
  ps.d_meta = s->meta;
  ps.d_tperm = s->tperm;
  ps.d_counters = s->counters;
  ps.d_status = s->status;
  ps.d_trace_release = nullptr;
  ps.d_ticket = s->ticket;
  SliceOrder so;
  so.n_chunks = n_chunks;
  so.per_rank = (B / R) / chunk_samples;
  so.self = o.self_rank;
  so.order = o.chunk_order;
  so.table_groups = ps.table_groups;
  PoolArgs a;
  fill_pool_args(ps, indices, offsets, weights, B, so, send_buf, flags, &a);
  if (a.nruns >= INT_MAX) return fail(EBAG_EINVAL, "too many runs (%lld) for one launch", (long long)a.nruns);
  const int block = 64 * o.waves_per_wg;
  const int grid = pool_grid(ps, a.nruns, true, weights != nullptr, block, a.out_floats);

  // Descriptors in batches of kInstallTables; the first launch also clears
  // the counters, ticket and status word (the previous call on this device
  // left them in whatever state it ended).
  for (int32_t first = 0; first < num_tables; first += kInstallTables) {
    InstallArgs ia;
    std::memset(&ia, 0, sizeof ia);
    ia.s = s;
    ia.first = first;
    ia.n = num_tables - first < kInstallTables ? num_tables - first : kInstallTables;
    ia.clear = first == 0;
    ia.n_counters = ia.clear ? (int32_t)n_flags : 0;
    for (int32_t i = 0; i < ia.n; ++i) {
      ia.meta[i] = meta[first + i];
      ia.tables[i] = tables[first + i];
      ia.tperm[i] = tperm[first + i];
    }
    const int64_t work = ia.n_counters > ia.n ? ia.n_counters : ia.n;
    int blocks = (int)((work + 255) / 256);
    blocks = blocks < 1 ? 1 : blocks > 256 ? 256 : blocks;
    hipLaunchKernelGGL(install_kernel, dim3(blocks), dim3(256), 0, stream, ia);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(EBAG_EHIP, "launch install kernel: %s", hipGetErrorString(e));
  }
  const hipError_t e = launch_pool(ps.dtype, o.rows_in_flight, weights != nullptr, true, needs_safe(ps), a, grid,
                                   block, stream);
  if (e != hipSuccess) return fail(EBAG_EHIP, "launch fused pooling kernel: %s", hipGetErrorString(e));
  return EBAG_OK;
}
