// Internal definitions shared by the host plan code and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ebag_a2a.h"

namespace ebag {

// Per-table constants, resident in device memory for the plan's lifetime.
struct TabMeta {
  int64_t rows;      // number of rows
  int64_t row_bytes; // D * elt (multiple of 16)
  int32_t dim;       // D
  int32_t col_off;   // first column of this table in a send-buffer row
  int32_t vecs;      // 16-byte vectors per row (= row_bytes / 16)
  int32_t vshift;    // log2(vecs) when vecs is a power of two <= 64, else -1
};

// Order in which slices are produced and drained.  order 0: natural; order
// 1: slices of destination `self` last, so slices bound for other
// destinations are finished (and can be shipped) first (Sec. III-A,
// communication-aware scheduling).  table_groups 0: runs go slice by slice,
// table positions fastest; G >= 1: table by table, slices (in the order
// above) inside a table, with run q taken by table group q mod G -- with G
// the number of XCDs, every XCD works through its own tables one at a time.
struct SliceOrder {
  int64_t n_chunks;    // B / C
  int64_t per_rank;    // (B / R) / C
  int64_t self;        // destination kept local
  int32_t order;
  int32_t table_groups;
};

__host__ __device__ inline int64_t slice_at(const SliceOrder& o, int64_t x) {
  if (o.order == 0) return x;
  const int64_t lo = o.self * o.per_rank;
  const int64_t others = o.n_chunks - o.per_rank;
  if (x < lo) return x;
  if (x < others) return x + o.per_rank;
  return lo + (x - others);
}

// Run q of a launch over n_chunks slices x T table positions x J runs per
// (slice, table) pair -> slice position gs (for slice_at), table position
// tpos, run j inside the pair.  Every q in [0, n_chunks * T * J) maps to a
// distinct triple; with table_groups G > 1, T is a multiple of G.
__host__ __device__ inline void run_at(const SliceOrder& o, int32_t T, int32_t J, int64_t q, int64_t* gs,
                                       int32_t* tpos, int32_t* j) {
  if (o.table_groups == 0) {
    const int64_t per_slice = (int64_t)T * J;
    *gs = q / per_slice;
    const int64_t rem = q - *gs * per_slice;
    *tpos = (int32_t)(rem % T);
    *j = (int32_t)(rem / T);
    return;
  }
  const int64_t G = o.table_groups;
  const int64_t per_table = o.n_chunks * J;
  const int64_t x = q % G, i = q / G;
  const int64_t k = i / per_table, r = i - k * per_table;
  *tpos = (int32_t)(k * G + x);
  *gs = r / J;
  *j = (int32_t)(r - *gs * J);
}

struct PoolArgs {
  const void* const* tables;  // [T] table base pointers
  const TabMeta* meta;        // [T]
  const int32_t* tperm;       // [T] position within a slice -> table
  const int32_t* indices;
  const int64_t* offsets;
  const float* weights;       // nullptr for plain sum
  float* out;                 // fused: send buffer; unfused: [T][B][D_t] scratch
  uint32_t* counters;         // [n_flags] bags finished per flag's slice (self-resetting)
  uint32_t* flags;            // [n_flags] epoch flags
  int32_t* status;            // plan status word
  uint64_t* trace_release;    // [n_flags] or nullptr
  uint32_t* ticket;           // [2] persistent grid: next run, workgroups done (self-resetting)
  int64_t B;
  int64_t nruns;
  int64_t suppress;           // flag index never released (-1: none)
  SliceOrder so;
  int32_t T;
  int32_t C;
  int32_t K;                  // bags per run
  int32_t J;                  // runs per (slice, table) = ceil(C / K)
  int32_t sum_dim;
  int32_t check;              // check offsets / indices
  int32_t release_mode;       // 0 agent-scope release fence, 1 device-scope stores + completion wait
  int32_t waves;              // wavefronts per workgroup (blockDim.x / 64)
  int32_t out_floats;         // LDS output buffer of the fast path: K x max dim
  int32_t stream_rows;        // 1: table rows loaded non-temporally
  int32_t mean;               // 1: mean pooling (sum / bag length)
  int32_t per_table;          // 1: one flag / counter per (slice, table), index g * T + t
};

// Host-side description of the plan behind a pooling launch: a plan from
// ebag_a2a_create, or one assembled per call by the plan-free forward.
struct PoolSetup {
  const ebag_a2a_opts_t* o;
  const TabMeta* meta;          // [T], host copy
  int32_t T;
  int32_t C;
  int32_t sum_dim;
  int32_t dtype;
  int32_t num_cus;
  int32_t table_groups;         // SliceOrder::table_groups under these options
  const void* const* d_tables;  // device arrays the kernels read and write
  const TabMeta* d_meta;
  const int32_t* d_tperm;
  uint32_t* d_counters;
  int32_t* d_status;
  uint64_t* d_trace_release;    // nullptr: no trace
  uint32_t* d_ticket;
};

// Host helpers shared by the plan and the plan-free forward (plan.hip).
constexpr int kMaxXcd = 64;
int check_opts(const ebag_a2a_opts_t& o);
int xcd_count(int num_cus);
int32_t table_groups_for(const ebag_a2a_opts_t& o, int32_t T, int n_xcd);
void table_order(const int64_t* row_bytes, int32_t T, int n_xcd, int32_t* perm, int32_t* work, int64_t* load);
bool needs_safe(const PoolSetup& s);
void fill_pool_args(const PoolSetup& s, const int32_t* indices, const int64_t* offsets, const float* weights,
                    int64_t B, const SliceOrder& so, float* out, uint32_t* flags, PoolArgs* a);
int pool_grid(const PoolSetup& s, int64_t nruns, bool fused, bool weighted, int block, int out_floats);

// Status word layout (int32[4]) and its initial value.
enum { ST_TIMED_OUT = 0, ST_FIRST_MISSING = 1, ST_OVERSHOOT = 2, ST_FIRST_BAD_BAG = 3 };
constexpr int32_t kStatusInit[4] = {0, 0x7fffffff, 0, 0x7fffffff};

// Error reporting shared by every entry point (thread-local message).
int fail(int code, const char* fmt, ...);
void clear_error();

// Launchers (return hipError_t of the launch).
hipError_t launch_pool(int dtype, int rows_in_flight, bool weighted, bool fused, bool safe, const PoolArgs& a,
                       int grid, int block, hipStream_t stream);
int pool_max_wgs_per_cu(int dtype, int rows_in_flight, bool weighted, bool fused, bool safe, int block,
                        int out_floats);

}  // namespace ebag
