// Unfused baseline's repack and publication, and the consumer: kernel
// arguments and launchers, shared by repack_consume.hip and the host side.
#pragma once
#include "common.h"

namespace ebag {

struct RepackArgs {
  const float* scratch;       // [T][B][D_t]
  float* send;                // [B][sum D]
  const TabMeta* meta;
  const int32_t* tperm;
  int64_t B;
  SliceOrder so;
  int32_t T;
  int32_t C;
  int32_t sum_dim;
  int32_t pad;
};

// Bulk-synchronous flag publication after the repack kernel.
struct PublishArgs {
  uint32_t* flags;
  uint64_t* trace_release;
  int64_t n_flags;
  int64_t suppress;
};

struct ConsumeArgs {
  const float* send;
  const uint32_t* flags;
  float* recv;
  int32_t* status;
  uint64_t* trace_drain;
  const TabMeta* meta;        // per-table slices: column range of each table
  const int32_t* tperm;       // per-table slices: production order of tables
  int64_t chunk_floats;       // C * sum D
  int64_t piece_f4;           // float4s per work item (whole-slice granule)
  int64_t pieces;             // work items per slice (whole-slice granule)
  uint64_t timeout_ticks;
  SliceOrder so;
  uint32_t epoch;
  int32_t coherent_loads;     // 1: device-scope loads of slice data (no cache invalidation)
  int32_t per_table;          // 1: one work item per (slice, table), flag g * T + t
  int32_t T;
  int32_t C;
  int32_t sum_dim;
  int32_t nontemporal;        // 1: slice data read and written non-temporally
};

hipError_t launch_repack(const RepackArgs& a, int grid, int block, hipStream_t stream);
hipError_t launch_publish(const PublishArgs& a, hipStream_t stream);
hipError_t launch_consume(const ConsumeArgs& a, int grid, int block, hipStream_t stream);

}  // namespace ebag
