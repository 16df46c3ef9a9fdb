// Embedding backward and the one-GPU gradient arrival: kernel arguments and
// launchers, shared by backward.hip and the host side.
#pragma once
#include "common.h"

namespace ebag {

// Embedding backward: gradient rows per lookup from the pooled gradient.
struct BackwardArgs {
  const float* grad;          // [B][sum D], the received pooled-output gradient
  const uint32_t* flags;      // per-slice epoch flags of the gradient, or nullptr (complete)
  float* values;              // per-lookup rows, table blocks in table order
  const int64_t* offsets;
  const float* weights;       // nullptr: unweighted
  const TabMeta* meta;
  const int32_t* tperm;
  const int64_t* value_base;  // [T + 1] first float of each table's block
  int32_t* status;
  int64_t B;
  int64_t nruns;
  uint64_t timeout_ticks;
  SliceOrder so;
  int32_t T;
  int32_t C;
  int32_t K;
  int32_t J;
  int32_t sum_dim;
  int32_t max_dim;
  int32_t per_table;
  int32_t mean;
  uint32_t epoch;
  int32_t pad;
};

// One-GPU stand-in for the gradient All-to-All's arrival.
struct DeliverArgs {
  const float* src;
  float* dst;
  uint32_t* flags;
  uint32_t* counters;         // [n_chunks] pieces stored per slice (self-resetting)
  const TabMeta* meta;
  const int32_t* tperm;
  int64_t chunk_floats;
  int64_t piece_f4;
  int64_t pieces;
  SliceOrder so;
  int32_t T;
  int32_t C;
  int32_t sum_dim;
  int32_t per_table;
};

hipError_t launch_backward(const BackwardArgs& a, int64_t* value_base, int block, size_t lds, hipStream_t stream);
hipError_t launch_deliver(const DeliverArgs& a, int grid, int block, hipStream_t stream);

}  // namespace ebag
