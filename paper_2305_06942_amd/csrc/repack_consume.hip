// Repack kernel of the unfused baseline and the flag-polling consumer.
#include "consume.h"

namespace ebag {
namespace {

// Unfused baseline, second kernel: one workgroup per (slice, table) copies
// the C pooled rows of table t from the per-table scratch [T][B][D_t] into
// the send layout [B][sum D] at columns [off_t, off_t + D_t) -- the repack a
// bulk-synchronous All-to-All needs between the pooling kernel and the
// collective (Sec. II-B, IV-A).
__global__ __launch_bounds__(256) void repack_kernel(const RepackArgs a) {
  const int64_t gs = blockIdx.x / a.T;
  const int tpos = (int)(blockIdx.x - gs * a.T);
  const int t = a.tperm[tpos];
  const int64_t g = slice_at(a.so, gs);
  const TabMeta m = a.meta[t];
  const int vpr = m.dim >> 2;  // float4 per row
  const int64_t b0 = g * a.C;
  const float4* src = reinterpret_cast<const float4*>(a.scratch + a.B * m.col_off + b0 * m.dim);
  float4* dst = reinterpret_cast<float4*>(a.send + b0 * a.sum_dim + m.col_off);
  const int ld4 = a.sum_dim >> 2;
  const int n = a.C * vpr;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int i = e / vpr;
    const int v = e - i * vpr;
    dst[(int64_t)i * ld4 + v] = src[e];
  }
}

// Unfused baseline, third step: after the repack kernel has ended (kernel
// boundary = all its stores visible device-wide), every flag is bumped at
// once -- the collective can only start once the whole batch is pooled.
__global__ __launch_bounds__(256) void publish_kernel(const PublishArgs a) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= a.n_flags) return;
  if (a.trace_release) a.trace_release[g] = wall_clock64();
  if (g != a.suppress) __hip_atomic_fetch_add(&a.flags[g], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef uint32_t u4v __attribute__((ext_vector_type(4)));
constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data format

// Wait until flag f reaches the epoch (relaxed device-scope loads with
// s_sleep back-off) or the wall-clock deadline passes.  Returns the value
// seen, or records the timeout and returns false in *ok.
__device__ __forceinline__ uint32_t wait_flag(const ConsumeArgs& a, int64_t f, uint64_t t0, bool* ok) {
  uint32_t v = __hip_atomic_load(&a.flags[f], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  bool timed_out = false;
  while ((int32_t)(v - a.epoch) < 0) {
    if (wall_clock64() - t0 > a.timeout_ticks) {
      timed_out = true;
      break;
    }
    __builtin_amdgcn_s_sleep(4);
    v = __hip_atomic_load(&a.flags[f], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  *ok = !__builtin_amdgcn_readfirstlane((int)timed_out);
  if (!*ok && threadIdx.x == 0) {
    __hip_atomic_store(&a.status[ST_TIMED_OUT], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    atomicMin(&a.status[ST_FIRST_MISSING], (int32_t)f);
  }
  return v;
}

// Cache policy bits of a buffer load: 16 = sc1 (device scope), 2 = nt.
__device__ __forceinline__ u4v load16(__amdgpu_buffer_rsrc_t rs, int off, bool coherent, bool nt) {
  if (coherent) return nt ? __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 18)
                          : __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 16);
  return nt ? __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 2) : __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
}

__device__ __forceinline__ void store16(u4v* p, const u4v& v, bool nt) {
  if (nt)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

// Receiver (Sec. III-A, "Book-keeping Flags").  Single-wave workgroups take
// work items in production order, so the slices that complete last are
// drained by many waves at once; each item waits for its flag, then copies
// its data from send to recv.  With coherent_loads the data is read with
// device-scope loads, which see the producer's device-scope stores without
// invalidating this XCD's L2; otherwise an agent-scope acquire precedes plain
// loads.
//   Whole-slice granule: an item is one 32 KiB piece of a slice's contiguous
//   C * sum(D) floats.
//   Per-table granule: an item is one (slice, table) pair: C rows of D_t
//   floats at columns off_t .. off_t + D_t, row stride sum(D).
__global__ __launch_bounds__(64) void consume_kernel(const ConsumeArgs a) {
  const int lane = threadIdx.x;
  const uint64_t t0 = wall_clock64();
  const int64_t per_slice = a.per_table ? a.T : a.pieces;
  const int64_t n_items = a.so.n_chunks * per_slice;
  const int64_t chunk_f4 = a.chunk_floats >> 2;
  for (int64_t x = blockIdx.x; x < n_items; x += gridDim.x) {
    int64_t gs, p;
    if (a.per_table) {  // (slice, table) items in production order
      int32_t tp, unused;
      run_at(a.so, a.T, 1, x, &gs, &tp, &unused);
      p = tp;
    } else {
      gs = x / per_slice;
      p = x - gs * per_slice;
    }
    const int64_t g = slice_at(a.so, gs);
    const int t = a.per_table ? __builtin_amdgcn_readfirstlane(a.tperm[p]) : 0;
    const int64_t f = a.per_table ? g * a.T + t : g;
    bool ok;
    const uint32_t v = wait_flag(a, f, t0, &ok);
    if (!ok) return;
    if (v != a.epoch && (a.per_table || p == 0) && lane == 0) atomicAdd(&a.status[ST_OVERSHOOT], 1);
    if (!a.coherent_loads) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    if (a.per_table) {
      // table constants are wave-uniform: keep them (and the descriptor) scalar
      const int dim = __builtin_amdgcn_readfirstlane(a.meta[t].dim);
      const int col_off = __builtin_amdgcn_readfirstlane(a.meta[t].col_off);
      const int v4 = dim >> 2;                         // float4s per row of this table
      const int64_t base = g * a.chunk_floats + col_off;
      const int n = a.C * v4;
      const int ld4 = a.sum_dim >> 2;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(a.send + base), 0, ((a.C - 1) * a.sum_dim + dim) * 4, kBufferWord3);
      float4* dst = reinterpret_cast<float4*>(a.recv + base);
      // Element e = i0 + 64 u + lane is float4 (e mod v4) of row e / v4; each
      // lane steps its (row, column) by 64 elements at a time, so the loop
      // divides once per item, and keeps 8 loads in flight.
      const int drow = 64 / v4, dcol = 64 - (64 / v4) * v4;
      int row = lane / v4, col = lane - (lane / v4) * v4;
      for (int i0 = 0; i0 < n; i0 += 8 * 64) {
        u4v r[8];
        int off[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          off[u] = i0 + u * 64 + lane < n ? row * ld4 + col : -1;
          r[u] = load16(rs, off[u] < 0 ? 0 : off[u] * 16, a.coherent_loads, a.nontemporal);
          row += drow;
          col += dcol;
          if (col >= v4) {
            col -= v4;
            ++row;
          }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (off[u] >= 0)
            store16(reinterpret_cast<u4v*>(dst) + off[u], r[u], a.nontemporal);
      }
    } else {
      const int64_t e0 = p * a.piece_f4;
      const int n = (int)min(a.piece_f4, chunk_f4 - e0);
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.send + g * a.chunk_floats + e0 * 4), 0, n * 16,
                                            kBufferWord3);
      float4* dst = reinterpret_cast<float4*>(a.recv + g * a.chunk_floats) + e0;
      for (int i0 = 0; i0 < n; i0 += 8 * 64) {
        u4v r[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) r[u] = load16(rs, (i0 + u * 64 + lane) * 16, a.coherent_loads, a.nontemporal);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = i0 + u * 64 + lane;
          if (i < n) store16(reinterpret_cast<u4v*>(dst) + i, r[u], a.nontemporal);
        }
      }
    }
    if (a.trace_drain && lane == 0) atomicMax(reinterpret_cast<unsigned long long*>(&a.trace_drain[f]),
                                              (unsigned long long)wall_clock64());
  }
}

}  // namespace

hipError_t launch_repack(const RepackArgs& a, int grid, int block, hipStream_t stream) {
  hipLaunchKernelGGL(repack_kernel, dim3(grid), dim3(block), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_publish(const PublishArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.n_flags + 255) / 256;
  hipLaunchKernelGGL(publish_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_consume(const ConsumeArgs& a, int grid, int block, hipStream_t stream) {
  hipLaunchKernelGGL(consume_kernel, dim3(grid), dim3(block), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ebag
