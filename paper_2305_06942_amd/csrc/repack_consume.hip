// Repack kernel of the unfused baseline and the flag-polling consumer.
#include "common.h"

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
// boundary = all its stores visible device-wide), every slice flag is bumped
// at once -- the collective can only start once the whole batch is pooled.
__global__ __launch_bounds__(256) void publish_kernel(const PublishArgs a) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= a.n_chunks) return;
  if (a.trace_release) a.trace_release[g] = wall_clock64();
  if (g != a.suppress) __hip_atomic_fetch_add(&a.flags[g], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef uint32_t u4v __attribute__((ext_vector_type(4)));
constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data format

// Receiver (Sec. III-A, "Book-keeping Flags"): each slice is cut into pieces
// and the single-wave workgroups take pieces in production order, so the
// pieces of the slices that complete last are drained by many waves at once.
// A wave polls the slice flag (relaxed device-scope loads with s_sleep
// back-off, bounded by a wall-clock deadline), then copies its piece from
// send to recv.  With coherent_loads the piece is read with device-scope
// loads, which see the producer's device-scope stores without invalidating
// this XCD's L2; otherwise an agent-scope acquire precedes plain loads.
__global__ __launch_bounds__(64) void consume_kernel(const ConsumeArgs a) {
  const int lane = threadIdx.x;
  const uint64_t t0 = wall_clock64();
  const int64_t n_items = a.so.n_chunks * a.pieces;
  const int64_t chunk_f4 = a.chunk_floats >> 2;
  for (int64_t x = blockIdx.x; x < n_items; x += gridDim.x) {
    const int64_t gs = x / a.pieces;
    const int64_t p = x - gs * a.pieces;
    const int64_t g = slice_at(a.so, gs);
    uint32_t v = __hip_atomic_load(&a.flags[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bool timed_out = false;
    while ((int32_t)(v - a.epoch) < 0) {
      if (wall_clock64() - t0 > a.timeout_ticks) {
        timed_out = true;
        break;
      }
      __builtin_amdgcn_s_sleep(4);
      v = __hip_atomic_load(&a.flags[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (__builtin_amdgcn_readfirstlane((int)timed_out)) {
      if (lane == 0) {
        __hip_atomic_store(&a.status[ST_TIMED_OUT], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        atomicMin(&a.status[ST_FIRST_MISSING], (int32_t)g);
      }
      return;
    }
    if (v != a.epoch && p == 0 && lane == 0) atomicAdd(&a.status[ST_OVERSHOOT], 1);
    if (!a.coherent_loads) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int64_t e0 = p * a.piece_f4;
    const int n = (int)min(a.piece_f4, chunk_f4 - e0);
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.send + g * a.chunk_floats + e0 * 4), 0, n * 16,
                                          kBufferWord3);
    float4* dst = reinterpret_cast<float4*>(a.recv + g * a.chunk_floats) + e0;
    for (int i0 = 0; i0 < n; i0 += 8 * 64) {
      u4v r[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * 64 + lane;
        r[u] = a.coherent_loads ? __builtin_amdgcn_raw_buffer_load_b128(rs, i * 16, 0, 16)
                                : __builtin_amdgcn_raw_buffer_load_b128(rs, i * 16, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * 64 + lane;
        if (i < n) dst[i] = make_float4(__uint_as_float(r[u].x), __uint_as_float(r[u].y), __uint_as_float(r[u].z),
                                        __uint_as_float(r[u].w));
      }
    }
    if (a.trace_drain && lane == 0) atomicMax(reinterpret_cast<unsigned long long*>(&a.trace_drain[g]),
                                              (unsigned long long)wall_clock64());
  }
}

}  // namespace

hipError_t launch_repack(const RepackArgs& a, int grid, int block, hipStream_t stream) {
  hipLaunchKernelGGL(repack_kernel, dim3(grid), dim3(block), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_publish(const PublishArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.n_chunks + 255) / 256;
  hipLaunchKernelGGL(publish_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_consume(const ConsumeArgs& a, int grid, int block, hipStream_t stream) {
  hipLaunchKernelGGL(consume_kernel, dim3(grid), dim3(block), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ebag
