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

// Receiver: workgroup w owns slices w, w + grid, ... (in production order).
// For each: one lane polls the flag (relaxed loads, s_sleep back-off,
// bounded by a wall-clock deadline), then acquires and the whole workgroup
// copies the slice's C * sum(D) floats from send to recv.
__global__ __launch_bounds__(256) void consume_kernel(const ConsumeArgs a) {
  __shared__ int s_state;
  const uint64_t t0 = wall_clock64();
  const int64_t n4 = a.chunk_floats >> 2;
  for (int64_t x = blockIdx.x; x < a.so.n_chunks; x += gridDim.x) {
    const int64_t g = slice_at(a.so, x);
    if (threadIdx.x == 0) {
      int st = 0;
      uint32_t v = __hip_atomic_load(&a.flags[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      while ((int32_t)(v - a.epoch) < 0) {
        if (wall_clock64() - t0 > a.timeout_ticks) {
          st = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(4);
        v = __hip_atomic_load(&a.flags[g], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      if (st == 0) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        if (v != a.epoch) st = 2;
      }
      s_state = st;
    }
    __syncthreads();
    const int st = s_state;
    if (st == 1) {
      if (threadIdx.x == 0) {
        __hip_atomic_store(&a.status[ST_TIMED_OUT], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        atomicMin(&a.status[ST_FIRST_MISSING], (int32_t)g);
      }
      return;  // uniform: every thread read the same s_state
    }
    if (st == 2 && threadIdx.x == 0) atomicAdd(&a.status[ST_OVERSHOOT], 1);
    const float4* src = reinterpret_cast<const float4*>(a.send) + g * n4;
    float4* dst = reinterpret_cast<float4*>(a.recv) + g * n4;
    int64_t e = threadIdx.x;
    for (; e + 3 * (int64_t)blockDim.x < n4; e += 4 * (int64_t)blockDim.x) {
      const float4 x0 = src[e], x1 = src[e + blockDim.x], x2 = src[e + 2 * blockDim.x], x3 = src[e + 3 * blockDim.x];
      dst[e] = x0;
      dst[e + blockDim.x] = x1;
      dst[e + 2 * blockDim.x] = x2;
      dst[e + 3 * blockDim.x] = x3;
    }
    for (; e < n4; e += blockDim.x) dst[e] = src[e];
    __syncthreads();
    if (a.trace_drain && threadIdx.x == 0) a.trace_drain[g] = wall_clock64();
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
