// Embedding backward fused with the arrival of the gradient All-to-All, and
// the one-GPU stand-in for that arrival (the deliver kernel).
//
// The table owner receives the gradient of every pooled vector in the
// destination-partitioned layout grad[R][S][sum D] (= [B][sum D]), slice by
// slice.  The gradient of lookup k of bag (t, b) is w_k * grad[b][off_t ..
// off_t + D_t) (sum mode; w_k = 1 without weights) or grad[b][...] / L (mean
// mode).  Output: per table, in lookup order, nnz_t rows of D_t fp32 values;
// table blocks follow each other in table order.
//
// Runs are the forward's: up to K consecutive samples of one table inside
// one slice, numbered slice-major.  With flags, a workgroup waits for its
// slice's flag before touching the gradient, so slices are expanded as they
// arrive.  The workgroup scales its K gradient rows once into LDS (the
// mean's division happens there, once per element); the run's output rows
// are contiguous (consecutive bags' lookups follow each other), so the whole
// workgroup writes them as one block with 16-byte non-temporal stores,
// balanced however the bag lengths vary.
#include "backward.h"

namespace ebag {
namespace {

typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef float f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void wait_all_memory() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <class T>
__device__ __forceinline__ T sld(const T* p, int64_t i) {
  return ((const __attribute__((address_space(4))) T*)p)[i];
}

// First float of every table's output block: base[t] = sum over t' < t of
// nnz_t' * D_t', base[T] the total.  One workgroup of 256 threads: the
// tables' sizes are loaded 256 at a time (independent loads, one memory
// latency per 256 tables) and prefix-summed in LDS.
__global__ __launch_bounds__(256) void value_base_kernel(const int64_t* offsets, const TabMeta* meta, int32_t T,
                                                         int64_t B, int64_t* base) {
  __shared__ int64_t s_scan[256];
  const int tid = threadIdx.x;
  int64_t carry = 0;
  for (int32_t c0 = 0; c0 < T; c0 += 256) {
    const int32_t t = c0 + tid;
    const int64_t v = t < T ? (offsets[(int64_t)(t + 1) * B] - offsets[(int64_t)t * B]) * meta[t].dim : 0;
    s_scan[tid] = v;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {  // inclusive Hillis-Steele scan
      const int64_t add = tid >= d ? s_scan[tid - d] : 0;
      __syncthreads();
      s_scan[tid] += add;
      __syncthreads();
    }
    if (t < T) base[t] = carry + s_scan[tid] - v;
    carry += s_scan[255];
    __syncthreads();
  }
  if (tid == 0) base[T] = carry;
}

__global__ __launch_bounds__(1024) void backward_kernel(const BackwardArgs a) {
  // LDS: the run's K scaled gradient rows [K][dim], then its K + 1 bag
  // offsets relative to the run's first lookup.
  extern __shared__ f4v s_lds[];
  __shared__ int s_bad;
  const int tid = threadIdx.x;
  int64_t gs;
  int32_t tpos, j;
  run_at(a.so, a.T, a.J, blockIdx.x, &gs, &tpos, &j);
  const int t = sld(a.tperm, tpos);
  const int64_t g = slice_at(a.so, gs);
  if (a.flags) {
    if (tid == 0) {
      const int64_t f = a.per_table ? g * a.T + t : g;
      const uint64_t t0 = wall_clock64();
      int bad = 0;
      while ((int32_t)(__hip_atomic_load(&a.flags[f], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - a.epoch) < 0) {
        if (wall_clock64() - t0 > a.timeout_ticks) {
          __hip_atomic_store(&a.status[ST_TIMED_OUT], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          atomicMin(&a.status[ST_FIRST_MISSING], (int32_t)f);
          bad = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(4);
      }
      s_bad = bad;
    }
    __syncthreads();
    if (s_bad) return;
  }
  const int dim = sld(&a.meta[t].dim, 0);
  const int col_off = sld(&a.meta[t].col_off, 0);
  const int V = dim >> 2;  // float4 per row
  const int64_t b0 = g * a.C + (int64_t)j * a.K;
  const int nb = (int)min((int64_t)a.K, (g + 1) * (int64_t)a.C - b0);
  const int64_t obase = (int64_t)t * a.B + b0;
  const int64_t lo0 = sld(a.offsets, obase);
  int64_t* s_off = reinterpret_cast<int64_t*>(s_lds + (int64_t)a.K * (a.max_dim >> 2));
  if (tid <= nb) s_off[tid] = a.offsets[obase + tid] - lo0;
  // the run's gradient rows, scaled once (device-scope loads: with flags the
  // rows were stored by a kernel that may still be running)
  float* s_rows = reinterpret_cast<float*>(s_lds);
  for (int e = tid; e < nb * dim; e += blockDim.x) {
    const int k = e / dim;
    const int c = e - k * dim;
    const float* gp = a.grad + (b0 + k) * a.sum_dim + col_off + c;
    float v = a.flags ? __hip_atomic_load(const_cast<float*>(gp), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : *gp;
    if (a.mean) {
      const int64_t L = a.offsets[obase + k + 1] - a.offsets[obase + k];
      v = v / (float)L;
    }
    s_rows[k * dim + c] = v;
  }
  __syncthreads();
  // The run's output is one contiguous block of (lookups of its bags) x dim
  // floats; the whole workgroup streams it out.  Each thread walks float4
  // elements tid, tid + blockDim, ... keeping its (row, vector) position
  // incrementally (no division inside the loop) and the end of its current
  // bag in a register (LDS is read only when a bag boundary is crossed).
  // Four elements at a time: their LDS rows and weights are all requested
  // before the first store.
  const int64_t rows = s_off[nb];
  const int64_t n = rows * V;
  f4v* out = reinterpret_cast<f4v*>(a.values + sld(a.value_base, t) + (lo0 - sld(a.offsets, (int64_t)t * a.B)) * dim);
  const int step = blockDim.x;
  const int dk = step / V, dc = step - (step / V) * V;
  int64_t k = tid / V;
  int c = tid - (tid / V) * V;
  int bag = 0;
  int64_t bag_end = s_off[1];  // nb >= 1
  const float* wts = a.weights ? a.weights + lo0 : nullptr;
  constexpr int UB = 4;
  for (int64_t e0 = tid; e0 < n; e0 += (int64_t)UB * step) {
    f4v x[UB];
    float wv[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const bool in = e0 + (int64_t)u * step < n;
      // k < rows = s_off[nb] for every element in range, so the walk stops
      // at a bag below nb.
      if (in)
        while (k >= bag_end) bag_end = s_off[++bag + 1];
      x[u] = s_lds[bag * V + c];
      wv[u] = wts && in ? wts[k] : 1.f;
      k += dk;
      c += dc;
      if (c >= V) {
        c -= V;
        ++k;
      }
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      if (e0 + (int64_t)u * step < n) {
        const f4v y = wts ? wv[u] * x[u] : x[u];
        __builtin_nontemporal_store(y, out + e0 + (int64_t)u * step);
      }
    }
  }
}

// One-GPU stand-in for the gradient All-to-All's arrival: every wavefront
// copies work items (32 KiB pieces of a whole slice, or one (slice, table)
// block per item with per-table slices) from src to dst in slice order with
// device-scope stores, eight 16-byte loads in flight per lane; when the last
// piece of a slice is stored, its flag is incremented.  A few multi-wave
// workgroups keep the copy on a few CUs, so the backward it feeds keeps its
// occupancy everywhere else (a real arrival comes through the links and DMA
// engines and holds no CU at all).
constexpr int DU = 8;  // loads in flight per lane

__global__ __launch_bounds__(1024) void deliver_kernel(const DeliverArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t n_waves = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int64_t per_slice = a.per_table ? a.T : a.pieces;
  const int64_t n_items = a.so.n_chunks * per_slice;
  for (int64_t x = __builtin_amdgcn_readfirstlane(wave); x < n_items; x += n_waves) {
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
    if (a.per_table) {
      const int t = __builtin_amdgcn_readfirstlane(a.tperm[p]);
      const int dim = __builtin_amdgcn_readfirstlane(a.meta[t].dim);
      const int col_off = __builtin_amdgcn_readfirstlane(a.meta[t].col_off);
      const int v4 = dim >> 2, ld4 = a.sum_dim >> 2;
      const int n = a.C * v4;
      const int64_t base = g * a.chunk_floats + col_off;
      const float4* src = reinterpret_cast<const float4*>(a.src + base);
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          a.dst + base, 0, ((a.C - 1) * a.sum_dim + dim) * 4, 0x00020000);
      for (int e0 = 0; e0 < n; e0 += 64 * DU) {
        float4 v[DU];
        int off[DU];
#pragma unroll
        for (int u = 0; u < DU; ++u) {
          const int e = e0 + u * 64 + lane;
          const int row = e / v4;
          off[u] = e < n ? row * ld4 + (e - row * v4) : -1;
          v[u] = off[u] >= 0 ? src[off[u]] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < DU; ++u) {
          const u4v w = {__float_as_uint(v[u].x), __float_as_uint(v[u].y), __float_as_uint(v[u].z),
                         __float_as_uint(v[u].w)};
          if (off[u] >= 0) __builtin_amdgcn_raw_buffer_store_b128(w, rs, off[u] * 16, 0, 16);  // device scope
        }
      }
      wait_all_memory();
      if (lane == 0)
        __hip_atomic_fetch_add(&a.flags[g * a.T + t], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      const int64_t chunk_f4 = a.chunk_floats >> 2;
      const int64_t e0 = p * a.piece_f4;
      const int n = (int)min(a.piece_f4, chunk_f4 - e0);
      const float4* src = reinterpret_cast<const float4*>(a.src + g * a.chunk_floats) + e0;
      float4* dst = reinterpret_cast<float4*>(a.dst + g * a.chunk_floats) + e0;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(dst, 0, n * 16, 0x00020000);
      for (int i0 = 0; i0 < n; i0 += 64 * DU) {
        float4 v[DU];
#pragma unroll
        for (int u = 0; u < DU; ++u) {
          const int i = i0 + u * 64 + lane;
          v[u] = i < n ? src[i] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < DU; ++u) {
          const int i = i0 + u * 64 + lane;
          const u4v w = {__float_as_uint(v[u].x), __float_as_uint(v[u].y), __float_as_uint(v[u].z),
                         __float_as_uint(v[u].w)};
          if (i < n) __builtin_amdgcn_raw_buffer_store_b128(w, rs, i * 16, 0, 16);  // device scope
        }
      }
      wait_all_memory();
      if (lane == 0 &&
          __hip_atomic_fetch_add(&a.counters[g], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              (uint32_t)a.pieces - 1) {
        __hip_atomic_store(&a.counters[g], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(&a.flags[g], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

}  // namespace

hipError_t launch_backward(const BackwardArgs& a, int64_t* value_base, int block, size_t lds, hipStream_t stream) {
  hipLaunchKernelGGL(value_base_kernel, dim3(1), dim3(256), 0, stream, a.offsets, a.meta, a.T, a.B, value_base);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(backward_kernel, dim3((unsigned)a.nruns), dim3(block), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_deliver(const DeliverArgs& a, int grid, int block, hipStream_t stream) {
  hipLaunchKernelGGL(deliver_kernel, dim3(grid), dim3(block), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ebag
