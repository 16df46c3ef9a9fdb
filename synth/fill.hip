// Device side of the seeded input generator: fills a table in place with the
// counter-based value function (SplitMix64, Steele/Lea/Flood 2014) so that
// 10^11-byte tables never cross PCIe, and two measurement kernels: a plain
// 16-byte copy (HBM bandwidth probe and byte-counter calibration for
// profiling) and a random-row read probe (the practical ceiling of a gather
// of rows of a given width).
//
// The value function must match synth/gen.py bit for bit:
//   u = splitmix64(seed ^ (row*dim + j)) >> 40
//   uniform: v = float(int(u) - 2^23) * 2^-24 * 0.1f   (two separate RNE ops)
//   cint:    v = float(int(u % 17) - 8)
// followed by round-to-nearest-even to fp16 / bf16 storage.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ float value_of(uint64_t seed, uint64_t e, int kind) {
  uint64_t u = splitmix64(seed ^ e) >> 40;
  if (kind == 0) {
    float x = (float)((int32_t)u - (1 << 23)) * 0x1p-24f;
    return __fmul_rn(x, 0.1f);
  }
  return (float)((int32_t)(u % 17u) - 8);
}

__device__ __forceinline__ uint16_t bf16_rne(float v) {
  uint32_t b = __float_as_uint(v);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

// One thread writes 8 consecutive elements (16 B for 16-bit, 32 B for fp32).
__global__ void fill_kernel(void* dst, uint64_t n_elems, uint64_t seed, int kind, int dtype) {
  uint64_t i0 = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8ull;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * 8ull;
  for (; i0 < n_elems; i0 += stride) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = value_of(seed, i0 + k, kind);
    if (i0 + 8 <= n_elems) {
      if (dtype == 0) {
        float4* p = reinterpret_cast<float4*>(static_cast<float*>(dst) + i0);
        p[0] = make_float4(v[0], v[1], v[2], v[3]);
        p[1] = make_float4(v[4], v[5], v[6], v[7]);
      } else {
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          uint16_t lo, hi;
          if (dtype == 1) {
            lo = __half_as_ushort(__float2half_rn(v[2 * k]));
            hi = __half_as_ushort(__float2half_rn(v[2 * k + 1]));
          } else {
            lo = bf16_rne(v[2 * k]);
            hi = bf16_rne(v[2 * k + 1]);
          }
          w[k] = (uint32_t)lo | ((uint32_t)hi << 16);
        }
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(dst) + i0) = make_uint4(w[0], w[1], w[2], w[3]);
      }
    } else {
      for (int k = 0; i0 + k < n_elems; ++k) {
        if (dtype == 0) static_cast<float*>(dst)[i0 + k] = v[k];
        else if (dtype == 1) static_cast<__half*>(dst)[i0 + k] = __float2half_rn(v[k]);
        else static_cast<uint16_t*>(dst)[i0 + k] = bf16_rne(v[k]);
      }
    }
  }
}

// Each thread moves 4 x 16 bytes per iteration (4 loads in flight, then 4
// stores); the grid strides over the buffer.
__global__ void copy_kernel(uint4* __restrict__ dst, const uint4* __restrict__ src, uint64_t n16) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    dst[i] = a;
    dst[i + stride] = b;
    dst[i + 2 * stride] = c;
    dst[i + 3 * stride] = d;
  }
  for (; i < n16; i += stride) dst[i] = src[i];
}

typedef uint32_t u4v __attribute__((ext_vector_type(4)));

// Random-row reads: every wave reads `steps` x (64 / lanes-per-row) rows of
// rb = 16 << lshift bytes at pseudo-random row numbers below nrows (16-byte
// loads, rb / 16 lanes per row, 8 loads in flight per lane) and folds them
// into one word per thread so the loads cannot be dropped.
template <bool NT>
__global__ __launch_bounds__(256) void gather_probe_kernel(const char* __restrict__ base, uint64_t nrows, int lshift,
                                                           int steps, uint32_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const uint64_t wave = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int sub = lane >> lshift;
  const uint64_t col = (uint64_t)(lane & ((1 << lshift) - 1)) * 16;
  const uint64_t rb = (uint64_t)16 << lshift;
  u4v acc = {0u, 0u, 0u, 0u};
  for (int s0 = 0; s0 < steps; s0 += 8) {
    u4v r[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint64_t row = splitmix64((wave << 32) ^ ((uint64_t)(s0 + u) << 8) ^ (uint64_t)sub) % nrows;
      const u4v* p = reinterpret_cast<const u4v*>(base + row * rb + col);
      r[u] = NT ? __builtin_nontemporal_load(p) : *p;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= r[u];
  }
  out[(uint64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

// Streaming reads: the grid walks base[0 : n16 * 16) in 16-byte vectors,
// thread i reading vectors i, i + stride, ... with 8 non-temporal loads in
// flight, folded into one word per thread so the loads cannot be dropped.
__global__ __launch_bounds__(256) void stream_read_kernel(const u4v* __restrict__ p, uint64_t n16,
                                                          uint32_t* __restrict__ out) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  u4v acc = {0u, 0u, 0u, 0u};
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u4v r[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) r[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= r[u];
  }
  for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(p + i);
  out[(uint64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

}  // namespace

extern "C" {

// Fill a rows x dim table with the counter-based values.  dtype 0 f32, 1 f16,
// 2 bf16; kind 0 uniform(-0.05, 0.05), 1 integers in [-8, 8].  Returns 0 or
// a hipError_t code.
int synth_fill(void* dst, int64_t rows, int32_t dim, int32_t dtype, uint64_t seed, int32_t kind,
               hipStream_t stream) {
  if (!dst || rows < 0 || dim <= 0 || dtype < 0 || dtype > 2 || kind < 0 || kind > 1) return -1;
  uint64_t n = (uint64_t)rows * (uint64_t)dim;
  if (n == 0) return 0;
  uint64_t threads = (n + 7) / 8;
  uint64_t blocks = (threads + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, dst, n, seed, kind, dtype);
  return (int)hipGetLastError();
}

// dst[0:bytes) = src[0:bytes); bytes must be a multiple of 16 and both
// pointers 16-byte aligned.  grid 0 = default.
int synth_copy(void* dst, const void* src, int64_t bytes, int32_t grid, hipStream_t stream) {
  if (!dst || !src || bytes < 0 || (bytes & 15) || ((uintptr_t)dst & 15) || ((uintptr_t)src & 15)) return -1;
  uint64_t n16 = (uint64_t)bytes / 16;
  if (n16 == 0) return 0;
  unsigned g = grid > 0 ? (unsigned)grid : 4096u;
  hipLaunchKernelGGL(copy_kernel, dim3(g), dim3(256), 0, stream, (uint4*)dst, (const uint4*)src, n16);
  return (int)hipGetLastError();
}

// Random-row read probe over base[0:bytes): grid workgroups of 256 threads,
// each wave reading steps x (1024 / row_bytes) rows of row_bytes (16..1024, a
// power of two) at pseudo-random positions; nt = 1 uses non-temporal loads.
// out: grid * 256 uint32 (device).  Bytes read = grid * 4 * steps * 1024.
int synth_gather_probe(const void* base, int64_t bytes, int32_t row_bytes, int32_t steps, int32_t grid, int32_t nt,
                       void* out, hipStream_t stream) {
  int lshift = 0;
  while ((16 << lshift) < row_bytes && lshift < 6) ++lshift;
  if (!base || !out || (16 << lshift) != row_bytes || bytes < row_bytes || steps <= 0 || steps % 8 || grid <= 0)
    return -1;
  const uint64_t nrows = (uint64_t)bytes / (uint64_t)row_bytes;
  if (nt)
    hipLaunchKernelGGL(gather_probe_kernel<true>, dim3(grid), dim3(256), 0, stream, (const char*)base, nrows, lshift,
                       steps, (uint32_t*)out);
  else
    hipLaunchKernelGGL(gather_probe_kernel<false>, dim3(grid), dim3(256), 0, stream, (const char*)base, nrows,
                       lshift, steps, (uint32_t*)out);
  return (int)hipGetLastError();
}

// Streaming read probe over base[0:bytes) (bytes a multiple of 16, base
// 16-byte aligned): grid workgroups of 256 threads.  out: grid * 256 uint32.
int synth_stream_read(const void* base, int64_t bytes, int32_t grid, void* out, hipStream_t stream) {
  if (!base || !out || bytes <= 0 || (bytes & 15) || ((uintptr_t)base & 15) || grid <= 0) return -1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(256), 0, stream, (const u4v*)base, (uint64_t)bytes / 16,
                     (uint32_t*)out);
  return (int)hipGetLastError();
}

}  // extern "C"
