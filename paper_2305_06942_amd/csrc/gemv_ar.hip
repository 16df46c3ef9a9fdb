// Fused GEMV + AllReduce (Sec. III-B) for gfx950, and its bulk-synchronous
// baseline; the C ABI is declared in include/gemv_ar.h.
//
// GEMV: a wave computes rows of its tile; for a row, lane l takes the 16-byte
// vectors l, l + 64, ... of the row (coalesced non-temporal loads -- the
// matrix is read once --, UJ per lane and row in flight, RPI rows at a time)
// and the matching vectors of x from LDS, where the
// workgroup staged its rank's x once.  Products are accumulated in fp32 per
// lane and combined with xor shuffles.
//
// AllReduce (fused), two-phase direct: workgroup (r, p) stores its partial
// tiles for owner q into the reduction slots part[r][rows] with device-scope
// stores and waits for them to complete.  Then either
//  - owner-waits mode (the paper's scheme, cooperative launch): it sets peer
//    flag (q, r, p) to the forward's epoch, and owner workgroup (q, p) polls
//    the flags of (s, p) for every s != q before reducing; or
//  - last-arriver mode (default): it counts itself in on counter (q, p), and
//    the workgroup completing the count reduces.
// The reduction sums part[0..R-1][rows] in rank order with device-scope loads
// and stores the result into every rank's output.
#include <climits>
#include <cstring>
#include <new>
#include <vector>

#include "common.h"
#include "device_guard.h"
#include "gemv_ar.h"

namespace ebag {
namespace {

constexpr int kMaxRanks = 16;
constexpr int UJ = 4;             // 16-byte loads in flight per lane per row
constexpr int RPI = 4;            // rows a wave works on at once (RPI * UJ loads in flight per lane)
constexpr int kMaxXBytes = 64 * 1024;

typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u4v gu4v;

struct GemvArgs {
  const char* A[kMaxRanks];
  const char* x[kMaxRanks];
  float* y[kMaxRanks];
  int64_t K[kMaxRanks];
  float* part;           // [R][M] partial vectors (the owners' reduction slots)
  uint32_t* peer;        // [R owner][R source][P] epoch flags (owner-waits mode)
  uint32_t* cnt;         // [R owner][P] arrival counters (last-arriver mode, self-resetting)
  uint32_t* out_flags;   // [R][P] or nullptr
  int32_t* status;       // [2]: timed out, first missing peer flag
  int64_t M;
  int64_t n_tiles;
  int64_t suppress;
  uint64_t timeout_ticks;
  uint32_t epoch;
  int32_t R;
  int32_t P;
  int32_t TM;
  int32_t comm_aware;
  int32_t pad;
};

// 16-byte vector of the storage type -> fp32 values.
template <int DT> struct Vec;
template <> struct Vec<0> {  // fp32
  static constexpr int N = 4;
  static __device__ __forceinline__ void widen(const u4v& r, float* f) {
    f[0] = __uint_as_float(r.x); f[1] = __uint_as_float(r.y); f[2] = __uint_as_float(r.z); f[3] = __uint_as_float(r.w);
  }
};
template <> struct Vec<1> {  // fp16
  static constexpr int N = 8;
  static __device__ __forceinline__ void widen(const u4v& r, float* f) {
    const uint32_t u[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = (float)__builtin_bit_cast(_Float16, (uint16_t)(u[e] & 0xffffu));
      f[2 * e + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(u[e] >> 16));
    }
  }
};
template <> struct Vec<2> {  // bf16
  static constexpr int N = 8;
  static __device__ __forceinline__ void widen(const u4v& r, float* f) {
    const uint32_t u[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = __uint_as_float(u[e] << 16);
      f[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
  }
};

template <int DT>
__device__ __forceinline__ float dot16(const u4v& a, const u4v& x) {
  float fa[Vec<DT>::N], fx[Vec<DT>::N];
  Vec<DT>::widen(a, fa);
  Vec<DT>::widen(x, fx);
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < Vec<DT>::N; ++e) s = __builtin_fmaf(fa[e], fx[e], s);
  return s;
}

__device__ __forceinline__ void store_f32(float* p, float v, bool device_scope) {
  if (device_scope)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}

__device__ __forceinline__ float load_f32_device(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// s_waitcnt vmcnt(0): every memory operation of this wave has completed.
__device__ __forceinline__ void wait_all_memory() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Stage x_r (K * elt bytes, a multiple of 16) into LDS.
__device__ __forceinline__ void stage_x(const char* x, int64_t bytes, u4v* lds_x) {
  for (int64_t v = threadIdx.x; v * 16 < bytes; v += blockDim.x) lds_x[v] = *(gu4v*)(x + v * 16);
}

// Partial product of rank r for the rows of tile `tile`, stored into
// part[r][rows] (device-scope stores when `device_scope`).
template <int DT>
__device__ void partial_tile(const GemvArgs& a, int r, int64_t tile, const u4v* lds_x, bool device_scope) {
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int W = blockDim.x >> 6;
  const int64_t row0 = tile * a.TM;
  const int nrows = (int)min((int64_t)a.TM, a.M - row0);
  const int per = (nrows + W - 1) / W;
  const int r0 = wid * per;
  const int r1 = min(r0 + per, nrows);
  const int64_t K = a.K[r];
  const int64_t row_bytes = K * (DT == 0 ? 4 : 2);
  const int V = (int)(row_bytes / 16);
  const char* Ar = a.A[r];
  float* out = a.part + (int64_t)r * a.M + row0;
  for (int base = r0; base < r1; base += 64) {  // results of up to 64 rows per store
    float res = 0.f;
    const int nb = min(64, r1 - base);
    for (int k = 0; k < nb; k += RPI) {
      const char* pr[RPI];
      bool has[RPI];
#pragma unroll
      for (int j = 0; j < RPI; ++j) {
        has[j] = k + j < nb;
        pr[j] = Ar + (row0 + base + k + (has[j] ? j : 0)) * row_bytes;
      }
      float acc[RPI];
#pragma unroll
      for (int j = 0; j < RPI; ++j) acc[j] = 0.f;
      for (int v0 = 0; v0 < V; v0 += 64 * UJ) {
        u4v ra[RPI][UJ];
#pragma unroll
        for (int u = 0; u < UJ; ++u) {
          const int v = v0 + u * 64 + lane;
#pragma unroll
          for (int j = 0; j < RPI; ++j) {
            ra[j][u] = u4v{0u, 0u, 0u, 0u};
            if (v < V && has[j]) ra[j][u] = __builtin_nontemporal_load((gu4v*)(pr[j] + (int64_t)v * 16));
          }
        }
#pragma unroll
        for (int u = 0; u < UJ; ++u) {
          const int v = v0 + u * 64 + lane;
          if (v < V) {
            const u4v xv = lds_x[v];
#pragma unroll
            for (int j = 0; j < RPI; ++j) acc[j] += dot16<DT>(ra[j][u], xv);
          }
        }
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
#pragma unroll
        for (int j = 0; j < RPI; ++j) acc[j] += __shfl_xor(acc[j], m);
      }
#pragma unroll
      for (int j = 0; j < RPI; ++j)
        if (has[j] && lane == k + j) res = acc[j];
    }
    if (lane < nb) store_f32(out + base + lane, res, device_scope);
  }
}

// First tile of the owner block [t0, t1) that physical workgroup p handles.
__device__ __forceinline__ int64_t first_tile(int64_t t0, int p, int P) {
  const int64_t m = t0 % P;
  return t0 + ((p - m) % P + P) % P;
}

// Tiles owned by rank q: [ceil(q * n / R), ceil((q + 1) * n / R)).
__device__ __forceinline__ int64_t owner_begin(int64_t n, int q, int R) { return (q * n + R - 1) / R; }

// Sum the R partials of owner q's tiles handled by workgroup p (rank order,
// device-scope loads) and store the result into every rank's output.
__device__ void reduce_owned(const GemvArgs& a, int q, int p) {
  const int64_t t0 = owner_begin(a.n_tiles, q, a.R), t1 = owner_begin(a.n_tiles, q + 1, a.R);
  for (int64_t i = first_tile(t0, p, a.P); i < t1; i += a.P) {
    const int64_t row0 = i * a.TM;
    const int nrows = (int)min((int64_t)a.TM, a.M - row0);
    for (int k = threadIdx.x; k < nrows; k += blockDim.x) {
      float sum = 0.f;
      for (int s = 0; s < a.R; ++s) sum += load_f32_device(a.part + (int64_t)s * a.M + row0 + k);
      for (int r = 0; r < a.R; ++r) store_f32(a.y[r] + row0 + k, sum, true);
    }
  }
}

// Fused kernel, last-arriver reduction (default): workgroup (r, p) computes
// its partial tiles owner by owner; after each owner's tiles are stored it
// counts itself in on that owner's counter (q, p), and the workgroup that
// completes the count -- the last of the R ranks to deliver -- reduces and
// broadcasts the owner's tiles, then re-arms the counter.  Nobody waits, so
// the grid needs no co-residency and launches normally.
template <int DT>
__global__ __launch_bounds__(1024) void gemv_ar_last_arriver_kernel(const GemvArgs a) {
  extern __shared__ u4v lds_x[];
  __shared__ uint32_t s_old;
  const int r = blockIdx.x / a.P;
  const int p = blockIdx.x - r * a.P;
  stage_x(a.x[r], a.K[r] * (DT == 0 ? 4 : 2), lds_x);
  __syncthreads();
  for (int qi = 0; qi < a.R; ++qi) {
    const int q = a.comm_aware ? (r + 1 + qi) % a.R : qi;
    const int64_t t0 = owner_begin(a.n_tiles, q, a.R), t1 = owner_begin(a.n_tiles, q + 1, a.R);
    const int64_t i0 = first_tile(t0, p, a.P);
    if (i0 >= t1) {
      // No tile of owner q for workgroup p (on every rank alike): the owner's
      // own workgroup advances the output flag, which has nothing to cover.
      if (q == r && a.out_flags && threadIdx.x == 0)
        __hip_atomic_fetch_add(&a.out_flags[(int64_t)q * a.P + p], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      continue;
    }
    for (int64_t i = i0; i < t1; i += a.P) partial_tile<DT>(a, r, i, lds_x, true);
    // every wave's partial stores complete (device scope) before counting in
    wait_all_memory();
    __syncthreads();
    uint32_t* c = &a.cnt[(int64_t)q * a.P + p];
    if (threadIdx.x == 0) s_old = __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (s_old == (uint32_t)a.R - 1) {
      reduce_owned(a, q, p);
      wait_all_memory();
      __syncthreads();
      if (threadIdx.x == 0) {
        __hip_atomic_store(c, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (a.out_flags)
          __hip_atomic_fetch_add(&a.out_flags[(int64_t)q * a.P + p], 1u, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __syncthreads();  // s_old is rewritten for the next owner
  }
}

template <int DT>
__global__ __launch_bounds__(1024) void gemv_ar_fused_kernel(const GemvArgs a) {
  extern __shared__ u4v lds_x[];
  __shared__ int s_bad;
  const int r = blockIdx.x / a.P;
  const int p = blockIdx.x - r * a.P;
  stage_x(a.x[r], a.K[r] * (DT == 0 ? 4 : 2), lds_x);
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();
  // Phase 1: partial tiles, other owners first (comm-aware) or in owner order.
  for (int qi = 0; qi < a.R; ++qi) {
    const int q = a.comm_aware ? (r + 1 + qi) % a.R : qi;
    const int64_t t0 = owner_begin(a.n_tiles, q, a.R), t1 = owner_begin(a.n_tiles, q + 1, a.R);
    for (int64_t i = first_tile(t0, p, a.P); i < t1; i += a.P) partial_tile<DT>(a, r, i, lds_x, true);
    if (q != r) {
      // every wave's partial stores done (device scope) before the flag
      wait_all_memory();
      __syncthreads();
      const int64_t f = ((int64_t)q * a.R + r) * a.P + p;
      if (threadIdx.x == 0 && f != a.suppress)
        __hip_atomic_store(&a.peer[f], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  wait_all_memory();
  __syncthreads();
  // Phase 2: as owner, wait for the partials of workgroup p of every rank.
  if (threadIdx.x == 0) {
    const uint64_t t0 = wall_clock64();
    for (int s = 0; s < a.R && !s_bad; ++s) {
      if (s == r) continue;
      const int64_t f = ((int64_t)r * a.R + s) * a.P + p;
      while (__hip_atomic_load(&a.peer[f], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != a.epoch) {
        if (wall_clock64() - t0 > a.timeout_ticks) {
          __hip_atomic_store(&a.status[0], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          atomicMin(&a.status[1], (int32_t)f);
          s_bad = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
  }
  __syncthreads();
  if (s_bad) return;
  // Reduce the owned tiles in rank order and store them to every rank.
  reduce_owned(a, r, p);
  if (a.out_flags) {
    wait_all_memory();
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_add(&a.out_flags[(int64_t)r * a.P + p], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Baseline, first kernel: one workgroup per (rank, tile).
template <int DT>
__global__ __launch_bounds__(1024) void gemv_partial_kernel(const GemvArgs a) {
  extern __shared__ u4v lds_x[];
  const int r = blockIdx.x / a.n_tiles;
  const int64_t tile = blockIdx.x - (int64_t)r * a.n_tiles;
  stage_x(a.x[r], a.K[r] * (DT == 0 ? 4 : 2), lds_x);
  __syncthreads();
  partial_tile<DT>(a, r, tile, lds_x, false);
}

// Baseline, second kernel: the AllReduce after the kernel boundary -- every
// output row is the rank-order sum of the partials, stored to every rank.
__global__ __launch_bounds__(256) void allreduce_kernel(const GemvArgs a) {
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= a.M) return;
  float sum = 0.f;
  for (int s = 0; s < a.R; ++s) sum += a.part[(int64_t)s * a.M + row];
  for (int q = 0; q < a.R; ++q) a.y[q][row] = sum;
}

__global__ __launch_bounds__(256) void bump_flags_kernel(uint32_t* flags, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) __hip_atomic_fetch_add(&flags[i], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef void (*gemv_fn)(const GemvArgs);

gemv_fn fused_fn(int dt) {
  return dt == 0 ? gemv_ar_fused_kernel<0> : dt == 1 ? gemv_ar_fused_kernel<1> : gemv_ar_fused_kernel<2>;
}
gemv_fn last_arriver_fn(int dt) {
  return dt == 0 ? gemv_ar_last_arriver_kernel<0>
                 : dt == 1 ? gemv_ar_last_arriver_kernel<1> : gemv_ar_last_arriver_kernel<2>;
}
gemv_fn partial_fn(int dt) {
  return dt == 0 ? gemv_partial_kernel<0> : dt == 1 ? gemv_partial_kernel<1> : gemv_partial_kernel<2>;
}

}  // namespace
}  // namespace ebag

using namespace ebag;

struct gemv_ar_plan {
  int device = 0;
  int32_t R = 0;
  int64_t M = 0;
  int dtype = 0;
  int elt = 4;
  int64_t K[kMaxRanks] = {};
  int64_t max_x_bytes = 0;
  int num_cus = 0;
  double ticks_per_us = 100.0;
  gemv_ar_opts_t opts{};
  int64_t n_tiles = 0;
  int32_t P = 0;
  int32_t block = 0;
  int32_t resident = 0;  // workgroups the device holds at once for the fused kernel
  uint32_t epoch = 0;
  // The last forward's completion, for refusing a forward on another stream
  // while it still runs (the reduction slots and counters are shared).
  hipEvent_t fwd_done = nullptr;
  hipStream_t fwd_stream = nullptr;
  bool fwd_pending = false;
  float* d_part = nullptr;
  uint32_t* d_peer = nullptr;
  uint32_t* d_cnt = nullptr;
  int32_t* d_status = nullptr;
};

namespace {

const int32_t kGemvStatusInit[2] = {0, INT_MAX};

void free_gemv(gemv_ar_plan* h) {
  if (!h) return;
  if (h->fwd_done) (void)hipEventDestroy(h->fwd_done);
  (void)hipFree(h->d_part);
  (void)hipFree(h->d_peer);
  (void)hipFree(h->d_cnt);
  (void)hipFree(h->d_status);
  delete h;
}

int hipf(hipError_t e, const char* what) { return fail(EBAG_EHIP, "%s: %s", what, hipGetErrorString(e)); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  return hipStreamIsCapturing(stream, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone;
}

// One forward in flight per plan: a forward on another stream than the last
// one, while the last one has not completed, would share its reduction slots
// and arrival counters.
int check_busy(gemv_ar_plan* h, hipStream_t stream) {
  if (!h->fwd_pending || stream == h->fwd_stream || capturing(stream)) return EBAG_OK;
  const hipError_t e = hipEventQuery(h->fwd_done);
  if (e == hipErrorNotReady)
    return fail(EBAG_EBUSY, "a forward of this plan is still running on another stream (the reduction slots and "
                            "counters are shared): order the forwards on one stream or wait for it");
  if (e != hipSuccess) return hipf(e, "query the last forward");
  h->fwd_pending = false;
  return EBAG_OK;
}

// Remember the forward just enqueued on `stream` (not under graph capture).
int note_forward(gemv_ar_plan* h, hipStream_t stream) {
  if (capturing(stream)) {
    h->fwd_pending = false;
    return EBAG_OK;
  }
  const hipError_t e = hipEventRecord(h->fwd_done, stream);
  if (e != hipSuccess) return hipf(e, "record the forward's completion");
  h->fwd_stream = stream;
  h->fwd_pending = true;
  return EBAG_OK;
}

int fill_args(gemv_ar_plan* h, const void* const* A, const void* const* x, float* const* y, uint32_t* out_flags,
              GemvArgs* a) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != h->device)
    return fail(EBAG_EINVAL, "the plan belongs to device %d, but device %d is current", h->device, dev);
  if (!A || !x || !y) return fail(EBAG_EINVAL, "null A, x or y pointer array");
  std::memset(a, 0, sizeof *a);
  for (int r = 0; r < h->R; ++r) {
    if (!A[r] || !x[r] || !y[r]) return fail(EBAG_EINVAL, "null A, x or y for rank %d", r);
    if (!aligned16(A[r]) || !aligned16(x[r])) return fail(EBAG_EINVAL, "A or x of rank %d not 16-byte aligned", r);
    a->A[r] = static_cast<const char*>(A[r]);
    a->x[r] = static_cast<const char*>(x[r]);
    a->y[r] = y[r];
    a->K[r] = h->K[r];
  }
  a->part = h->d_part;
  a->peer = h->d_peer;
  a->cnt = h->d_cnt;
  a->out_flags = out_flags;
  a->status = h->d_status;
  a->M = h->M;
  a->n_tiles = h->n_tiles;
  a->suppress = h->opts.debug_suppress_flag;
  a->timeout_ticks = (uint64_t)((double)h->opts.timeout_us * h->ticks_per_us);
  a->R = h->R;
  a->P = h->P;
  a->TM = h->opts.tile_rows;
  a->comm_aware = h->opts.comm_aware;
  return EBAG_OK;
}

}  // namespace

extern "C" {

int gemv_ar_default_opts(gemv_ar_opts_t* o) {
  if (!o) return fail(EBAG_EINVAL, "null opts");
  std::memset(o, 0, sizeof *o);
  o->tile_rows = 0;
  o->wgs_per_rank = 0;
  o->waves_per_wg = 2;
  o->comm_aware = 1;
  o->debug_suppress_flag = -1;
  o->reduce_mode = 0;
  o->timeout_us = 5000000;
  return EBAG_OK;
}

int gemv_ar_create(gemv_ar_t* out, int32_t R, int64_t M, const int64_t* K, int32_t dtype,
                   const gemv_ar_opts_t* opts) {
  if (!out) return fail(EBAG_EINVAL, "null output handle");
  *out = nullptr;
  if (R < 1 || R > kMaxRanks) return fail(EBAG_EINVAL, "R=%d outside [1, %d]", R, kMaxRanks);
  if (M < 1 || M > INT_MAX) return fail(EBAG_EINVAL, "M=%lld outside [1, 2^31)", (long long)M);
  if (!K) return fail(EBAG_EINVAL, "null K array");
  if (dtype != EBAG_F32 && dtype != EBAG_F16 && dtype != EBAG_BF16) return fail(EBAG_EINVAL, "bad dtype %d", (int)dtype);
  gemv_ar_opts_t o;
  if (opts) o = *opts; else gemv_ar_default_opts(&o);
  if (o.tile_rows < 0 || o.tile_rows > 4096) return fail(EBAG_EINVAL, "tile_rows must be 0 (auto) or in [1, 4096]");
  if (o.tile_rows == 0) {
    // 128-row tiles, halved (down to 64) until the R ranks hold at least
    // 2048 tiles: with about 1024 workgroups (below), each then computes two
    // or more tiles, and the reduction that follows its first tile overlaps
    // the GEMV of its next one instead of all waiting at the kernel's end.
    o.tile_rows = 128;
    while (o.tile_rows > 64 && (int64_t)R * ((M + o.tile_rows - 1) / o.tile_rows) < 2048) o.tile_rows /= 2;
  }
  if (o.waves_per_wg < 1 || o.waves_per_wg > 16) return fail(EBAG_EINVAL, "waves_per_wg must be in [1, 16]");
  if (o.wgs_per_rank < 0) return fail(EBAG_EINVAL, "wgs_per_rank must be >= 0");
  if (o.comm_aware != 0 && o.comm_aware != 1) return fail(EBAG_EINVAL, "comm_aware must be 0 or 1");
  if (o.reduce_mode != 0 && o.reduce_mode != 1) return fail(EBAG_EINVAL, "reduce_mode must be 0 or 1");
  if (o.timeout_us < 1) return fail(EBAG_EINVAL, "timeout_us must be >= 1");
  const int elt = dtype == EBAG_F32 ? 4 : 2;
  int64_t max_x = 0;
  for (int r = 0; r < R; ++r) {
    if (K[r] < 1) return fail(EBAG_EINVAL, "K[%d]=%lld must be positive", r, (long long)K[r]);
    if ((K[r] * elt) % 16) return fail(EBAG_EINVAL, "K[%d] * element size is not a multiple of 16 bytes", r);
    if (K[r] * elt > kMaxXBytes)
      return fail(EBAG_EUNSUPPORTED, "K[%d] * element size above %d bytes (x is staged in LDS)", r, kMaxXBytes);
    if (K[r] * elt > max_x) max_x = K[r] * elt;
  }
  gemv_ar_plan* h = new (std::nothrow) gemv_ar_plan();
  if (!h) return fail(EBAG_ENOMEM, "host allocation failed");
  h->R = R;
  h->M = M;
  h->dtype = (int)dtype;
  h->elt = elt;
  for (int r = 0; r < R; ++r) h->K[r] = K[r];
  h->max_x_bytes = max_x;
  h->opts = o;
  h->n_tiles = (M + o.tile_rows - 1) / o.tile_rows;
  h->block = 64 * o.waves_per_wg;
  hipError_t e = hipGetDevice(&h->device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&h->num_cus, hipDeviceAttributeMultiprocessorCount, h->device);
  int khz = 0;
  if (e == hipSuccess && hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->device) == hipSuccess &&
      khz > 0)
    h->ticks_per_us = khz / 1000.0;
  const bool owner_mode = o.reduce_mode == 1;
  int per_cu = 0;
  if (e == hipSuccess)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, owner_mode ? fused_fn(h->dtype) : last_arriver_fn(h->dtype), h->block, (size_t)max_x);
  if (e != hipSuccess) {
    free_gemv(h);
    return hipf(e, "query device");
  }
  h->resident = per_cu * h->num_cus;
  // Owner-waits mode needs every workgroup resident (cooperative launch);
  // the last-arriver mode does not and defaults to about 1024 workgroups in
  // all (at most one tile each): one resident wave on 256 CUs.
  int64_t P = o.wgs_per_rank > 0 ? o.wgs_per_rank : owner_mode ? h->resident / R : (1024 + R - 1) / R;
  if (P > h->n_tiles) P = h->n_tiles;
  if (P * R > INT_MAX) P = INT_MAX / R;
  if (P < 1 || (owner_mode && P * R > h->resident)) {
    const int rc = fail(EBAG_EUNSUPPORTED, "%lld workgroups per rank x %d ranks cannot all be resident (%d fit)",
                        (long long)P, R, h->resident);
    free_gemv(h);
    return rc;
  }
  h->P = (int32_t)P;
#define GEMV_TRY(call, what)        \
  do {                              \
    hipError_t e_ = (call);         \
    if (e_ != hipSuccess) {         \
      const int r_ = hipf(e_, what); \
      free_gemv(h);                 \
      return r_;                    \
    }                               \
  } while (0)
  GEMV_TRY(hipMalloc((void**)&h->d_part, sizeof(float) * (size_t)R * (size_t)M), "alloc reduction slots");
  GEMV_TRY(hipMalloc((void**)&h->d_peer, sizeof(uint32_t) * (size_t)R * R * P), "alloc peer flags");
  GEMV_TRY(hipMemset(h->d_peer, 0, sizeof(uint32_t) * (size_t)R * R * P), "zero peer flags");
  GEMV_TRY(hipMalloc((void**)&h->d_cnt, sizeof(uint32_t) * (size_t)R * P), "alloc arrival counters");
  GEMV_TRY(hipMemset(h->d_cnt, 0, sizeof(uint32_t) * (size_t)R * P), "zero arrival counters");
  GEMV_TRY(hipMalloc((void**)&h->d_status, sizeof(kGemvStatusInit)), "alloc status");
  GEMV_TRY(hipMemcpy(h->d_status, kGemvStatusInit, sizeof(kGemvStatusInit), hipMemcpyHostToDevice), "init status");
  GEMV_TRY(hipEventCreateWithFlags(&h->fwd_done, hipEventDisableTiming), "create forward event");
#undef GEMV_TRY
  *out = h;
  clear_error();
  return EBAG_OK;
}

int gemv_ar_forward(gemv_ar_t h, const void* const* A, const void* const* x, float* const* y, uint32_t* out_flags,
                    hipStream_t stream) {
  GemvArgs a;
  int rc = fill_args(h, A, x, y, out_flags, &a);
  if (rc) return rc;
  // The peer flags carry this call's epoch, fixed at capture: a graph replay
  // would see the previous replay's flags and not wait.
  if (h->opts.reduce_mode == 1 && capturing(stream))
    return fail(EBAG_EUNSUPPORTED, "reduce_mode 1 cannot be captured into a graph (use reduce_mode 0)");
  rc = check_busy(h, stream);
  if (rc) return rc;
  // A fresh epoch per forward: peer flags of earlier forwards never match.
  // Epoch 0 is the value the flags start from, so it is skipped.
  if (++h->epoch == 0) ++h->epoch;
  a.epoch = h->epoch;
  if (h->opts.reduce_mode == 0) {
    hipLaunchKernelGGL(last_arriver_fn(h->dtype), dim3((unsigned)(h->R * h->P)), dim3(h->block),
                       (size_t)h->max_x_bytes, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hipf(e, "launch the fused GEMV + AllReduce kernel");
    return note_forward(h, stream);
  }
  void* args[] = {&a};
  const hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(fused_fn(h->dtype)),
                                                  dim3((unsigned)(h->R * h->P)), dim3(h->block), args,
                                                  (unsigned)h->max_x_bytes, stream);
  if (e != hipSuccess) return hipf(e, "cooperative launch of the fused GEMV + AllReduce kernel");
  return note_forward(h, stream);
}

int gemv_ar_unfused_forward(gemv_ar_t h, const void* const* A, const void* const* x, float* const* y,
                            uint32_t* out_flags, hipStream_t stream) {
  GemvArgs a;
  int rc = fill_args(h, A, x, y, out_flags, &a);
  if (rc) return rc;
  rc = check_busy(h, stream);
  if (rc) return rc;
  const int64_t g1 = (int64_t)h->R * h->n_tiles;
  if (g1 > INT_MAX) return fail(EBAG_EINVAL, "too many tiles for one launch");
  hipLaunchKernelGGL(partial_fn(h->dtype), dim3((unsigned)g1), dim3(h->block), (size_t)h->max_x_bytes, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hipf(e, "launch GEMV kernel");
  hipLaunchKernelGGL(allreduce_kernel, dim3((unsigned)((h->M + 255) / 256)), dim3(256), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return hipf(e, "launch AllReduce kernel");
  if (out_flags) {
    const int64_t n = (int64_t)h->R * h->P;
    hipLaunchKernelGGL(bump_flags_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, out_flags, n);
    e = hipGetLastError();
    if (e != hipSuccess) return hipf(e, "launch flag kernel");
  }
  return note_forward(h, stream);
}

int gemv_ar_status(gemv_ar_t h, int32_t out[2]) {
  if (!h || !out) return fail(EBAG_EINVAL, "null plan or output");
  const DeviceGuard dg(h->device);
  if (dg.error() != hipSuccess) return hipf(dg.error(), "make the plan's device current");
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hipf(e, "synchronize");
  int32_t s[2];
  e = hipMemcpy(s, h->d_status, sizeof s, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hipf(e, "read status");
  out[0] = s[0];
  out[1] = s[1] == INT_MAX ? -1 : s[1];
  return s[0] ? EBAG_ETIMEOUT : EBAG_OK;
}

int gemv_ar_reset(gemv_ar_t h) {
  if (!h) return fail(EBAG_EINVAL, "null plan");
  const DeviceGuard dg(h->device);
  if (dg.error() != hipSuccess) return hipf(dg.error(), "make the plan's device current");
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(h->d_status, kGemvStatusInit, sizeof(kGemvStatusInit), hipMemcpyHostToDevice);
  if (e != hipSuccess) return hipf(e, "reset status");
  return EBAG_OK;
}

int gemv_ar_launch_info(gemv_ar_t h, int32_t out[5]) {
  if (!h || !out) return fail(EBAG_EINVAL, "null plan or output");
  out[0] = h->P;
  out[1] = h->block;
  out[2] = (int32_t)(h->n_tiles > INT_MAX ? INT_MAX : h->n_tiles);
  out[3] = h->resident;
  out[4] = h->opts.tile_rows;
  return EBAG_OK;
}

void gemv_ar_destroy(gemv_ar_t h) { free_gemv(h); }

}  // extern "C"
