// Embedding-bag pooling kernels for gfx950.
//
// One wavefront pools one bag at a time (the paper's "logical workgroup" of
// the EmbeddingBag kernel, Sec. III-A).  A workgroup takes a *run* of up to K
// consecutive samples of one table inside one slice and its waves share the
// run's bags; after the run the workgroup bumps that slice's counter once,
// and the arrival that completes the slice releases the slice's flag
// (Sec. III-A, "Book-keeping Flags").
//
// Gather: a row of D_t elements is V = D_t*elt/16 sixteen-byte vectors.  For
// V a power of two <= 64 the 64 lanes form G = 64/V row groups, lane (g, v)
// loads vector v of rows g, g+G, g+2G, ... so one wave instruction fetches G
// whole rows (1 KiB) with fully coalesced 16-byte loads; every wave keeps U
// such loads in flight.  A wave's block of bags has its index run staged in
// LDS with coalesced loads and read back by broadcast.  Partial sums of the G
// groups are combined with cross-lane xor-shuffles.
//
// Fast path (tables < 4 GiB, V = 2^k, no index checks): each pooled row goes
// to an LDS tile of the run; the last wave of the workgroup to finish writes
// the whole run to its destination slots with contiguous 16-byte stores,
// waits for them and updates the slice counter -- no workgroup barrier, and
// no store queued ahead of a gather load.  General path (any width, index
// checks): per-bag staging, rows stored directly, a barrier before the
// counter update.
//
// Run order (run_at): by default runs are numbered slice-major (all runs of
// slice 0, then slice 1 ...), tables fastest inside a slice, so slices
// complete progressively and a consumer can drain them while later slices
// are still being pooled.  Table-major order pools one table at a time, on
// each XCD separately (table_major = 1: the table's hot rows stay in that
// XCD's L2) or on the whole device (table_major = 2: the table shares the
// Infinity Cache); with per-table slices those still complete progressively.
#include "common.h"

namespace ebag {
namespace {

constexpr int SEG = 128;       // indices staged in LDS per wave per step

typedef uint32_t u4v __attribute__((ext_vector_type(4)));

struct EF32 { static constexpr int EPV = 4; };
struct EF16 { static constexpr int EPV = 8; };
struct EBF16 { static constexpr int EPV = 8; };

template <class E> struct Widen;

template <> struct Widen<EF32> {
  template <bool WT>
  static __device__ __forceinline__ void add(float* acc, const u4v& r, float w) {
    const float x[4] = {__uint_as_float(r.x), __uint_as_float(r.y), __uint_as_float(r.z), __uint_as_float(r.w)};
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = WT ? __builtin_fmaf(w, x[e], acc[e]) : acc[e] + x[e];
  }
};

__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

// fp16 rows: every element goes through one fma(w, widen(h), acc), also
// without weights.  There the caller's w is 1 for a row it loaded and 0 for a
// slot it left empty (whose row bits are zero), a value the compiler cannot
// fold, so it emits one mixed-precision FMA per element (the fp16 operand is
// widened inside the instruction) instead of a convert and an add.  Since
// 1 * x and 0 * (+0) are exact, the single rounding gives the bits acc + x and
// acc + 0 would: the result does not change, only the instruction count.
template <> struct Widen<EF16> {
  template <bool WT>
  static __device__ __forceinline__ void add(float* acc, const u4v& r, float w) {
    const uint32_t u[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = h2f(u[e] & 0xffffu), hi = h2f(u[e] >> 16);
      acc[2 * e] = __builtin_fmaf(w, lo, acc[2 * e]);
      acc[2 * e + 1] = __builtin_fmaf(w, hi, acc[2 * e + 1]);
    }
  }
};

template <> struct Widen<EBF16> {
  template <bool WT>
  static __device__ __forceinline__ void add(float* acc, const u4v& r, float w) {
    const uint32_t u[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(u[e] << 16), hi = __uint_as_float(u[e] & 0xffff0000u);
      acc[2 * e] = WT ? __builtin_fmaf(w, lo, acc[2 * e]) : acc[2 * e] + lo;
      acc[2 * e + 1] = WT ? __builtin_fmaf(w, hi, acc[2 * e + 1]) : acc[2 * e + 1] + hi;
    }
  }
};

// Mean pooling: divide the bag's pooled sum by its length (div > 0; an IEEE
// division, so an exact fp32 sum gives the correctly rounded mean).
template <int EPV>
__device__ __forceinline__ void divide(float* acc, int div) {
  if (div > 0) {
    const float d = (float)div;
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] = acc[e] / d;
  }
}

// LDS written by some lanes of a wave and read by others: keep the compiler
// from reordering across this point and wait for the LDS writes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Table rows live in global memory; say so, so the loads are global_load
// (vmcnt only) rather than flat loads that would also hold up LDS reads.
typedef __attribute__((address_space(1))) const u4v gu4v;
typedef __attribute__((address_space(1))) const int32_t gint;
typedef __attribute__((address_space(1))) const float gfloat;

__device__ __forceinline__ u4v ld_row(const char* colp, int32_t r, uint32_t row_bytes) {
  return *(gu4v*)(colp + (uint64_t)(uint32_t)r * row_bytes);
}

constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data format

// Row loads through a buffer descriptor covering exactly one table (tables
// below 4 GiB): 32-bit offsets keep one address register per load instead
// of two, and the hardware range check turns any offset past the table into
// zeros, so even invalid indices cannot read outside the table.
// NT: non-temporal (streaming) loads -- rows that will not be read again do
// not displace reusable lines (such as the pooled output being written) from
// L2 and the Infinity Cache.
template <bool NT>
struct BufRows {
  __amdgpu_buffer_rsrc_t rs;
  uint32_t col;  // byte offset of this lane's 16-byte vector inside a row
  uint32_t rb;   // row bytes
  __device__ __forceinline__ u4v load(int32_t r) const {
    return __builtin_amdgcn_raw_buffer_load_b128(rs, (uint32_t)r * rb + col, 0, NT ? 2 : 0);
  }
};

// Plain 64-bit addressed row loads (any table size).
struct GlobalRows {
  const char* colp;
  uint32_t rb;
  __device__ __forceinline__ u4v load(int32_t r) const { return ld_row(colp, r, rb); }
};

// Output stores go through a buffer descriptor spanning exactly one pooled
// row (out-of-range lanes are dropped by the hardware).  sc1 = 1 gives
// device-scope stores: they complete at device scope, so a release needs no
// L2 writeback for them; sc1 = 0 gives plain write-back stores.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(float* row, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(row, 0, bytes, kBufferWord3);
}

__device__ __forceinline__ void store16(__amdgpu_buffer_rsrc_t r, int off, float a, float b, float c, float d,
                                        bool sc1) {
  const u4v x = {__float_as_uint(a), __float_as_uint(b), __float_as_uint(c), __float_as_uint(d)};
  if (sc1)
    __builtin_amdgcn_raw_buffer_store_b128(x, r, off, 0, 16);
  else
    __builtin_amdgcn_raw_buffer_store_b128(x, r, off, 0, 0);
}

// Stage indices (and weights) [base, base + n) into this wave's LDS slot
// with coalesced loads.
template <bool WT>
__device__ __forceinline__ void stage(const int32_t* __restrict__ idx, const float* __restrict__ wts, int64_t base,
                                      int n, int lane, int32_t* lds_i, float* lds_w) {
  // Four 64-index loads in flight before the first LDS write.
  for (int i0 = 0; i0 < n; i0 += 256) {
    int32_t x[4];
    float y[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + 64 * u + lane;
      x[u] = i < n ? ((gint*)idx)[base + i] : 0;
      y[u] = (WT && i < n) ? ((gfloat*)wts)[base + i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + 64 * u + lane;
      if (i < n) {
        lds_i[i] = x[u];
        if (WT) lds_w[i] = y[u];
      }
    }
  }
}

// Gather and accumulate n staged rows whose width is V = 2^vs <= 64 vectors:
// lane (g, v) with g = lane >> vs takes vector v of rows g, g + G, ... (G = 64
// / V); U index reads from LDS first (clamped into the staged run, no
// branches), then U predicated 16-byte row loads, then the accumulation.
// Returns true in lanes that met an out-of-range index (CHECK only; such rows
// are skipped).
template <class E, int U, bool WT, bool CHECK, class Rows>
__device__ __forceinline__ bool gather_p2(const Rows& rows_ld, int vs, int64_t rows, const int32_t* li,
                                          const float* lw, int n, int lane, float* acc) {
  const int G = 64 >> vs;
  const int g = lane >> vs;
  bool bad = false;
  for (int k0 = 0; k0 < n; k0 += G * U) {
    int32_t r[U];
    float wv[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = k0 + u * G + g;
      ok[u] = k < n;
      const int kc = ok[u] ? k : n - 1;
      r[u] = li[kc];
      wv[u] = WT ? lw[kc] : 1.f;
    }
    if (CHECK) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = r[u] >= 0 && (int64_t)r[u] < rows;
        bad |= ok[u] && !in;
        ok[u] = ok[u] && in;
      }
    }
    u4v raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      raw[u] = u4v{0u, 0u, 0u, 0u};
      if (ok[u]) raw[u] = rows_ld.load(r[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) Widen<E>::template add<WT>(acc, raw[u], ok[u] ? wv[u] : 0.f);
  }
  return bad;
}

// Any row width: 64-vector column blocks, one row per wave step, indices
// staged SEG at a time.  Used for widths that are not 2^k <= 64 vectors.
template <class E, int U, bool WT>
__device__ __forceinline__ bool pool_bag_generic(const char* __restrict__ tab, const TabMeta& m,
                                                 const int32_t* __restrict__ idx, const float* __restrict__ wts,
                                                 int64_t lo, int L, int32_t* lds_i, float* lds_w, int lane,
                                                 int check, float* __restrict__ orow, bool sc1, int div) {
  constexpr int EPV = E::EPV;
  bool bad = false;
  for (int cb = 0; cb < m.vecs; cb += 64) {
    const int vv = cb + lane;
    const bool act = vv < m.vecs;
    const char* colp = tab + (int64_t)vv * 16;
    float acc[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] = 0.f;
    for (int s0 = 0; s0 < L; s0 += SEG) {
      const int n = min(SEG, L - s0);
      stage<WT>(idx, wts, lo + s0, n, lane, lds_i, lds_w);
      wave_lds_sync();
      for (int k0 = 0; k0 < n; k0 += U) {
        int32_t r[U];
        float wv[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = k0 + u;
          ok[u] = k < n && act;
          const int kc = k < n ? k : n - 1;
          r[u] = lds_i[kc];
          wv[u] = WT ? lds_w[kc] : 1.f;
        }
        if (check) {
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const bool in = r[u] >= 0 && (int64_t)r[u] < m.rows;
            bad |= ok[u] && !in;
            ok[u] = ok[u] && in;
          }
        }
        u4v raw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          raw[u] = u4v{0u, 0u, 0u, 0u};
          if (ok[u]) raw[u] = ld_row(colp, r[u], (uint32_t)m.row_bytes);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) Widen<E>::template add<WT>(acc, raw[u], ok[u] ? wv[u] : 0.f);
      }
      wave_lds_sync();
    }
    divide<EPV>(acc, div);
    if (act) {
      const __amdgpu_buffer_rsrc_t rs = row_rsrc(orow, m.dim * 4);
#pragma unroll
      for (int h = 0; h < EPV / 4; ++h)
        store16(rs, (vv * EPV + 4 * h) * 4, acc[4 * h], acc[4 * h + 1], acc[4 * h + 2], acc[4 * h + 3], sc1);
    }
  }
  return bad;
}

// Combine the G row groups (lane bits vs..5) with xor shuffles, then store
// the row with 16-byte stores laid out so that one instruction covers the row
// contiguously: fp32 tables -- lane v of group 0 writes floats [4v, 4v + 4);
// 16-bit tables (8 values per lane) -- groups 0 and 1 write the two halves
// of lane v's 32 bytes (every lane holds the total after the xor butterfly).
template <int EPV>
__device__ __forceinline__ void reduce_store(float* acc, int vs, int lane, float* __restrict__ orow, int dim,
                                             bool sc1, int div) {
  const int V = 1 << vs;
  for (int msk = 32; msk >= V; msk >>= 1) {
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] += __shfl_xor(acc[e], msk);
  }
  divide<EPV>(acc, div);
  const int g = lane >> vs;
  const int v = lane & (V - 1);
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(orow, dim * 4);
  if (EPV == 4) {
    if (g == 0) store16(rs, 16 * v, acc[0], acc[1], acc[2], acc[3], sc1);
  } else if (vs <= 5) {
    if (g < 2) {
      const bool hi = g == 1;
      store16(rs, 32 * v + 16 * g, hi ? acc[4] : acc[0], hi ? acc[5] : acc[1], hi ? acc[6] : acc[2],
              hi ? acc[7] : acc[3], sc1);
    }
  } else {
    store16(rs, 32 * v, acc[0], acc[1], acc[2], acc[3], sc1);
    store16(rs, 32 * v + 16, acc[4], acc[5], acc[6], acc[7], sc1);
  }
}

// Read-only inputs read with wave-uniform addresses (table order, table
// constants and pointers, CSR offsets) go through the scalar data cache:
// their latency then does not queue behind the row gathers in the vector
// memory pipeline.  Nothing the kernel writes is read this way.
template <class T>
__device__ __forceinline__ T sload(const T* p, int64_t i) {
  return ((const __attribute__((address_space(4))) T*)p)[i];
}

__device__ __forceinline__ TabMeta load_meta(const TabMeta* p) {
  TabMeta m;
  m.rows = sload(&p->rows, 0);
  m.row_bytes = sload(&p->row_bytes, 0);
  m.dim = sload(&p->dim, 0);
  m.col_off = sload(&p->col_off, 0);
  m.vecs = sload(&p->vecs, 0);
  m.vshift = sload(&p->vshift, 0);
  return m;
}

// Combine the G row groups and write the bag's pooled row (dim floats) into
// the workgroup's LDS output buffer (lanes of group 0, EPV floats each);
// div > 0: mean pooling over div rows.
template <int EPV>
__device__ __forceinline__ void reduce_to_lds(float* acc, int vs, int lane, float* lrow, int div) {
  const int V = 1 << vs;
  for (int msk = 32; msk >= V; msk >>= 1) {
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] += __shfl_xor(acc[e], msk);
  }
  divide<EPV>(acc, div);
  if ((lane >> vs) == 0) {
    float4* d = reinterpret_cast<float4*>(lrow + (lane & (V - 1)) * EPV);
#pragma unroll
    for (int h = 0; h < EPV / 4; ++h) d[h] = make_float4(acc[4 * h], acc[4 * h + 1], acc[4 * h + 2], acc[4 * h + 3]);
  }
}

// Write nb pooled rows of dim floats (dim / 4 = 2^s4 float4s each) from LDS
// to global rows base + i * stride: 64 lanes x 16 bytes per instruction,
// each row contiguous.
__device__ __forceinline__ void store_rows(const float* lds, int nb, int s4, float* base, int64_t stride, int dim,
                                           int lane, bool sc1) {
  const int n4 = 1 << s4;
  const int64_t span = ((int64_t)(nb - 1) * stride + dim) * 4;
  const __amdgpu_buffer_rsrc_t rs = row_rsrc(base, (int)span);
  const float4* l4 = reinterpret_cast<const float4*>(lds);
  for (int e = lane; e < (nb << s4); e += 64) {
    const int i = e >> s4;
    const int c4 = e & (n4 - 1);
    const float4 x = l4[e];
    store16(rs, (int)((int64_t)i * stride * 4) + c4 * 16, x.x, x.y, x.z, x.w, sc1);
  }
}

// Completion of one run (fused only).  release_mode 0: the workgroup's
// stores are published by an agent-scope release on the slice counter (an L2
// writeback on every run).  release_mode 1: the pooled vectors were stored
// with device-scope stores, each wave waited for them to complete at device
// scope (vmcnt 0) before the barrier, so the counter update needs no cache
// writeback.  The arrival that completes the slice re-arms the counter and
// increments the slice flag.
__device__ __forceinline__ void release_slice(uint32_t* counters, uint32_t* flags, int64_t g, uint32_t n,
                                              uint32_t target, int64_t suppress, uint64_t* trace, int mode) {
  uint32_t old;
  if (mode == 0)
    old = __hip_atomic_fetch_add(&counters[g], n, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  else
    old = __hip_atomic_fetch_add(&counters[g], n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (old + n == target) {
    if (mode == 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    __hip_atomic_store(&counters[g], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (trace) trace[g] = wall_clock64();
    if (g != suppress) {
      if (mode == 0)
        __hip_atomic_fetch_add(&flags[g], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      else
        __hip_atomic_fetch_add(&flags[g], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// s_waitcnt vmcnt(0): every vector memory operation of this wave, stores
// included, has completed (for device-scope stores: at device scope).
__device__ __forceinline__ void wait_stores_complete() { __builtin_amdgcn_s_waitcnt(0x0F70); }

constexpr int SEGW = 512;  // indices a wave stages at once for a block of bags

// Persistent grid: workgroups claim runs in production order from an atomic
// ticket (ticket[0]).  The leading barrier makes sure every wave is done with
// the previous run (its LDS tile and the broadcast slot) before the slot is
// rewritten.
__device__ __forceinline__ int64_t draw_run(uint32_t* ticket, uint32_t* s_tick) {
  __syncthreads();
  if (threadIdx.x == 0) *s_tick = __hip_atomic_fetch_add(&ticket[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return (int64_t)__builtin_amdgcn_readfirstlane(*s_tick);
}

// A workgroup whose draw came back past the last run counts itself out in
// ticket[1]; the last one re-arms both words for the next launch.  Every
// workgroup's final draw has returned (its value decided the exit) before it
// counts itself out, so no draw of this launch can follow the re-arm.
__device__ __forceinline__ void leave_runs(uint32_t* ticket) {
  if (threadIdx.x == 0 &&
      __hip_atomic_fetch_add(&ticket[1], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gridDim.x - 1) {
    __hip_atomic_store(&ticket[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&ticket[1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// One workgroup per run: up to K consecutive samples of one table inside one
// slice.  The counter it feeds is the slice's (target C * T bags) or, with
// per-table slices, the (slice, table) pair's (target C bags).  On the fast
// path wave w pools a contiguous block of the run's bags: it reads the
// block's CSR offsets with scalar loads, stages the block's whole index
// segment into its LDS slot when it fits (else bag by bag, SEGW at a time),
// then gathers and reduces every bag into the run's LDS tile.
template <class E, int U, bool WT, bool FUSED, bool SAFE>
__device__ __forceinline__ void pool_body(const PoolArgs& a) {
  constexpr int EPV = E::EPV;
  extern __shared__ int32_t s_dyn[];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int W = a.waves;
  const int slot = SAFE ? SEG : SEGW;
  int32_t* lds_i = s_dyn + wid * slot;
  float* lds_w = WT ? reinterpret_cast<float*>(s_dyn + W * slot) + wid * slot : nullptr;
  // Fast path: pooled rows of the current run (K x max dim floats, 16-byte
  // aligned) and the arrival counter of the run's waves.
  float* lds_out = reinterpret_cast<float*>(s_dyn + W * slot * (WT ? 2 : 1));
  int32_t* s_arrive = reinterpret_cast<int32_t*>(lds_out + a.out_floats);
  if (!SAFE) {
    if (threadIdx.x == 0) *s_arrive = 0;
    __syncthreads();
  }
  const bool sc1 = FUSED && a.release_mode == 1;
  const int64_t nnz = (!SAFE || a.check) ? sload(a.offsets, (int64_t)a.T * a.B) : 0;
  // One-shot grid: workgroup i pools run i.  Persistent grid (fewer
  // workgroups than runs): runs are claimed from the ticket.
  const bool persistent = gridDim.x < a.nruns;
  uint32_t* s_tick = SAFE ? reinterpret_cast<uint32_t*>(lds_out) : reinterpret_cast<uint32_t*>(s_arrive + 1);
  for (int64_t q = persistent ? draw_run(a.ticket, s_tick) : (int64_t)blockIdx.x; q < a.nruns;
       q = persistent ? draw_run(a.ticket, s_tick) : a.nruns) {
    int64_t gs;
    int32_t tpos, j;
    run_at(a.so, a.T, a.J, q, &gs, &tpos, &j);
    const int t = sload(a.tperm, tpos);
    const int64_t g = slice_at(a.so, gs);
    const int64_t b0 = g * a.C + (int64_t)j * a.K;
    const int64_t b1 = min(b0 + (int64_t)a.K, (g + 1) * (int64_t)a.C);
    const TabMeta m = load_meta(a.meta + t);
    const char* tab = static_cast<const char*>(sload(a.tables, t));
    const int64_t nb = b1 - b0;
    const int64_t per = (nb + W - 1) / W;
    const int64_t bb = b0 + wid * per;
    const int64_t be = min(bb + per, b1);
    const int64_t obase = (int64_t)t * a.B;
    const float* outbase = FUSED ? a.out + m.col_off : a.out + a.B * m.col_off;
    const int64_t ostride = FUSED ? a.sum_dim : m.dim;
    if (!SAFE) {
      BufRows<false> rl;
      rl.rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(tab), 0, (int)(uint32_t)(m.rows * m.row_bytes),
                                                kBufferWord3);
      rl.col = (uint32_t)(lane & ((1 << m.vshift) - 1)) * 16u;
      rl.rb = (uint32_t)m.row_bytes;
      BufRows<true> rn;
      rn.rs = rl.rs;
      rn.col = rl.col;
      rn.rb = rl.rb;
      const bool nt = a.stream_rows;
      for (int64_t blk = bb; blk < be; blk += 63) {
        const int c = (int)min((int64_t)63, be - blk);
        // Offsets are clamped into [0, nnz] and each bag into the block's
        // segment, so malformed CSR input can never drive a read outside the
        // index array (results are then meaningless but memory-safe).
        const int64_t seg_lo = min(max(sload(a.offsets, obase + blk), (int64_t)0), nnz);
        const int64_t seg_hi = min(max(sload(a.offsets, obase + blk + c), seg_lo), nnz);
        const int64_t seg_len = seg_hi - seg_lo;
        const bool all = seg_len <= SEGW;
        if (all) {
          stage<WT>(a.indices, a.weights, seg_lo, (int)seg_len, lane, lds_i, lds_w);
          wave_lds_sync();
        }
        int64_t lo = seg_lo;
        for (int i = 0; i < c; ++i) {
          lo = min(max(sload(a.offsets, obase + blk + i), lo), seg_hi);
          const int64_t hi = min(max(sload(a.offsets, obase + blk + i + 1), lo), seg_hi);
          const int L = (int)(hi - lo);
          float acc[EPV];
#pragma unroll
          for (int e = 0; e < EPV; ++e) acc[e] = 0.f;
          if (all) {
            const int32_t* li = lds_i + (lo - seg_lo);
            const float* lw = WT ? lds_w + (lo - seg_lo) : nullptr;
            if (nt)
              gather_p2<E, U, WT, false>(rn, m.vshift, m.rows, li, lw, L, lane, acc);
            else
              gather_p2<E, U, WT, false>(rl, m.vshift, m.rows, li, lw, L, lane, acc);
          } else {
            for (int s0 = 0; s0 < L; s0 += SEGW) {
              const int n = min(SEGW, L - s0);
              stage<WT>(a.indices, a.weights, lo + s0, n, lane, lds_i, lds_w);
              wave_lds_sync();
              if (nt)
                gather_p2<E, U, WT, false>(rn, m.vshift, m.rows, lds_i, lds_w, n, lane, acc);
              else
                gather_p2<E, U, WT, false>(rl, m.vshift, m.rows, lds_i, lds_w, n, lane, acc);
              wave_lds_sync();
            }
          }
          reduce_to_lds<EPV>(acc, m.vshift, lane, lds_out + (blk + i - b0) * m.dim, a.mean ? L : 0);
        }
        if (all) wave_lds_sync();
      }
      // The last wave to finish its bags writes the whole run from LDS to
      // global memory and (fused) completes the run for the slice; the other
      // waves leave at once.  No workgroup barrier on the fast path, and no
      // store ever sits in front of a gather load of the same wave.
      int old = 0;
      if (lane == 0) old = __hip_atomic_fetch_add(s_arrive, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
      old = __builtin_amdgcn_readfirstlane(old);
      if (old == W - 1) {
        if (lane == 0) __hip_atomic_store(s_arrive, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        const int s4 = m.vshift + (EPV == 8 ? 1 : 0);
        store_rows(lds_out, (int)nb, s4, const_cast<float*>(outbase) + b0 * ostride, ostride, m.dim, lane, sc1);
        if (FUSED) {
          if (a.release_mode == 1) wait_stores_complete();
          if (lane == 0)
            release_slice(a.counters, a.flags, a.per_table ? g * a.T + t : g, (uint32_t)nb,
                          a.per_table ? (uint32_t)a.C : (uint32_t)a.C * (uint32_t)a.T, a.suppress, a.trace_release,
                          a.release_mode);
        }
      }
    } else {
      for (int64_t b = bb; b < be; ++b) {
        int64_t lo = a.offsets[obase + b];
        int64_t hi = a.offsets[obase + b + 1];
        bool bad = false;
        if (a.check && !(lo >= 0 && lo <= hi && hi <= nnz)) {
          bad = true;
          lo = hi = 0;
        }
        const int L = (int)(hi - lo);
        float* orow = const_cast<float*>(outbase) + b * ostride;
        if (m.vshift >= 0) {
          GlobalRows rl;
          rl.colp = tab + (lane & ((1 << m.vshift) - 1)) * 16;
          rl.rb = (uint32_t)m.row_bytes;
          float acc[EPV];
#pragma unroll
          for (int e = 0; e < EPV; ++e) acc[e] = 0.f;
          for (int s0 = 0; s0 < L; s0 += SEG) {
            const int n = min(SEG, L - s0);
            stage<WT>(a.indices, a.weights, lo + s0, n, lane, lds_i, lds_w);
            wave_lds_sync();
            bad |= a.check ? gather_p2<E, U, WT, true>(rl, m.vshift, m.rows, lds_i, lds_w, n, lane, acc)
                           : gather_p2<E, U, WT, false>(rl, m.vshift, m.rows, lds_i, lds_w, n, lane, acc);
            wave_lds_sync();
          }
          reduce_store<EPV>(acc, m.vshift, lane, orow, m.dim, sc1, a.mean ? L : 0);
        } else {
          bad |= pool_bag_generic<E, U, WT>(tab, m, a.indices, a.weights, lo, L, lds_i, lds_w, lane, a.check, orow,
                                            sc1, a.mean ? L : 0);
        }
        if (a.check && __any(bad) && lane == 0) atomicMin(&a.status[ST_FIRST_BAD_BAG], (int32_t)(obase + b));
      }
    }
    if (FUSED && SAFE) {
      if (a.release_mode == 1) wait_stores_complete();
      __syncthreads();
      if (threadIdx.x == 0)
        release_slice(a.counters, a.flags, a.per_table ? g * a.T + t : g, (uint32_t)nb,
                      a.per_table ? (uint32_t)a.C : (uint32_t)a.C * (uint32_t)a.T, a.suppress, a.trace_release,
                      a.release_mode);
    }
  }
  if (persistent) leave_runs(a.ticket);
}

// Fused operator: pooled vectors go straight to the send layout and slices
// are released as they complete.
template <class E, int U, bool WT, bool SAFE>
__global__ __launch_bounds__(1024) void fused_pool_kernel(const PoolArgs a) {
  pool_body<E, U, WT, true, SAFE>(a);
}

// Unfused baseline, first kernel: plain per-table EmbeddingBag output.
template <class E, int U, bool WT, bool SAFE>
__global__ __launch_bounds__(1024) void unfused_pool_kernel(const PoolArgs a) {
  pool_body<E, U, WT, false, SAFE>(a);
}

typedef void (*pool_fn)(const PoolArgs);

template <class E, int U, bool WT, bool SAFE>
pool_fn pick_f(bool fused) {
  return fused ? &fused_pool_kernel<E, U, WT, SAFE> : &unfused_pool_kernel<E, U, WT, SAFE>;
}

template <class E, int U>
pool_fn pick_wf(bool weighted, bool fused, bool safe) {
  if (weighted) return safe ? pick_f<E, U, true, true>(fused) : pick_f<E, U, true, false>(fused);
  return safe ? pick_f<E, U, false, true>(fused) : pick_f<E, U, false, false>(fused);
}

template <class E>
pool_fn pick_u(int u, bool weighted, bool fused, bool safe) {
  switch (u) {
    case 4: return pick_wf<E, 4>(weighted, fused, safe);
    case 16: return pick_wf<E, 16>(weighted, fused, safe);
    default: return pick_wf<E, 8>(weighted, fused, safe);
  }
}

pool_fn pick(int dtype, int u, bool weighted, bool fused, bool safe) {
  switch (dtype) {
    case 1: return pick_u<EF16>(u, weighted, fused, safe);
    case 2: return pick_u<EBF16>(u, weighted, fused, safe);
    default: return pick_u<EF32>(u, weighted, fused, safe);
  }
}

size_t lds_bytes(bool safe, bool weighted, int block, int out_floats) {
  // + 16 bytes: the run-arrival counter and the ticket broadcast slot
  const size_t staging = (size_t)(block / 64) * (safe ? SEG : SEGW) * (weighted ? 8 : 4);
  return safe ? staging + 16 : staging + (size_t)out_floats * 4 + 16;
}

}  // namespace

hipError_t launch_pool(int dtype, int rows_in_flight, bool weighted, bool fused, bool safe, const PoolArgs& a,
                       int grid, int block, hipStream_t stream) {
  pool_fn f = pick(dtype, rows_in_flight, weighted, fused, safe);
  hipLaunchKernelGGL(f, dim3(grid), dim3(block), lds_bytes(safe, weighted, block, a.out_floats), stream, a);
  return hipGetLastError();
}

int pool_max_wgs_per_cu(int dtype, int rows_in_flight, bool weighted, bool fused, bool safe, int block,
                        int out_floats) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, pick(dtype, rows_in_flight, weighted, fused, safe), block,
                                                   lds_bytes(safe, weighted, block, out_floats)) != hipSuccess)
    return 0;
  return n;
}

}  // namespace ebag
