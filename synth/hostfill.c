/*
 * Host side of the seeded input generator: fills a table in host memory with
 * the counter-based value function, multithreaded, so that multi-GB tables
 * for the CPU baseline are produced in seconds.  Must match synth/gen.py and
 * synth/fill.hip bit for bit:
 *   u = splitmix64(seed ^ (row*dim + j)) >> 40
 *   uniform: v = (float)((int)u - 2^23) * 2^-24, then v * 0.1f (two RNE ops)
 *   cint:    v = (float)((int)(u % 17) - 8)
 * then round-to-nearest-even to fp16 / bf16 storage.
 * SplitMix64: Steele, Lea, Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014.
 */
#include <pthread.h>
#include <stdint.h>
#include <string.h>

static uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static float value_of(uint64_t seed, uint64_t e, int kind) {
  uint64_t u = splitmix64(seed ^ e) >> 40;
  if (kind == 0) {
    const float x = (float)((int32_t)u - (1 << 23)) * 0x1p-24f;
    return x * 0.1f;
  }
  return (float)((int32_t)(u % 17u) - 8);
}

static uint32_t f2u(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

static uint16_t bf16_rne(float v) {
  uint32_t b = f2u(v);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

/* IEEE binary32 -> binary16, round to nearest even (finite inputs of the
 * generator: |v| < 2^16; subnormal results handled). */
static uint16_t half_rne(float v) {
  uint32_t b = f2u(v);
  uint16_t sign = (uint16_t)((b >> 16) & 0x8000u);
  int32_t e = (int32_t)((b >> 23) & 0xff) - 127;
  uint32_t m = b & 0x7fffffu;
  if (((b >> 23) & 0xff) == 0 && m == 0) return sign;
  if (e > 15) return (uint16_t)(sign | 0x7c00u); /* overflow -> inf (not produced here) */
  uint32_t full = m | 0x800000u;                 /* 24-bit significand */
  int shift;                                     /* bits to drop from the 24-bit significand */
  uint32_t exp_field;
  if (e >= -14) {
    shift = 13;
    exp_field = (uint32_t)(e + 15);
  } else {
    shift = 13 + (-14 - e);
    exp_field = 0;
    if (shift > 24) return sign;
  }
  uint32_t kept = full >> shift;
  uint32_t rem = full & ((1u << shift) - 1u);
  uint32_t half = 1u << (shift - 1);
  if (rem > half || (rem == half && (kept & 1u))) kept += 1;
  uint32_t out;
  if (exp_field == 0) {
    out = kept; /* subnormal; a carry into bit 10 makes it the smallest normal */
  } else {
    out = (exp_field << 10) + (kept - 0x400u); /* carry propagates into the exponent */
  }
  return (uint16_t)(sign | out);
}

typedef struct {
  void* dst;
  uint64_t begin, end;
  int32_t dtype, kind;
  uint64_t seed;
} job_t;

static void* fill_range(void* arg) {
  const job_t* J = (const job_t*)arg;
  for (uint64_t e = J->begin; e < J->end; ++e) {
    float v = value_of(J->seed, e, J->kind);
    if (J->dtype == 0)
      ((float*)J->dst)[e] = v;
    else if (J->dtype == 1)
      ((uint16_t*)J->dst)[e] = half_rne(v);
    else
      ((uint16_t*)J->dst)[e] = bf16_rne(v);
  }
  return 0;
}

/* Fill rows x dim elements (dtype 0 f32, 1 f16, 2 bf16; kind 0 uniform,
 * 1 integers in [-8, 8]) using nthreads threads. */
int synth_host_fill(void* dst, int64_t rows, int32_t dim, int32_t dtype, uint64_t seed, int32_t kind,
                    int32_t nthreads) {
  if (!dst || rows < 0 || dim <= 0 || dtype < 0 || dtype > 2 || kind < 0 || kind > 1) return -1;
  uint64_t n = (uint64_t)rows * (uint64_t)dim;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  job_t jobs[256];
  pthread_t th[256];
  for (int i = 0; i < nthreads; ++i) {
    job_t J = {dst, n * (uint64_t)i / (uint64_t)nthreads, n * (uint64_t)(i + 1) / (uint64_t)nthreads, dtype, kind, seed};
    jobs[i] = J;
  }
  for (int i = 1; i < nthreads; ++i) pthread_create(&th[i], 0, fill_range, &jobs[i]);
  fill_range(&jobs[0]);
  for (int i = 1; i < nthreads; ++i) pthread_join(th[i], 0);
  return 0;
}

/* Exposed for tests of the conversion. */
uint16_t synth_half_rne(float v) { return half_rne(v); }
