/*
 * CPU oracle for the fused embedding-pooling + All-to-All send layout, and
 * for the GEMV + AllReduce operator (at the end of this file).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the GPU path.
 *
 * What it computes (the plain definition the fused operator must reach):
 *
 *   Embedding pooling (Sec. III-A): one logical workgroup of the original
 *   EmbeddingBag kernel (a sum / mean pooling kernel) produces one pooled
 *   output vector; for table t and sample b the bag is the index run
 *   offsets[t*B+b] .. offsets[t*B+b+1] and the output is the (optionally
 *   per-index weighted) sum of the indexed rows, or in mean mode that sum
 *   divided by the bag length L (zeros for an empty bag; mean takes no
 *   weights).  Accumulation is in fp64, in index order; fp32/fp16/bf16 widen
 *   exactly.
 *
 *   All-to-All placement (Sec. III-A, worked example): the global batch is
 *   split into R equal contiguous parts, the first part going to destination
 *   0; destination r receives an array of shape {local batch S = B/R,
 *   numTables x D} in which table t occupies the column range
 *   [off_t, off_t + D_t) with off_t = sum of D over the tables before t.
 *   So pooled vector (t, b) lands at send[r][s][off_t + j] with r = b / S,
 *   s = b mod S.
 *
 *   Ready flags (Sec. III-A, "Book-keeping Flags"): one flag per slice; a
 *   slice here is C consecutive samples of one destination for all tables, so
 *   destination r has S / C slices and flag (r, c) is at r * (S / C) + c --
 *   or, with per-table slices, one flag per (slice, table) at
 *   (r * (S / C) + c) * T + t.  After `epoch` complete forwards from a zeroed
 *   array every flag equals `epoch`.
 *
 * Readings of points the paper leaves open: empty bags give zeros; repeated
 * indices count with multiplicity; out-of-range indices, non-monotone offsets,
 * B % R != 0 and S % C != 0 are rejected; output is fp32 for every storage
 * type, obtained by rounding the fp64 sum to nearest-even.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };

enum {
  OR_OK = 0,
  OR_BAD_ARGS = -1,
  OR_BAD_SPLIT = -2,    /* B % R != 0 or (B / R) % C != 0 */
  OR_BAD_OFFSETS = -3,  /* offsets[0] != 0, decreasing, or last != nnz */
  OR_BAD_INDEX = -4     /* index outside [0, rows_t) */
};

/* fp16 bit pattern -> exact double (IEEE 754 binary16: 1 sign, 5 exponent
 * bits with bias 15, 10 fraction bits; exponent 0 is subnormal). */
double oracle_half_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int f = h & 0x3ff;
  double v;
  if (e == 0)
    v = ldexp((double)f, -24); /* f * 2^-10 * 2^-14 */
  else if (e == 31)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(f + 1024), e - 25); /* (1 + f/1024) * 2^(e-15) */
  return sign ? -v : v;
}

/* bf16 bit pattern -> exact double: bf16 is the upper half of an fp32. */
double oracle_bf16_to_double(uint16_t h) {
  uint32_t bits = (uint32_t)h << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

static double load_elem(const void* table, int dtype, int64_t e) {
  if (dtype == OR_F32) return (double)((const float*)table)[e];
  if (dtype == OR_F16) return oracle_half_to_double(((const uint16_t*)table)[e]);
  return oracle_bf16_to_double(((const uint16_t*)table)[e]);
}

/* Step 1: validate the inputs the way the definition needs them. */
int oracle_validate(int32_t T, const int64_t* rows, const int32_t* dims, const int32_t* indices, int64_t nnz,
                    const int64_t* offsets, int64_t B, int32_t R, int32_t C) {
  if (T <= 0 || B <= 0 || R <= 0 || C <= 0 || !rows || !dims || !offsets || (nnz > 0 && !indices))
    return OR_BAD_ARGS;
  for (int32_t t = 0; t < T; ++t)
    if (rows[t] < 0 || dims[t] <= 0) return OR_BAD_ARGS;
  if (B % R != 0) return OR_BAD_SPLIT;
  if ((B / R) % C != 0) return OR_BAD_SPLIT;
  if (offsets[0] != 0 || offsets[(int64_t)T * B] != nnz) return OR_BAD_OFFSETS;
  for (int64_t q = 0; q < (int64_t)T * B; ++q)
    if (offsets[q + 1] < offsets[q]) return OR_BAD_OFFSETS;
  for (int32_t t = 0; t < T; ++t)
    for (int64_t k = offsets[(int64_t)t * B]; k < offsets[(int64_t)(t + 1) * B]; ++k)
      if (indices[k] < 0 || (int64_t)indices[k] >= rows[t]) return OR_BAD_INDEX;
  return OR_OK;
}

typedef struct {
  int32_t T;
  const void* const* tables;
  const int32_t* dims;
  const int64_t* col_off;
  int64_t sum_dim;
  int32_t dtype;
  const int32_t* indices;
  const int64_t* offsets;
  const float* weights;
  int32_t mean;
  int64_t B;
  int32_t R;
  double* sum64;
  double* abs64;
  float* send;
  int64_t b_begin, b_end;
} job_t;

/* Steps 2 and 3 for the samples [b_begin, b_end): pool every bag of those
 * samples in fp64 and place it in the destination-partitioned layout. */
static void* pool_range(void* arg) {
  const job_t* J = (const job_t*)arg;
  const int64_t S = J->B / J->R;
  for (int64_t b = J->b_begin; b < J->b_end; ++b) {
    const int64_t r = b / S;      /* destination rank: first S samples go to rank 0 */
    const int64_t s = b % S;      /* row inside the destination's local batch */
    for (int32_t t = 0; t < J->T; ++t) {
      const int64_t D = J->dims[t];
      const int64_t lo = J->offsets[(int64_t)t * J->B + b];
      const int64_t hi = J->offsets[(int64_t)t * J->B + b + 1];
      const int64_t out = (r * S + s) * J->sum_dim + J->col_off[t];
      for (int64_t j = 0; j < D; ++j) {
        double sum = 0.0, mag = 0.0;
        for (int64_t k = lo; k < hi; ++k) {
          const double w = J->weights ? (double)J->weights[k] : 1.0;
          const double term = w * load_elem(J->tables[t], J->dtype, (int64_t)J->indices[k] * D + j);
          sum += term;
          mag += fabs(term);
        }
        if (J->mean && hi > lo) {
          sum /= (double)(hi - lo);
          mag /= (double)(hi - lo);
        }
        if (J->sum64) J->sum64[out + j] = sum;
        if (J->abs64) J->abs64[out + j] = mag;
        if (J->send) J->send[out + j] = (float)sum;
      }
    }
  }
  return NULL;
}

/*
 * Full pooled send buffer for one forward.
 *   tables   : T host pointers, table t is rows[t] x dims[t], row-major, dtype
 *   indices  : int32 [nnz], table-major CSR; offsets: int64 [T*B + 1]
 *   weights  : fp32 [nnz] or NULL (plain sum)
 *   mode     : 0 sum, 1 mean (weights must then be NULL)
 *   sum64/abs64 : [B * sum(D)] fp64 (either may be NULL); send: fp32 [B * sum(D)]
 *   nthreads : worker threads over sample ranges (<= 0 means 1)
 * Returns OR_OK or a negative OR_* code (outputs untouched on error).
 */
int oracle_pool(int32_t T, const void* const* tables, const int64_t* rows, const int32_t* dims, int32_t dtype,
                const int32_t* indices, int64_t nnz, const int64_t* offsets, const float* weights, int32_t mode,
                int64_t B, int32_t R, int32_t C, double* sum64, double* abs64, float* send, int32_t nthreads) {
  if (!tables || dtype < OR_F32 || dtype > OR_BF16) return OR_BAD_ARGS;
  if (mode < 0 || mode > 1 || (mode == 1 && weights)) return OR_BAD_ARGS;
  int rc = oracle_validate(T, rows, dims, indices, nnz, offsets, B, R, C);
  if (rc != OR_OK) return rc;
  int64_t* col_off = (int64_t*)malloc(sizeof(int64_t) * (size_t)T);
  if (!col_off) return OR_BAD_ARGS;
  int64_t sum_dim = 0;
  for (int32_t t = 0; t < T; ++t) {
    col_off[t] = sum_dim;
    sum_dim += dims[t];
  }
  if (nthreads <= 0) nthreads = 1;
  if (nthreads > B) nthreads = (int32_t)B;
  job_t* jobs = (job_t*)calloc((size_t)nthreads, sizeof(job_t));
  pthread_t* th = (pthread_t*)calloc((size_t)nthreads, sizeof(pthread_t));
  for (int32_t i = 0; i < nthreads; ++i) {
    job_t J = {T, tables, dims, col_off, sum_dim, dtype, indices, offsets, weights, mode, B, R, sum64, abs64,
               send, B * i / nthreads, B * (i + 1) / nthreads};
    jobs[i] = J;
  }
  for (int32_t i = 1; i < nthreads; ++i) pthread_create(&th[i], NULL, pool_range, &jobs[i]);
  pool_range(&jobs[0]);
  for (int32_t i = 1; i < nthreads; ++i) pthread_join(th[i], NULL);
  free(th);
  free(jobs);
  free(col_off);
  return OR_OK;
}

/* Step 4: the ready flags after `epoch` complete forwards.  per_slice = 1:
 * R * (S / C) entries, slice (r, c) at r * (S / C) + c.  per_slice = T
 * (the per-table slices of Sec. III-A): each slice is split per table and
 * (r, c, t) is at (r * (S / C) + c) * T + t.  Every entry equals epoch. */
int oracle_flags(int64_t B, int32_t R, int32_t C, int32_t per_slice, uint32_t epoch, uint32_t* flags,
                 int64_t n_flags) {
  if (B <= 0 || R <= 0 || C <= 0 || B % R || (B / R) % C) return OR_BAD_SPLIT;
  const int64_t S = B / R, nC = S / C;
  if (per_slice <= 0 || n_flags != R * nC * per_slice || !flags) return OR_BAD_ARGS;
  for (int64_t r = 0; r < R; ++r)
    for (int64_t c = 0; c < nC; ++c)
      for (int32_t t = 0; t < per_slice; ++t) flags[(r * nC + c) * per_slice + t] = epoch;
  return OR_OK;
}

/*
 * GEMV + AllReduce (Sec. III-B, scale-up operator): R ranks; rank r holds a
 * row-major M x K_r matrix A_r and a vector x_r of K_r elements (the
 * column split of y = A x in a tensor-parallel layer).  The AllReduce leaves
 * on every rank y = sum over r of A_r x_r, M elements.
 *   A, x   : R host pointers each, storage dtype (fp32 / fp16 / bf16)
 *   Ks     : K_r per rank (> 0)
 *   y64, abs64 : [M] fp64 sum and sum of |terms| (either may be NULL)
 *   y      : [M] fp32, the fp64 sum rounded to nearest-even (may be NULL)
 * Terms are accumulated in fp64, rank by rank, then column by column.
 */
typedef struct {
  int32_t R;
  int64_t M;
  const int64_t* Ks;
  int32_t dtype;
  const void* const* A;
  const void* const* x;
  double* y64;
  double* abs64;
  float* y;
  int64_t i_begin, i_end;
} gemv_job_t;

static void* gemv_rows(void* arg) {
  const gemv_job_t* J = (const gemv_job_t*)arg;
  for (int64_t i = J->i_begin; i < J->i_end; ++i) {
    double sum = 0.0, mag = 0.0;
    for (int32_t r = 0; r < J->R; ++r) {
      const int64_t K = J->Ks[r];
      for (int64_t k = 0; k < K; ++k) {
        const double term = load_elem(J->A[r], J->dtype, i * K + k) * load_elem(J->x[r], J->dtype, k);
        sum = sum + term;
        mag = mag + fabs(term);
      }
    }
    if (J->y64) J->y64[i] = sum;
    if (J->abs64) J->abs64[i] = mag;
    if (J->y) J->y[i] = (float)sum;
  }
  return NULL;
}

int oracle_gemv_ar(int32_t R, int64_t M, const int64_t* Ks, int32_t dtype, const void* const* A,
                   const void* const* x, double* y64, double* abs64, float* y, int32_t nthreads) {
  if (R <= 0 || M <= 0 || !Ks || !A || !x || dtype < OR_F32 || dtype > OR_BF16) return OR_BAD_ARGS;
  for (int32_t r = 0; r < R; ++r)
    if (Ks[r] <= 0 || !A[r] || !x[r]) return OR_BAD_ARGS;
  if (nthreads <= 0) nthreads = 1;
  if (nthreads > M) nthreads = (int32_t)M;
  gemv_job_t* jobs = (gemv_job_t*)calloc((size_t)nthreads, sizeof(gemv_job_t));
  pthread_t* th = (pthread_t*)calloc((size_t)nthreads, sizeof(pthread_t));
  if (!jobs || !th) {
    free(jobs);
    free(th);
    return OR_BAD_ARGS;
  }
  for (int32_t t = 0; t < nthreads; ++t) {
    gemv_job_t J = {R, M, Ks, dtype, A, x, y64, abs64, y, M * t / nthreads, M * (t + 1) / nthreads};
    jobs[t] = J;
  }
  for (int32_t t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, gemv_rows, &jobs[t]);
  gemv_rows(&jobs[0]);
  for (int32_t t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
  free(th);
  free(jobs);
  return OR_OK;
}

/*
 * Embedding backward (the backward counterpart of the pooling above, which
 * the paper overlaps with its All-to-All as well, Sec. IV-D): the owner of
 * the tables receives the gradient of every pooled vector in the same
 * destination-partitioned layout, grad[R][S][sum D] (= [B][sum D]).  The
 * gradient of lookup k of bag (t, b) -- the row indices[k] contributed once
 * to that bag -- is
 *   sum mode:   w_k * grad[b][off_t .. off_t + D_t)   (w_k = 1 without weights)
 *   mean mode:  grad[b][off_t .. off_t + D_t) / L      (L = the bag's length)
 * Output: for each table, in lookup order, a block of nnz_t rows of D_t
 * fp32 values; the blocks follow each other in table order (table t starts
 * at sum over t' < t of nnz_t' * D_t' floats).  Each value is the exact
 * result rounded to fp32 once (fp32 x fp32 products and quotients by L are
 * computed exactly enough in fp64 for that rounding to be the correct one).
 */
int oracle_backward(int32_t T, const int32_t* dims, const int64_t* offsets, const float* weights, int32_t mode,
                    int64_t B, int32_t R, const float* grad, float* values) {
  if (T <= 0 || B <= 0 || R <= 0 || !dims || !offsets || !grad || !values) return OR_BAD_ARGS;
  if (mode < 0 || mode > 1 || (mode == 1 && weights)) return OR_BAD_ARGS;
  if (B % R != 0) return OR_BAD_SPLIT;
  if (offsets[0] != 0) return OR_BAD_OFFSETS;
  for (int64_t q = 0; q < (int64_t)T * B; ++q)
    if (offsets[q + 1] < offsets[q]) return OR_BAD_OFFSETS;
  int64_t sum_dim = 0;
  for (int32_t t = 0; t < T; ++t) {
    if (dims[t] <= 0) return OR_BAD_ARGS;
    sum_dim += dims[t];
  }
  int64_t block = 0;  /* first float of table t's block */
  int64_t col = 0;    /* off_t */
  for (int32_t t = 0; t < T; ++t) {
    const int64_t D = dims[t];
    const int64_t first = offsets[(int64_t)t * B];
    for (int64_t b = 0; b < B; ++b) {
      const int64_t lo = offsets[(int64_t)t * B + b], hi = offsets[(int64_t)t * B + b + 1];
      const float* g = grad + b * sum_dim + col; /* [B][sum D] row b = send[r][s] with b = r * S + s */
      for (int64_t k = lo; k < hi; k++) {
        float* out = values + block + (k - first) * D;
        for (int64_t j = 0; j < D; ++j) {
          double v = (double)g[j];
          if (mode == 1)
            v = v / (double)(hi - lo);
          else if (weights)
            v = (double)weights[k] * v;
          out[j] = (float)v;
        }
      }
    }
    block += (offsets[(int64_t)(t + 1) * B] - first) * D;
    col += D;
  }
  return OR_OK;
}
