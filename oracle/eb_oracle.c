/*
 * eb_oracle.c — plain, slow CPU oracle for the pooled EmbeddingBag forward.
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library.  The product path (libeb and its Python
 * binding) never does, and this file shares no code, header, table or
 * constant with it.
 *
 * What it computes (the plain definition).  The paper's DLRM study
 * (Sec. IV-A.2) describes sparse_arch as lookups into embedding tables that
 * produce one output embedding per example and categorical feature; its
 * inputs are jagged categorical features (Abstract, Sec. IV-A.3: embedding-bag
 * lookups over jagged inputs).  For T tables, batch B and bag g = t*B + b
 * covering index positions [off[g], off[g+1]):
 *
 *   S[d] = sum_i w_i * x(t, idx[i], d)        (w_i = 1 without weights)
 *   out  = fl32(S)            for sum pooling
 *        = fl32(S / L)        for mean pooling, L = off[g+1] - off[g]
 *        = +0.0               for an empty bag,
 *
 * written to out[b, Doff[t] .. Doff[t] + D_t).  S is accumulated in fp64
 * (the product of two fp32 values is exact in fp64) in index order and
 * rounded to fp32 once.  x is the fp32 value of a table element:
 *   fp32 rows:     the stored value;
 *   fp16 rows:     the binary16 value, decoded here from its bit fields
 *                  (exact in fp32);
 *   int8 row-wise: D unsigned codes q, then fp16 scale s and fp16 bias c;
 *                  x = fp32(s*q + c) rounded once, i.e. fmaf(s, q, c);
 *   int8 row-wise, split layout: the same values stored apart: row r's D
 *                  codes at data + r*stride, and the scale/bias words of all
 *                  rows in one block after the codes, row r's (s, then c) at
 *                  data + num_rows*stride + 4*r.
 * The paper fixes none of pooling mode, weights, row format or rounding; the
 * readings taken here are the ones listed with the oracle's design notes.
 *
 * Besides `out`, the oracle can return absum = sum_i |w_i * x_i| (divided by
 * L for mean) per output element, in fp64: the scale of the a-priori
 * rounding-error bound that the GPU results are held to.
 *
 * Validation mirrors the checks a caller must satisfy: offsets start at 0,
 * never decrease and end at N; every index lies in [0, R_t).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define EBO_OK 0
#define EBO_ERR_INVALID_ARG (-1)
#define EBO_ERR_DTYPE (-2)
#define EBO_ERR_SHAPE (-3)
#define EBO_ERR_INDEX_OOB (-5)
#define EBO_ERR_OFFSETS (-6)

#define EBO_ROW_F32 0
#define EBO_ROW_F16 1
#define EBO_ROW_U8 2
#define EBO_ROW_U8_SPLIT 3

#define EBO_IDX_I32 0
#define EBO_IDX_I64 1

#define EBO_MODE_SUM 0
#define EBO_MODE_MEAN 1

typedef struct {
  const void *data; /* host pointer to row 0, or NULL if no bag asked for reads it */
  int64_t num_rows;
  int32_t dim;
  int32_t dtype;
  int64_t row_stride_bytes;
} ebo_table;

/* IEEE 754 binary16 -> double, from the bit fields. */
double ebo_half_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int expo = (h >> 10) & 0x1f;
  int mant = h & 0x3ff;
  double v;
  if (expo == 0) {
    v = ldexp((double)mant, -24); /* zero or subnormal: mant * 2^-24 */
  } else if (expo == 31) {
    v = mant ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + mant), expo - 25); /* (1 + mant/1024) * 2^(expo-15) */
  }
  return sign ? -v : v;
}

/* fp32 value of element d of row r (see the header comment). */
static float ebo_element(const ebo_table *tb, int64_t r, int32_t d) {
  const unsigned char *row =
      (const unsigned char *)tb->data + (size_t)r * (size_t)tb->row_stride_bytes;
  if (tb->dtype == EBO_ROW_F32) {
    float v;
    memcpy(&v, row + 4 * (size_t)d, 4);
    return v;
  }
  if (tb->dtype == EBO_ROW_F16) {
    uint16_t h;
    memcpy(&h, row + 2 * (size_t)d, 2);
    return (float)ebo_half_to_double(h);
  }
  /* int8 row-wise: the scale/bias word follows the row's codes, or (split
     layout) sits in the block after all rows' codes */
  const unsigned char *word =
      tb->dtype == EBO_ROW_U8_SPLIT
          ? (const unsigned char *)tb->data + (size_t)tb->num_rows * (size_t)tb->row_stride_bytes + 4 * (size_t)r
          : row + tb->dim;
  uint16_t hs, hc;
  memcpy(&hs, word, 2);
  memcpy(&hc, word + 2, 2);
  float s = (float)ebo_half_to_double(hs);
  float c = (float)ebo_half_to_double(hc);
  return fmaf(s, (float)row[d], c);
}

static int64_t ebo_read_index(const void *p, int32_t type, int64_t i) {
  if (type == EBO_IDX_I32) return (int64_t)((const int32_t *)p)[i];
  return ((const int64_t *)p)[i];
}

/* Pool one bag g into dst[0 .. D_t) (and its error scale into asum, if set). */
static void ebo_pool_bag(const ebo_table *tb, const void *indices, int32_t index_type,
                         int64_t lo, int64_t hi, const float *weights, int32_t mode,
                         float *dst, double *asum) {
  int64_t L = hi - lo;
  for (int32_t d = 0; d < tb->dim; ++d) {
    double acc = 0.0, mag = 0.0;
    for (int64_t i = lo; i < hi; ++i) {
      int64_t r = ebo_read_index(indices, index_type, i);
      double w = weights ? (double)weights[i] : 1.0;
      double term = w * (double)ebo_element(tb, r, d);
      acc += term;
      mag += fabs(term);
    }
    if (mode == EBO_MODE_MEAN && L > 0) {
      acc /= (double)L;
      mag /= (double)L;
    }
    dst[d] = (float)acc;
    if (asum) asum[d] = mag;
  }
}

/*
 * Forward over all bags (bags == NULL) or over the listed bag ids.
 *
 * tables[num_tables]; indices [num_indices]; offsets [num_offsets] with
 * num_offsets = T*B + 1; weights [num_indices] or NULL.
 * bags == NULL: out is [B, sum D] row-major (out_ld must be 0 or sum D).
 * bags != NULL: the k-th listed bag is written to out[k*out_ld .. + D_t);
 *               out_ld >= max D_t over the listed bags' tables.
 * asum (optional) has out's layout.  num_threads <= 0 lets OpenMP choose.
 * Returns 0 or a negative error code; out is not written on error.
 */
int ebo_forward(const ebo_table *tables, int32_t num_tables, const void *indices,
                const void *offsets, int32_t index_type, int64_t num_indices,
                int64_t num_offsets, const float *weights, int32_t mode,
                const int64_t *bags, int64_t num_bags, float *out, int64_t out_ld,
                double *asum, int32_t num_threads) {
  if (!tables || num_tables < 1 || !offsets || !out) return EBO_ERR_INVALID_ARG;
  if (num_indices < 0 || (num_indices > 0 && !indices)) return EBO_ERR_INVALID_ARG;
  if (index_type != EBO_IDX_I32 && index_type != EBO_IDX_I64) return EBO_ERR_DTYPE;
  if (mode != EBO_MODE_SUM && mode != EBO_MODE_MEAN) return EBO_ERR_INVALID_ARG;
  if (weights && mode == EBO_MODE_MEAN) return EBO_ERR_INVALID_ARG;
  if (num_offsets < 2 || (num_offsets - 1) % num_tables != 0) return EBO_ERR_SHAPE;
  const int64_t B = (num_offsets - 1) / num_tables;
  const int64_t nbags = num_offsets - 1;

  int64_t sum_d = 0;
  for (int32_t t = 0; t < num_tables; ++t) {
    const ebo_table *tb = &tables[t];
    if (tb->dtype != EBO_ROW_F32 && tb->dtype != EBO_ROW_F16 && tb->dtype != EBO_ROW_U8 &&
        tb->dtype != EBO_ROW_U8_SPLIT)
      return EBO_ERR_DTYPE;
    if (tb->dim < 1 || tb->num_rows < 1) return EBO_ERR_INVALID_ARG;
    sum_d += tb->dim;
  }

  /* offsets must partition [0, N) into T*B consecutive bags */
  if (ebo_read_index(offsets, index_type, 0) != 0) return EBO_ERR_OFFSETS;
  for (int64_t g = 0; g < nbags; ++g)
    if (ebo_read_index(offsets, index_type, g + 1) < ebo_read_index(offsets, index_type, g))
      return EBO_ERR_OFFSETS;
  if (ebo_read_index(offsets, index_type, nbags) != num_indices) return EBO_ERR_OFFSETS;

  /* every index must name a row of its bag's table */
  for (int32_t t = 0; t < num_tables; ++t) {
    int64_t lo = ebo_read_index(offsets, index_type, (int64_t)t * B);
    int64_t hi = ebo_read_index(offsets, index_type, (int64_t)(t + 1) * B);
    for (int64_t i = lo; i < hi; ++i) {
      int64_t r = ebo_read_index(indices, index_type, i);
      if (r < 0 || r >= tables[t].num_rows) return EBO_ERR_INDEX_OOB;
    }
  }

  int64_t count = bags ? num_bags : nbags;
  if (count < 0) return EBO_ERR_INVALID_ARG;
  if (bags) {
    for (int64_t k = 0; k < count; ++k) {
      if (bags[k] < 0 || bags[k] >= nbags) return EBO_ERR_INVALID_ARG;
      const ebo_table *tb = &tables[bags[k] / B];
      if (out_ld < tb->dim) return EBO_ERR_SHAPE;
      if (!tb->data && ebo_read_index(offsets, index_type, bags[k] + 1) >
                           ebo_read_index(offsets, index_type, bags[k]))
        return EBO_ERR_INVALID_ARG;
    }
  } else {
    if (out_ld != 0 && out_ld != sum_d) return EBO_ERR_SHAPE;
    out_ld = sum_d;
    for (int32_t t = 0; t < num_tables; ++t)
      if (!tables[t].data) return EBO_ERR_INVALID_ARG;
  }

  /* Doff[t]: first output column of table t */
  int64_t *doff = (int64_t *)malloc(sizeof(int64_t) * (size_t)num_tables);
  if (!doff) return EBO_ERR_INVALID_ARG;
  doff[0] = 0;
  for (int32_t t = 1; t < num_tables; ++t) doff[t] = doff[t - 1] + tables[t - 1].dim;

  int nthreads = 1;
#ifdef _OPENMP
  nthreads = num_threads > 0 ? num_threads : omp_get_max_threads();
#endif
  (void)nthreads;
#pragma omp parallel for schedule(dynamic, 16) num_threads(nthreads)
  for (int64_t k = 0; k < count; ++k) {
    int64_t g = bags ? bags[k] : k;
    int64_t t = g / B, b = g % B;
    int64_t pos = bags ? k * out_ld : b * out_ld + doff[t];
    ebo_pool_bag(&tables[t], indices, index_type, ebo_read_index(offsets, index_type, g),
                 ebo_read_index(offsets, index_type, g + 1), weights, mode, out + pos,
                 asum ? asum + pos : NULL);
  }
  free(doff);
  return EBO_OK;
}

/* Number of threads a parallel region would use when num_threads <= 0. */
int ebo_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ========================================================================
 * Backward with a fused row-wise optimizer update (test infrastructure).
 *
 * The paper's component benchmark profiles both the forward and the
 * backward pass of each submodule (Sec. III-A); for sparse_arch the backward
 * is the gradient of the pooled lookup with respect to the table rows,
 * followed by the optimizer's sparse update of the rows that were read.
 * With c_i = w_i (weighted sum), 1 (sum) or 1/L (mean, L = the bag's length),
 * for every table t and every row r that occurs in the batch:
 *
 *   G[d] = sum over positions i of table t with idx_i = r of
 *          c_i * grad_out[b(i), Doff[t] + d]          (fp64, in position order)
 *   SGD:                 W[r] <- W[r] - lr * G
 *   row-wise Adagrad:    s[r] <- s[r] + (1/D) sum_d G[d]^2
 *                        W[r] <- W[r] - lr * G / (sqrt(s[r]) + eps)
 *
 * computed in fp64 from the stored values and rounded once to the table's
 * storage type (and s to fp32).  Rows that do not occur are left alone.
 * Only fp32 and fp16 tables train; the optimizer and its state layout are
 * readings (the paper names neither).
 * ======================================================================== */

/* double -> IEEE binary16, round to nearest even, from the bit-level
 * definition (normal, subnormal, overflow to infinity, NaN). */
uint16_t ebo_double_to_half(double x) {
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs(x);
  if (isnan(x)) return 0x7E00;
  if (a >= 65520.0) return sign | 0x7C00; /* at or past max + half ulp: infinity */
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: value = m * 2^-24, m in [0, 1024] (1024 = smallest normal) */
    double m = a * ldexp(1.0, 24);
    double f = floor(m);
    double rem = m - f;
    uint32_t mi = (uint32_t)f;
    if (rem > 0.5 || (rem == 0.5 && (mi & 1u))) ++mi;
    return sign | (uint16_t)mi; /* mi = 1024 encodes the smallest normal */
  }
  int e;
  double fr = frexp(a, &e); /* a = fr * 2^e, fr in [0.5, 1) */
  /* a = 1.m * 2^(e-1); significand with 10 fraction bits: fr * 2^11 in [1024, 2048) */
  double m = ldexp(fr, 11);
  double f = floor(m);
  double rem = m - f;
  uint32_t mi = (uint32_t)f;
  if (rem > 0.5 || (rem == 0.5 && (mi & 1u))) ++mi;
  int ex = e - 1 + 15;
  if (mi == 2048) { mi = 1024; ++ex; }
  if (ex >= 31) return sign | 0x7C00;
  return sign | (uint16_t)((ex << 10) | (mi - 1024));
}

typedef struct {
  int64_t row; /* row number */
  int64_t pos; /* position in indices */
  int64_t bag; /* global bag id g */
} ebo_occ;

static int ebo_occ_cmp(const void *pa, const void *pb) {
  const ebo_occ *a = (const ebo_occ *)pa, *b = (const ebo_occ *)pb;
  if (a->row != b->row) return a->row < b->row ? -1 : 1;
  return a->pos < b->pos ? -1 : (a->pos > b->pos ? 1 : 0);
}

/* Optional per-table report of the touched rows: row ids (ascending), G and
 * S = sum_i |c_i g| per element (fp64, [rows x D]) and occurrence counts.
 * Arrays must hold at least as many rows as the table has positions. */
typedef struct {
  int64_t *rows;
  double *grad;
  double *scale;
  int64_t *count;
  int64_t num_rows; /* out */
} ebo_row_report;

#define EBO_OPT_SGD 0
#define EBO_OPT_ROWWISE_ADAGRAD 1

/*
 * tables: writable rows (data == NULL: table skipped, left alone);
 * grad_out: [B, sum D] fp32; state: fp32, table t's rows at
 * state + sum_{s<t} R_s (row-wise Adagrad only, else NULL);
 * reports: NULL or one entry per table (entries may have rows == NULL).
 */
int ebo_backward_update(const ebo_table *tables, int32_t num_tables, const void *indices,
                        const void *offsets, int32_t index_type, int64_t num_indices,
                        int64_t num_offsets, const float *weights, int32_t mode,
                        const float *grad_out, int32_t opt, float lr, float eps, float *state,
                        ebo_row_report *reports, int32_t num_threads) {
  if (!tables || num_tables < 1 || !offsets || !grad_out) return EBO_ERR_INVALID_ARG;
  if (num_indices < 0 || (num_indices > 0 && !indices)) return EBO_ERR_INVALID_ARG;
  if (index_type != EBO_IDX_I32 && index_type != EBO_IDX_I64) return EBO_ERR_DTYPE;
  if (mode != EBO_MODE_SUM && mode != EBO_MODE_MEAN) return EBO_ERR_INVALID_ARG;
  if (weights && mode == EBO_MODE_MEAN) return EBO_ERR_INVALID_ARG;
  if (opt != EBO_OPT_SGD && opt != EBO_OPT_ROWWISE_ADAGRAD) return EBO_ERR_INVALID_ARG;
  if (opt == EBO_OPT_ROWWISE_ADAGRAD && !state) return EBO_ERR_INVALID_ARG;
  if (num_offsets < 2 || (num_offsets - 1) % num_tables != 0) return EBO_ERR_SHAPE;
  const int64_t B = (num_offsets - 1) / num_tables;
  const int64_t nbags = num_offsets - 1;
  int64_t sum_d = 0;
  for (int32_t t = 0; t < num_tables; ++t) {
    if (tables[t].dtype != EBO_ROW_F32 && tables[t].dtype != EBO_ROW_F16) return EBO_ERR_DTYPE;
    if (tables[t].dim < 1 || tables[t].num_rows < 1) return EBO_ERR_INVALID_ARG;
    sum_d += tables[t].dim;
  }
  if (ebo_read_index(offsets, index_type, 0) != 0) return EBO_ERR_OFFSETS;
  for (int64_t g = 0; g < nbags; ++g)
    if (ebo_read_index(offsets, index_type, g + 1) < ebo_read_index(offsets, index_type, g))
      return EBO_ERR_OFFSETS;
  if (ebo_read_index(offsets, index_type, nbags) != num_indices) return EBO_ERR_OFFSETS;
  for (int32_t t = 0; t < num_tables; ++t) {
    int64_t lo = ebo_read_index(offsets, index_type, (int64_t)t * B);
    int64_t hi = ebo_read_index(offsets, index_type, (int64_t)(t + 1) * B);
    for (int64_t i = lo; i < hi; ++i) {
      int64_t r = ebo_read_index(indices, index_type, i);
      if (r < 0 || r >= tables[t].num_rows) return EBO_ERR_INDEX_OOB;
    }
  }

  int nthreads = 1;
#ifdef _OPENMP
  nthreads = num_threads > 0 ? num_threads : omp_get_max_threads();
#endif
  (void)nthreads;
  int64_t doff = 0, state_base = 0;
  for (int32_t t = 0; t < num_tables; ++t) {
    const ebo_table *tb = &tables[t];
    const int32_t D = tb->dim;
    int64_t lo = ebo_read_index(offsets, index_type, (int64_t)t * B);
    int64_t hi = ebo_read_index(offsets, index_type, (int64_t)(t + 1) * B);
    int64_t n = hi - lo;
    ebo_row_report *rep = reports ? &reports[t] : NULL;
    if (rep) rep->num_rows = 0;
    if (tb->data && n > 0) {
      /* every occurrence of table t: (row, position, bag), sorted by row then position */
      ebo_occ *occ = (ebo_occ *)malloc(sizeof(ebo_occ) * (size_t)n);
      if (!occ) return EBO_ERR_INVALID_ARG;
      int64_t k = 0;
      for (int64_t g = (int64_t)t * B; g < (int64_t)(t + 1) * B; ++g)
        for (int64_t i = ebo_read_index(offsets, index_type, g);
             i < ebo_read_index(offsets, index_type, g + 1); ++i) {
          occ[k].row = ebo_read_index(indices, index_type, i);
          occ[k].pos = i;
          occ[k].bag = g;
          ++k;
        }
      qsort(occ, (size_t)n, sizeof(ebo_occ), ebo_occ_cmp);
      /* run starts */
      int64_t *starts = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1));
      int64_t nruns = 0;
      for (int64_t j = 0; j < n; ++j)
        if (j == 0 || occ[j].row != occ[j - 1].row) starts[nruns++] = j;
      starts[nruns] = n;
      if (rep) rep->num_rows = nruns;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads)
      for (int64_t u = 0; u < nruns; ++u) {
        const int64_t row = occ[starts[u]].row;
        unsigned char *w = (unsigned char *)tb->data + (size_t)row * (size_t)tb->row_stride_bytes;
        double *G = (double *)malloc(sizeof(double) * (size_t)D);
        double *S = (double *)malloc(sizeof(double) * (size_t)D);
        for (int32_t d = 0; d < D; ++d) {
          double acc = 0.0, mag = 0.0;
          for (int64_t j = starts[u]; j < starts[u + 1]; ++j) {
            const ebo_occ *o = &occ[j];
            double c = 1.0;
            if (weights) c = (double)weights[o->pos];
            if (mode == EBO_MODE_MEAN) {
              int64_t L = ebo_read_index(offsets, index_type, o->bag + 1) -
                          ebo_read_index(offsets, index_type, o->bag);
              c = 1.0 / (double)L;
            }
            double term = c * (double)grad_out[(o->bag % B) * sum_d + doff + d];
            acc += term;
            mag += fabs(term);
          }
          G[d] = acc;
          S[d] = mag;
        }
        double step = (double)lr;
        if (opt == EBO_OPT_ROWWISE_ADAGRAD) {
          double sq = 0.0;
          for (int32_t d = 0; d < D; ++d) sq += G[d] * G[d];
          double s_new = (double)state[state_base + row] + sq / (double)D;
          state[state_base + row] = (float)s_new;
          step = (double)lr / (sqrt(s_new) + (double)eps);
        }
        for (int32_t d = 0; d < D; ++d) {
          if (tb->dtype == EBO_ROW_F32) {
            float v;
            memcpy(&v, w + 4 * (size_t)d, 4);
            v = (float)((double)v - step * G[d]);
            memcpy(w + 4 * (size_t)d, &v, 4);
          } else {
            uint16_t h;
            memcpy(&h, w + 2 * (size_t)d, 2);
            h = ebo_double_to_half(ebo_half_to_double(h) - step * G[d]);
            memcpy(w + 2 * (size_t)d, &h, 2);
          }
        }
        if (rep && rep->rows) {
          rep->rows[u] = row;
          rep->count[u] = starts[u + 1] - starts[u];
          for (int32_t d = 0; d < D; ++d) {
            rep->grad[u * D + d] = G[d];
            rep->scale[u * D + d] = S[d];
          }
        }
        free(G);
        free(S);
      }
      free(starts);
      free(occ);
    }
    doff += D;
    state_base += tb->num_rows;
  }
  return EBO_OK;
}

/* ========================================================================
 * Factorization-machine cross term over the pooled embeddings (test
 * infrastructure).
 *
 * The paper's DLRM is DeepFM-based; its inter_arch.fm submodule computes the
 * factorization-machine cross term over the embeddings that sparse_arch
 * produces (Sec. IV-A.2, inter_arch zoom-in), the second-order term of the
 * factorization machine the Introduction cites (Rendle, 2010).  With each
 * categorical feature (field) f of example b represented by its pooled
 * embedding e_{b,f} (D values, all fields the same D), the term is the sum of
 * the inner products of every unordered pair of distinct fields:
 *
 *   y_b = sum_{f < f'} sum_d e_{b,f,d} * e_{b,f',d}
 *
 * pooled is [B, ld] with field f in columns [f*D, f*D + D) (the pooled
 * output's layout).  Every product of two fp32 values is exact in fp64; the
 * pairs are summed in fp64 in (f, f', d) order and returned unrounded.
 *
 * scale (optional): M_b = sum_d (sum_f A_{b,f,d})^2 with A the per-element
 * error scale of the pooled values (asum of ebo_forward), the quantity a
 * computed y_b's rounding error is bounded against.
 * ======================================================================== */
int ebo_fm(const float *pooled, int64_t ld, int32_t num_fields, int32_t dim, int64_t num_examples,
           const double *asum, double *y, double *scale, int32_t num_threads) {
  if (!pooled || !y || num_fields < 1 || dim < 1 || num_examples < 0) return EBO_ERR_INVALID_ARG;
  if (ld < (int64_t)num_fields * dim) return EBO_ERR_SHAPE;
  int nthreads = 1;
#ifdef _OPENMP
  nthreads = num_threads > 0 ? num_threads : omp_get_max_threads();
#endif
  (void)nthreads;
#pragma omp parallel for schedule(dynamic, 16) num_threads(nthreads)
  for (int64_t b = 0; b < num_examples; ++b) {
    const float *e = pooled + b * ld;
    double acc = 0.0;
    for (int32_t f = 0; f < num_fields; ++f)
      for (int32_t g = f + 1; g < num_fields; ++g)
        for (int32_t d = 0; d < dim; ++d)
          acc += (double)e[(int64_t)f * dim + d] * (double)e[(int64_t)g * dim + d];
    y[b] = acc;
    if (scale) {
      const double *a = asum + b * ld;
      double m = 0.0;
      for (int32_t d = 0; d < dim; ++d) {
        double col = 0.0;
        for (int32_t f = 0; f < num_fields; ++f) col += a[(int64_t)f * dim + d];
        m += col * col;
      }
      scale[b] = m;
    }
  }
  return EBO_OK;
}

/* ========================================================================
 * Un-pooled (sequence) lookup (test infrastructure).
 *
 * Sequence recommenders (the Introduction names HSTU among the architectures
 * the paper's profiling targets) consume the embedding of every position of a
 * jagged feature instead of a pooled sum.  For every table t and position i
 * in [start_t, end_t) = [offsets[t*B], offsets[(t+1)*B]):
 *
 *   out[base_t + (i - start_t) * D_t + d] = x(t, idx[i], d)
 *
 * with base_t = sum_{s<t} N_s * D_s, N_s = end_s - start_s: table t's
 * positions form a [N_t, D_t] row-major block, the blocks in table order
 * ([N, D] when every table has the same D).  x is the fp32 element value of
 * the pooled lookup (the stored value, the exact widening of a binary16, or
 * fp32(s*q + c) for int8 row-wise rows).
 * out_numel must equal sum_t N_t * D_t (else EBO_ERR_SHAPE).
 * ======================================================================== */
int ebo_forward_seq(const ebo_table *tables, int32_t num_tables, const void *indices,
                    const void *offsets, int32_t index_type, int64_t num_indices,
                    int64_t num_offsets, float *out, int64_t out_numel, int32_t num_threads) {
  if (!tables || num_tables < 1 || !offsets || (!out && out_numel > 0)) return EBO_ERR_INVALID_ARG;
  if (num_indices < 0 || (num_indices > 0 && !indices)) return EBO_ERR_INVALID_ARG;
  if (index_type != EBO_IDX_I32 && index_type != EBO_IDX_I64) return EBO_ERR_DTYPE;
  if (num_offsets < 2 || (num_offsets - 1) % num_tables != 0) return EBO_ERR_SHAPE;
  const int64_t B = (num_offsets - 1) / num_tables;
  const int64_t nbags = num_offsets - 1;
  for (int32_t t = 0; t < num_tables; ++t) {
    const ebo_table *tb = &tables[t];
    if (tb->dtype != EBO_ROW_F32 && tb->dtype != EBO_ROW_F16 && tb->dtype != EBO_ROW_U8 &&
        tb->dtype != EBO_ROW_U8_SPLIT)
      return EBO_ERR_DTYPE;
    if (tb->dim < 1 || tb->num_rows < 1 || !tb->data) return EBO_ERR_INVALID_ARG;
  }
  if (ebo_read_index(offsets, index_type, 0) != 0) return EBO_ERR_OFFSETS;
  for (int64_t g = 0; g < nbags; ++g)
    if (ebo_read_index(offsets, index_type, g + 1) < ebo_read_index(offsets, index_type, g))
      return EBO_ERR_OFFSETS;
  if (ebo_read_index(offsets, index_type, nbags) != num_indices) return EBO_ERR_OFFSETS;

  int64_t *base = (int64_t *)malloc(sizeof(int64_t) * (size_t)(num_tables + 1));
  if (!base) return EBO_ERR_INVALID_ARG;
  base[0] = 0;
  for (int32_t t = 0; t < num_tables; ++t) {
    int64_t lo = ebo_read_index(offsets, index_type, (int64_t)t * B);
    int64_t hi = ebo_read_index(offsets, index_type, (int64_t)(t + 1) * B);
    for (int64_t i = lo; i < hi; ++i) {
      int64_t r = ebo_read_index(indices, index_type, i);
      if (r < 0 || r >= tables[t].num_rows) {
        free(base);
        return EBO_ERR_INDEX_OOB;
      }
    }
    base[t + 1] = base[t] + (hi - lo) * tables[t].dim;
  }
  if (base[num_tables] != out_numel) {
    free(base);
    return EBO_ERR_SHAPE;
  }

  int nthreads = 1;
#ifdef _OPENMP
  nthreads = num_threads > 0 ? num_threads : omp_get_max_threads();
#endif
  (void)nthreads;
  for (int32_t t = 0; t < num_tables; ++t) {
    const ebo_table *tb = &tables[t];
    const int64_t lo = ebo_read_index(offsets, index_type, (int64_t)t * B);
    const int64_t hi = ebo_read_index(offsets, index_type, (int64_t)(t + 1) * B);
#pragma omp parallel for schedule(static) num_threads(nthreads)
    for (int64_t i = lo; i < hi; ++i) {
      const int64_t r = ebo_read_index(indices, index_type, i);
      float *dst = out + base[t] + (i - lo) * tb->dim;
      for (int32_t d = 0; d < tb->dim; ++d) dst[d] = ebo_element(tb, r, d);
    }
  }
  free(base);
  return EBO_OK;
}
