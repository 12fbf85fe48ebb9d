/*
 * CRVQ CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously-correct fp64 definitions of the quantities the
 * GPU library computes.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's shared object; the
 * product path never does.  It shares no source with the HIP library.
 *
 * Every input array is fp32 (bf16 data is widened to fp32 exactly by the
 * Python wrapper before it gets here); every sum, product and difference
 * is carried out in double precision in the order written, with no FMA
 * contraction (built with -ffp-contract=off, no fast-math).
 *
 * Paper: "CRVQ: Channel-Relaxed Vector Quantization for Extreme
 * Compression of LLMs" (arXiv 2412.09282).
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Squared Euclidean distance in fp64, summed over t = 0..d-1 in ascending
 * order.  The paper's encoding (Sec. 3.1, Eq. 3-4) minimises the L2 norm;
 * its square has the same minimiser. */
static double sqdist(const float* v, const float* c, int d) {
  double acc = 0.0;
  for (int t = 0; t < d; ++t) {
    double diff = (double)v[t] - (double)c[t];
    acc = acc + diff * diff;
  }
  return acc;
}

/* Nearest-codeword encoding, Sec. 3.1 Eq. 3-4:
 *   q_i = argmin_j || w_i - c_j ||,  ties broken towards the lowest j.
 * V is n x d (row-major), C is K x d.  dist[i] = the fp64 squared distance
 * to the chosen codeword. */
void oracle_assign(const float* V, int64_t n, int d, const float* C, int64_t K,
                   int32_t* codes, double* dist) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const float* v = V + i * d;
    double best = INFINITY;
    int64_t best_k = 0;
    for (int64_t k = 0; k < K; ++k) {
      double e = sqdist(v, C + k * d, d);
      if (e < best) { /* strict: equal distances keep the lower index */
        best = e;
        best_k = k;
      }
    }
    codes[i] = (int32_t)best_k;
    if (dist) dist[i] = best;
  }
}

/* One Lloyd update of the K-means codebook of Sec. 3.1 Eq. 2:
 *   c_k = (sum of the vectors v with q_v = k, in ascending v) / count_k,
 * all in fp64.  A cluster with no members keeps its previous centroid
 * (C_old).  means[k*d+t] receives the fp64 mean (or the old value);
 * rounding to the codebook's storage type is done by the caller. */
void oracle_kmeans_means(const float* V, int64_t n, int d, const int32_t* codes, int64_t K,
                         const float* C_old, double* means, int64_t* counts) {
  double* sums = (double*)calloc((size_t)K * (size_t)d, sizeof(double));
  int64_t* cnt = (int64_t*)calloc((size_t)K, sizeof(int64_t));
  for (int64_t i = 0; i < n; ++i) {
    int64_t k = codes[i];
    for (int t = 0; t < d; ++t) sums[k * d + t] = sums[k * d + t] + (double)V[i * d + t];
    cnt[k] += 1;
  }
  for (int64_t k = 0; k < K; ++k) {
    for (int t = 0; t < d; ++t) {
      if (cnt[k] > 0)
        means[k * d + t] = sums[k * d + t] / (double)cnt[k];
      else
        means[k * d + t] = (double)C_old[k * d + t];
    }
    if (counts) counts[k] = cnt[k];
  }
  free(sums);
  free(cnt);
}

/* Column (input-channel) reduction behind the importance metrics of
 * Sec. 4.1 (Eq. 7), Appendix A.2 (Eq. 9-10) and the Hessian diagonal:
 *   out[j] = s_j * R_{i<M} (A[i,j] - B[i,j])^2
 * with R = sum (reduce == 0, rows taken in ascending i) or max (reduce ==
 * 1); B may be NULL (treated as 0) and scale may be NULL (s_j = 1). */
void oracle_colreduce(const float* A, int64_t lda, const float* B, int64_t ldb, int64_t M,
                      int64_t N, const double* scale, int reduce, double* out) {
  /* Every thread owns a contiguous range of columns and walks the rows in ascending i, so each
   * column is still reduced in row order while the matrix is read row by row. */
#pragma omp parallel
  {
    int64_t nt = 1, id = 0;
#ifdef _OPENMP
    nt = omp_get_num_threads();
    id = omp_get_thread_num();
#endif
    int64_t j0 = N * id / nt, j1 = N * (id + 1) / nt;
    double* acc = (double*)calloc((size_t)(j1 - j0 + 1), sizeof(double));
    for (int64_t i = 0; i < M; ++i) {
      for (int64_t j = j0; j < j1; ++j) {
        double x = (double)A[i * lda + j];
        if (B) x = x - (double)B[i * ldb + j];
        double sq = x * x;
        if (reduce == 0)
          acc[j - j0] = acc[j - j0] + sq;
        else if (sq > acc[j - j0])
          acc[j - j0] = sq;
      }
    }
    for (int64_t j = j0; j < j1; ++j) out[j] = scale ? scale[j] * acc[j - j0] : acc[j - j0];
    free(acc);
  }
}

/* Sequential residual beam search over n_books additive codebooks
 * (Sec. 3.1 "beam search ... multi-step encoding"; Sec. 4.3 additive
 * extended codebooks; Alg. 1 BeamSearchOptimize under the squared
 * Euclidean objective).
 *
 * For each vector x: start from one empty tuple whose residual is x.  For
 * book t, every kept tuple (parent, with residual r) is extended by every
 * codeword c of book t; the candidate's key is
 *   ( sum_j (r_j - c_j)^2 in fp64 , rank of the parent , codeword index )
 * and the `beam` smallest keys survive, ranked by that key.  A survivor's
 * residual is r - c, computed component-wise in fp64.  The answer is the
 * rank-0 tuple after the last book; err is its key's first component.
 *
 * books[t] is Ks[t] x d.  codes is n_books arrays of n entries laid out as
 * codes[t*n + i]. */
typedef struct {
  double e;
  int32_t parent;
  int32_t code;
} cand_t;

static int cand_less(const cand_t* a, const cand_t* b) {
  if (a->e != b->e) return a->e < b->e;
  if (a->parent != b->parent) return a->parent < b->parent;
  return a->code < b->code;
}

void oracle_beam(const float* V, int64_t n, int d, int n_books, const float* const* books,
                 const int64_t* Ks, int beam, int32_t* codes, double* err) {
#pragma omp parallel
  {
    double* res = (double*)malloc(sizeof(double) * (size_t)beam * (size_t)d);
    double* res_new = (double*)malloc(sizeof(double) * (size_t)beam * (size_t)d);
    int32_t* tup = (int32_t*)malloc(sizeof(int32_t) * (size_t)beam * (size_t)n_books);
    int32_t* tup_new = (int32_t*)malloc(sizeof(int32_t) * (size_t)beam * (size_t)n_books);
    cand_t* keep = (cand_t*)malloc(sizeof(cand_t) * (size_t)(beam + 1));
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < n; ++i) {
      int n_par = 1;
      for (int t = 0; t < d; ++t) res[t] = (double)V[i * d + t];
      double last_e = 0.0;
      for (int b = 0; b < n_books; ++b) {
        const float* Cb = books[b];
        int n_keep = 0;
        for (int p = 0; p < n_par; ++p) {
          const double* r = res + (size_t)p * d;
          for (int64_t k = 0; k < Ks[b]; ++k) {
            cand_t c;
            c.e = 0.0;
            for (int t = 0; t < d; ++t) {
              double diff = r[t] - (double)Cb[k * d + t];
              c.e = c.e + diff * diff;
            }
            c.parent = p;
            c.code = (int32_t)k;
            /* insertion into the sorted list of the best `beam` keys */
            if (n_keep < beam || cand_less(&c, &keep[n_keep - 1])) {
              int pos = n_keep < beam ? n_keep : beam - 1;
              while (pos > 0 && cand_less(&c, &keep[pos - 1])) {
                keep[pos] = keep[pos - 1];
                --pos;
              }
              keep[pos] = c;
              if (n_keep < beam) ++n_keep;
            }
          }
        }
        for (int s = 0; s < n_keep; ++s) {
          const double* r = res + (size_t)keep[s].parent * d;
          const float* c = Cb + (int64_t)keep[s].code * d;
          for (int t = 0; t < d; ++t) res_new[(size_t)s * d + t] = r[t] - (double)c[t];
          for (int bb = 0; bb < b; ++bb)
            tup_new[(size_t)s * n_books + bb] = tup[(size_t)keep[s].parent * n_books + bb];
          tup_new[(size_t)s * n_books + b] = keep[s].code;
        }
        memcpy(res, res_new, sizeof(double) * (size_t)n_keep * d);
        memcpy(tup, tup_new, sizeof(int32_t) * (size_t)n_keep * n_books);
        n_par = n_keep;
        last_e = keep[0].e;
      }
      for (int b = 0; b < n_books; ++b) codes[(int64_t)b * n + i] = tup[b];
      if (err) err[i] = last_e;
    }
    free(res);
    free(res_new);
    free(tup);
    free(tup_new);
    free(keep);
  }
}

/* Additive reconstruction (Sec. 4.3: a critical vector is the sum of its
 * codewords from the basic and all extended codebooks; non-critical
 * vectors use the basic codebook only).
 *   R[i,t] = sum over books b = 0..nb_i-1 of books[b][codes[b][i], t]
 * in fp64, in book order; nb_i = n_books when crit[i] != 0, else n_full (the
 * basic books, 1 unless the layout has several).  codes is n_books arrays of
 * n entries (codes[b*n + i]); entries of books b >= n_full are ignored for
 * non-critical vectors. */
void oracle_reconstruct(int64_t n, int d, int n_books, int n_full, const float* const* books,
                        const int32_t* codes, const uint8_t* crit, double* R) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    int nb = crit[i] ? n_books : n_full;
    for (int t = 0; t < d; ++t) {
      double acc = 0.0;
      for (int b = 0; b < nb; ++b) {
        int64_t k = codes[(int64_t)b * n + i];
        acc = acc + (double)books[b][k * d + t];
      }
      R[i * d + t] = acc;
    }
  }
}

/* Round fp64 values to the nearest bfloat16 (8 significant bits, 8-bit
 * exponent), ties to even, by the definition: scale the significand to
 * [128, 256), round to the nearest integer (nearbyint uses the current
 * rounding mode, round-to-nearest-even by default), scale back.  Values
 * below the smallest normal use the fixed subnormal quantum 2^-133.
 * Returns the bf16 bit patterns. */
uint16_t oracle_bf16_bits_of(double x) {
  float f;
  if (isnan(x)) {
    f = NAN;
  } else if (x == 0.0 || isinf(x)) {
    f = (float)x;
  } else {
    double ax = fabs(x), r;
    if (ax < ldexp(1.0, -126)) {
      r = ldexp(nearbyint(ldexp(ax, 133)), -133);
    } else {
      int e;
      double m = frexp(ax, &e); /* ax = m * 2^e, m in [0.5, 1) */
      r = ldexp(nearbyint(ldexp(m, 8)), e - 8);
    }
    /* largest finite bf16 is (2 - 2^-7) * 2^127; anything that rounds past it overflows */
    if (r > ldexp(255.0, 120)) r = INFINITY;
    f = (float)(x < 0 ? -r : r); /* exact: r is a bf16 value */
  }
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

void oracle_round_bf16(const double* x, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16_bits_of(x[i]);
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Host threads of the parallel loops from now on (n >= 1); for timing the oracle on fewer cores. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
