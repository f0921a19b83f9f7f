/*
 * Plain CPU oracle for batched HDC inference.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the bench's CPU
 * baseline leg do. It shares no code, header or constant with the GPU
 * library.
 *
 * What it computes (ScalableHD, Sec. II-D, Eq. 7-9 and Alg. 1):
 *   v[n,d] = sum_f X[n,f] * B[f,d]                 (Eq. 2 per sample, Eq. 7)
 *   H[n,d] = HardSign(v[n,d])                      (Eq. 1 / Eq. 3)
 *   S[n,k] = sum_d H[n,d] * C[k,d]                 (Eq. 5 per sample, Eq. 8)
 *   y[n]   = argmax_k S[n,k]                       (Eq. 6 / Eq. 9)
 * The paper's blocked Stage I / Stage II algorithms only re-associate these
 * sums, so the oracle is the plain definition with no blocking, fusion or
 * reordering: loops in the order of the definition, float64 accumulation.
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - HardSign(0) = +1 exactly as Eq. 1 states (a literal v >= 0 test, so
 *     -0.0 maps to +1 and NaN maps to -1).
 *   - argmax ties go to the lowest class index.
 *   - similarity is the raw inner product (Sec. II, Eq. 5): no normalisation.
 *   - act = 1 ("identity") skips HardSign, a linear test mode in which
 *     S = X B C^T; the paper's nonlinear encoding always applies HardSign.
 *
 * Inputs are float64 arrays holding the exact values the GPU receives
 * (fp32 or bf16 values widened exactly); every product of two such values is
 * exact in float64, so the only rounding is in the float64 sums.
 *
 * Extra outputs used by the tests' tolerance rule:
 *   A[n,d] = sum_f |X[n,f]| * |B[f,d]|  (the scale of the encoding sum, which
 *   bounds how far any fp32 summation order can move v[n,d]).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Eq. 1: +1 if x >= 0, otherwise -1. */
static double hardsign(double x) { return (x >= 0.0) ? 1.0 : -1.0; }

/* Eq. 2 for one sample: bind each feature scalar to its base hypervector
 * (scalar times row f of B) and bundle the bound vectors (elementwise sum). */
static void encode_sample(const double *x, const double *B, int64_t F, int64_t D,
                          double *v, double *a) {
  for (int64_t d = 0; d < D; ++d) {
    v[d] = 0.0;
    if (a) a[d] = 0.0;
  }
  for (int64_t f = 0; f < F; ++f) {
    const double xf = x[f];
    const double *bf = B + f * D;
    for (int64_t d = 0; d < D; ++d) v[d] += xf * bf[d];
    if (a) {
      const double ax = fabs(xf);
      for (int64_t d = 0; d < D; ++d) a[d] += ax * fabs(bf[d]);
    }
  }
}

/* Eq. 5 and Eq. 6 for one sample: inner product with every class
 * hypervector, then the first index of the maximum. */
static int32_t classify_sample(const double *h, const double *C, int64_t D, int64_t K,
                               double *s) {
  int32_t best = 0;
  for (int64_t k = 0; k < K; ++k) {
    const double *ck = C + k * D;
    double acc = 0.0;
    for (int64_t d = 0; d < D; ++d) acc += h[d] * ck[d];
    s[k] = acc;
    if (k > 0 && acc > s[best]) best = (int32_t)k;
  }
  return best;
}

static int pick_threads(int nthreads) {
#ifdef _OPENMP
  return nthreads > 0 ? nthreads : omp_get_max_threads();
#else
  (void)nthreads;
  return 1;
#endif
}

/* Stage I alone (Eq. 7, Eq. 1): H = act(X B). Any of V, A, H may be NULL.
 * Returns 0 on success, -1 on a bad argument or allocation failure. */
int oracle_encode(const double *X, const double *B, int64_t N, int64_t F, int64_t D,
                  int act, double *V, double *A, double *H, int nthreads) {
  if (!X || !B || N < 0 || F < 1 || D < 1) return -1;
  int err = 0;
  const int nt = pick_threads(nthreads);
#pragma omp parallel num_threads(nt) reduction(| : err)
  {
    double *v = (double *)malloc(sizeof(double) * (size_t)D);
    double *a = (double *)malloc(sizeof(double) * (size_t)D);
    if (!v || !a) {
      err |= 1;
    } else {
#pragma omp for schedule(static)
      for (int64_t n = 0; n < N; ++n) {
        encode_sample(X + n * F, B, F, D, v, A ? a : NULL);
        for (int64_t d = 0; d < D; ++d) {
          if (V) V[n * D + d] = v[d];
          if (A) A[n * D + d] = a[d];
          if (H) H[n * D + d] = act ? v[d] : hardsign(v[d]);
        }
      }
    }
    free(v);
    free(a);
  }
  return err ? -1 : 0;
}

/* Stage II alone (Eq. 8, Eq. 9) on a given real matrix H[N, D]. S may be NULL. */
int oracle_similarity(const double *H, const double *C, int64_t N, int64_t D, int64_t K,
                      double *S, int32_t *y, int nthreads) {
  if (!H || !C || !y || N < 0 || D < 1 || K < 1) return -1;
  int err = 0;
  const int nt = pick_threads(nthreads);
#pragma omp parallel num_threads(nt) reduction(| : err)
  {
    double *s = (double *)malloc(sizeof(double) * (size_t)K);
    if (!s) {
      err |= 1;
    } else {
#pragma omp for schedule(static)
      for (int64_t n = 0; n < N; ++n) {
        y[n] = classify_sample(H + n * D, C, D, K, s);
        if (S)
          for (int64_t k = 0; k < K; ++k) S[n * K + k] = s[k];
      }
    }
    free(s);
  }
  return err ? -1 : 0;
}

/* Alg. 1 end to end for the rows listed in `rows` (or all N rows when rows is
 * NULL; then nrows must equal N). Outputs are indexed by position in the row
 * list: y[i], S[i*K + k], V[i*D + d], A[i*D + d]. S, V and A may be NULL. */
int oracle_infer(const double *X, const double *B, const double *C, int64_t N, int64_t F,
                 int64_t D, int64_t K, int act, const int64_t *rows, int64_t nrows,
                 int32_t *y, double *S, double *V, double *A, int nthreads) {
  if (!X || !B || !C || !y || N < 0 || F < 1 || D < 1 || K < 1 || nrows < 0) return -1;
  if (!rows && nrows != N) return -1;
  if (rows)
    for (int64_t i = 0; i < nrows; ++i)
      if (rows[i] < 0 || rows[i] >= N) return -1;
  int err = 0;
  const int nt = pick_threads(nthreads);
#pragma omp parallel num_threads(nt) reduction(| : err)
  {
    double *v = (double *)malloc(sizeof(double) * (size_t)D);
    double *a = (double *)malloc(sizeof(double) * (size_t)D);
    double *h = (double *)malloc(sizeof(double) * (size_t)D);
    double *s = (double *)malloc(sizeof(double) * (size_t)K);
    if (!v || !a || !h || !s) {
      err |= 1;
    } else {
#pragma omp for schedule(static)
      for (int64_t i = 0; i < nrows; ++i) {
        const int64_t n = rows ? rows[i] : i;
        /* Stage I: Feature Encoding */
        encode_sample(X + n * F, B, F, D, v, A ? a : NULL);
        for (int64_t d = 0; d < D; ++d) h[d] = act ? v[d] : hardsign(v[d]);
        /* Stage II: Similarity Search & Classification */
        y[i] = classify_sample(h, C, D, K, s);
        if (S)
          for (int64_t k = 0; k < K; ++k) S[i * K + k] = s[k];
        if (V) memcpy(V + i * D, v, sizeof(double) * (size_t)D);
        if (A) memcpy(A + i * D, a, sizeof(double) * (size_t)D);
      }
    }
    free(v);
    free(a);
    free(h);
    free(s);
  }
  return err ? -1 : 0;
}

/* Single-pass training (Sec. II-C): the class codebook row of class k is the
 * normalised bundle (Sec. II-A bundling, then HardSign) of the encoded
 * hypervectors (Eq. 2-3) of the samples labelled k:
 *   counts[k,d] = sum over n with y[n] == k of HardSign(v[n,d])
 *   M[k,d]      = HardSign(counts[k,d])
 * A class with no sample, or a tied count, gives +1 (Eq. 1: ties to +1).
 * Samples whose label lies outside [0, K) are skipped. counts are int64
 * (exact); M may be NULL. Samples are encoded in parallel, chunk by chunk,
 * and added in sample order. */
int oracle_bundle(const double *X, const double *B, const int32_t *y, int64_t N, int64_t F,
                  int64_t D, int64_t K, int64_t *counts, double *M, int nthreads) {
  if (!X || !B || !y || !counts || N < 0 || F < 1 || D < 1 || K < 1) return -1;
  for (int64_t i = 0; i < K * D; ++i) counts[i] = 0;
  const int64_t chunk = 64;
  double *h = (double *)malloc(sizeof(double) * (size_t)(chunk * D));
  if (!h) return -1;
  int err = 0;
  const int nt = pick_threads(nthreads);
  for (int64_t n0 = 0; n0 < N && !err; n0 += chunk) {
    const int64_t n1 = n0 + chunk < N ? n0 + chunk : N;
#pragma omp parallel num_threads(nt) reduction(| : err)
    {
      double *v = (double *)malloc(sizeof(double) * (size_t)D);
      if (!v) {
        err |= 1;
      } else {
#pragma omp for schedule(static)
        for (int64_t n = n0; n < n1; ++n) {
          encode_sample(X + n * F, B, F, D, v, NULL);
          for (int64_t d = 0; d < D; ++d) h[(n - n0) * D + d] = hardsign(v[d]);
        }
      }
      free(v);
    }
    for (int64_t n = n0; n < n1; ++n) {
      const int32_t k = y[n];
      if (k < 0 || k >= K) continue;
      for (int64_t d = 0; d < D; ++d) counts[k * D + d] += (int64_t)h[(n - n0) * D + d];
    }
  }
  free(h);
  if (M)
    for (int64_t i = 0; i < K * D; ++i) M[i] = hardsign((double)counts[i]);
  return err ? -1 : 0;
}

/* Number of threads an OpenMP region started with `nthreads` would use. */
int oracle_threads(int nthreads) { return pick_threads(nthreads); }
