/*
 * Oracle for the tiled GEMM C = A B -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain definition of the product the warp-specialised kernel
 * computes (paper, Background, "General Matrix Multiplication": A is M x K,
 * B is K x N, C = A B is M x N).  Tiling and the producer/consumer split
 * reorder the work but not the mathematics, so the oracle ignores both and
 * evaluates C[i][j] = sum_k A[i][k] * B[k][j] directly, in double precision.
 *
 * Inputs are the raw 16-bit patterns of the rounded operands (row-major A with
 * K columns, row-major B with N columns), decoded here by field extraction
 * from the format definitions.  Products of two 16-bit floats are exact in
 * double; the sums carry at most ~K * 2^-53 relative error.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this code.  It shares nothing with the GPU library.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_F16 0
#define ORACLE_BF16 1

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
double oracle_decode_f16(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int f = h & 0x3ff;
  double v;
  if (e == 0)
    v = ldexp((double)f, -24); /* subnormal: f * 2^(1-15-10) */
  else if (e == 31)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(f | 0x400), e - 25); /* (1 + f/2^10) * 2^(e-15) */
  return sign ? -v : v;
}

/* bfloat16: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits. */
double oracle_decode_bf16(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 7) & 0xff;
  int f = h & 0x7f;
  double v;
  if (e == 0)
    v = ldexp((double)f, -133); /* subnormal: f * 2^(1-127-7) */
  else if (e == 255)
    v = f ? NAN : INFINITY;
  else
    v = ldexp((double)(f | 0x80), e - 134); /* (1 + f/2^7) * 2^(e-127) */
  return sign ? -v : v;
}

static double decode(uint16_t h, int dtype) {
  return dtype == ORACLE_BF16 ? oracle_decode_bf16(h) : oracle_decode_f16(h);
}

/* Decode n patterns into doubles.  Returns 0, or -1 on a bad dtype. */
int oracle_decode(const uint16_t* bits, int64_t n, int dtype, double* out) {
  if (dtype != ORACLE_F16 && dtype != ORACLE_BF16) return -1;
  for (int64_t i = 0; i < n; i++) out[i] = decode(bits[i], dtype);
  return 0;
}

/*
 * For every requested row i = rows[r] (0 <= i < M) write
 *   C[r][j]     = sum_k A[i][k] * B[k][j]
 *   absAB[r][j] = sum_k |A[i][k]| * |B[k][j]|     (absAB may be NULL)
 * for j in [0, N).  C and absAB are nrows x N, row-major, caller-owned.
 * B is decoded once into a K x N double array; each row of A is decoded as it
 * is used.  Rows are independent and are shared out over nthreads OpenMP
 * threads (nthreads <= 0 leaves the OpenMP default).
 * Returns 0, -1 on a bad argument, -2 if memory runs out.
 */
int oracle_gemm_rows(int64_t M, int64_t N, int64_t K, const uint16_t* A, const uint16_t* B,
                     int dtype, int64_t nrows, const int64_t* rows, double* C, double* absAB,
                     int nthreads) {
  if (M < 0 || N < 0 || K < 0 || nrows < 0) return -1;
  if (dtype != ORACLE_F16 && dtype != ORACLE_BF16) return -1;
  for (int64_t r = 0; r < nrows; r++)
    if (rows[r] < 0 || rows[r] >= M) return -1;
  if (nrows == 0 || N == 0) return 0;
  double* Bd = (double*)malloc(sizeof(double) * (size_t)(K > 0 ? K * N : 1));
  if (!Bd) return -2;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static)
#endif
  for (int64_t x = 0; x < K * N; x++) Bd[x] = decode(B[x], dtype);
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1)
#endif
  for (int64_t r = 0; r < nrows; r++) {
    int64_t i = rows[r];
    double* c = C + r * N;
    double* s = absAB ? absAB + r * N : NULL;
    for (int64_t j = 0; j < N; j++) c[j] = 0.0;
    if (s)
      for (int64_t j = 0; j < N; j++) s[j] = 0.0;
    for (int64_t k = 0; k < K; k++) {
      double a = decode(A[i * K + k], dtype);
      const double* b = Bd + k * N;
#ifdef ORACLE_PLANT_DROP_LAST_K /* planted mistake, used only by the pin self-test */
      if (k == K - 1) break;
#endif
      for (int64_t j = 0; j < N; j++) {
#ifdef ORACLE_PLANT_TRANSPOSE_B /* planted mistake: reads B[j][k] on square shapes */
        double bb = (K == N) ? Bd[j * N + k] : b[j];
#else
        double bb = b[j];
#endif
#ifdef ORACLE_PLANT_SIGN /* planted mistake: subtracts odd-k terms */
        c[j] += (k & 1) ? -a * bb : a * bb;
#else
        c[j] += a * bb;
#endif
      }
      if (s) {
        double aa = fabs(a);
        for (int64_t j = 0; j < N; j++) s[j] += aa * fabs(b[j]);
      }
    }
  }
  free(Bd);
  return failed;
}

/* All rows: C (and absAB, may be NULL) are M x N row-major doubles. */
int oracle_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* A, const uint16_t* B, int dtype,
                double* C, double* absAB, int nthreads) {
  if (M < 0) return -1;
  int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(M > 0 ? M : 1));
  if (!rows) return -2;
  for (int64_t i = 0; i < M; i++) rows[i] = i;
  int rc = oracle_gemm_rows(M, N, K, A, B, dtype, M, rows, C, absAB, nthreads);
  free(rows);
  return rc;
}

/* Number of OpenMP threads a parallel region would use (1 without OpenMP). */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
