/*
 * CPU oracle for the GEMM + communication-share hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP library.
 *
 * Every routine is the plain definition of what the method computes, written
 * for a reader to check by eye, with no blocking, fusion or reordering:
 *
 *   - GEMM (Background, item 1: C = alpha*op(A)*op(B) + beta*C, read here
 *     with alpha = 1, beta = 0), two definitions: (a) the workload's, the
 *     products accumulated in binary32 in increasing k (each bf16*bf16
 *     product is exact in binary32: 8-bit significands), then rounded once
 *     to bfloat16; (b) the sum accumulated in binary64 (each product exact,
 *     the sum's rounding error far below one bfloat16 step at these
 *     magnitudes: a stand-in for the exact sum), then rounded once to
 *     bfloat16.  Both round to nearest, ties to even.
 *   - Local share of an allreduce (Background, item 2: local gradients are
 *     aggregated across GPUs): element-wise sum of the chunks in binary32,
 *     strict left-to-right order c0 + c1 + ... + c_{n-1}.  The fixed order
 *     and binary32 arithmetic are a requirement of the workload, not of the
 *     paper, which is silent on both.  When this GPU's own term is its bf16
 *     GEMM output, that term comes first, converted exactly to binary32.
 *   - Local share of an alltoall (Background, item 2: tokens are routed
 *     between devices): chunk i of the destination is chunk perm[i] of the
 *     source, byte for byte.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC.
 * On x86-64 binary32 arithmetic is done in SSE registers (FLT_EVAL_METHOD 0),
 * so each float addition below is one IEEE-754 binary32 RNE addition.
 */
#include <float.h>
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#include <omp.h>

#if FLT_EVAL_METHOD != 0
#error "binary32 additions must not be evaluated in a wider format"
#endif

/* bfloat16: the upper 16 bits of an IEEE-754 binary32 value. */
double oracle_bf16_to_double(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/*
 * Round a binary64 value once to bfloat16, ties to even.
 * bfloat16 has 8 significand bits (7 stored) and binary32's exponent range:
 * normal numbers have a spacing of 2^(e-7) in [2^e, 2^(e+1)), e >= -126;
 * below 2^-126 the spacing is fixed at 2^-133 (subnormals).  Magnitudes that
 * round to 2^128 or beyond overflow to infinity.  NaN becomes the quiet NaN
 * 0x7FC0 with the input's sign.
 */
uint16_t oracle_double_to_bf16(double x) {
  uint16_t sign = signbit(x) ? 0x8000u : 0u;
  if (isnan(x)) return (uint16_t)(sign | 0x7FC0u);
  double a = fabs(x);
  if (isinf(a)) return (uint16_t)(sign | 0x7F80u);
  if (a == 0.0) return sign;
  int e2;
  (void)frexp(a, &e2);          /* a = f * 2^e2, f in [0.5, 1) => a in [2^(e2-1), 2^e2) */
  int e = e2 - 1;               /* a in [2^e, 2^(e+1)) */
  if (e < -126) e = -126;       /* subnormal range: fixed spacing 2^-133 */
  double ulp = ldexp(1.0, e - 7);
  double q = rint(a / ulp);     /* default rounding mode: nearest, ties to even */
  double r = q * ulp;
  if (r >= ldexp(1.0, 128)) return (uint16_t)(sign | 0x7F80u);
  float rf = (float)r;          /* exact: r has at most 8 significant bits */
  uint32_t u;
  memcpy(&u, &rf, sizeof u);
  return (uint16_t)(sign | (uint16_t)(u >> 16));
}

/*
 * C[m][n] = bf16( sum_k A[m][k] * Bop[k][n] ) for m in [m0, m1), n in [n0, n1).
 *   A : M x K, row-major bfloat16 bits.
 *   B : b_layout == 0 -> stored N x K row-major, Bop[k][n] = B[n*K + k]
 *                        (op(B) = B^T, the weight layout of a linear layer);
 *       b_layout == 1 -> stored K x N row-major, Bop[k][n] = B[k*N + n].
 *   out : (m1-m0) x (n1-n0) row-major bfloat16 bits.
 * K == 0 gives the empty sum, +0.
 */
void oracle_gemm_bf16_block(const uint16_t *A, const uint16_t *B, int M, int N, int K,
                            int b_layout, int m0, int m1, int n0, int n1, uint16_t *out) {
  (void)M;
  int ncols = n1 - n0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = m0; m < m1; ++m) {
    for (int n = n0; n < n1; ++n) {
      double acc = 0.0;
      for (int k = 0; k < K; ++k) {
        double a = oracle_bf16_to_double(A[(size_t)m * K + k]);
        double b = b_layout == 0 ? oracle_bf16_to_double(B[(size_t)n * K + k])
                                 : oracle_bf16_to_double(B[(size_t)k * N + n]);
        acc += a * b;
      }
      out[(size_t)(m - m0) * ncols + (n - n0)] = oracle_double_to_bf16(acc);
    }
  }
}

/*
 * The same block with the products accumulated in binary32, one addition per
 * k in increasing order (acc = acc + a*b, no fused multiply-add: the build
 * forbids contraction), then rounded once to bfloat16 through binary64 (the
 * widening is exact).
 */
void oracle_gemm_bf16_f32acc_block(const uint16_t *A, const uint16_t *B, int M, int N, int K,
                                   int b_layout, int m0, int m1, int n0, int n1, uint16_t *out) {
  (void)M;
  int ncols = n1 - n0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = m0; m < m1; ++m) {
    for (int n = n0; n < n1; ++n) {
      float acc = 0.0f;
      for (int k = 0; k < K; ++k) {
        float a = (float)oracle_bf16_to_double(A[(size_t)m * K + k]);
        float b = b_layout == 0 ? (float)oracle_bf16_to_double(B[(size_t)n * K + k])
                                : (float)oracle_bf16_to_double(B[(size_t)k * N + n]);
        float p = a * b;
        acc = acc + p;
      }
      out[(size_t)(m - m0) * ncols + (n - n0)] = oracle_double_to_bf16((double)acc);
    }
  }
}

/* out[j] = (((c_0[j] + c_1[j]) + c_2[j]) + ...) + c_{n-1}[j], binary32. */
void oracle_chunk_sum_f32(const float *const *chunks, int nchunks, size_t len, float *out) {
#pragma omp parallel for schedule(static)
  for (long long j = 0; j < (long long)len; ++j) {
    float acc = chunks[0][j];
    for (int c = 1; c < nchunks; ++c) acc = acc + chunks[c][j];
    out[j] = acc;
  }
}

/*
 * The same share when this GPU's own contribution is bf16 (its GEMM output):
 * out[j] = (((own[j] + c_0[j]) + c_1[j]) + ...) + c_{n-1}[j], binary32, with
 * own[j] first made a binary32 by the definition of bfloat16: its 16 bits are
 * the high half of the binary32 word (exact for every value, NaN payloads
 * included).  n may be 0 (out = own as binary32).
 */
void oracle_chunk_sum_own_f32(const uint16_t *own, const float *const *chunks, int nchunks, size_t len,
                              float *out) {
#pragma omp parallel for schedule(static)
  for (long long j = 0; j < (long long)len; ++j) {
    uint32_t w = (uint32_t)own[j] << 16;
    float acc;
    memcpy(&acc, &w, sizeof acc);
    for (int c = 0; c < nchunks; ++c) acc = acc + chunks[c][j];
    out[j] = acc;
  }
}

/* dst[i*chunk_bytes + b] = src[perm[i]*chunk_bytes + b] for b < chunk_bytes. */
void oracle_permute(const uint8_t *src, uint8_t *dst, const int32_t *perm, int nchunks,
                    size_t chunk_bytes) {
#pragma omp parallel for schedule(static)
  for (int i = 0; i < nchunks; ++i)
    memcpy(dst + (size_t)i * chunk_bytes, src + (size_t)perm[i] * chunk_bytes, chunk_bytes);
}

/* Threads the parallel loops above use (OpenMP's limit for this process). */
int oracle_num_threads(void) { return omp_get_max_threads(); }
