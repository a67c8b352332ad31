/*
 * CPU oracle for the bf16 GEMM of the hot path.  TEST INFRASTRUCTURE ONLY:
 * this file is compiled into liboracle.so, which only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark load.  The product
 * path never links or calls it, and it shares no code with the HIP library.
 *
 * What it computes.  The paper's full-GPU case study (Section 7.1, "Integration
 * with popular kernels") changes only WHICH persistent block computes each
 * output tile; what is computed is the plain matrix product.  The paper fixes
 * no numeric precision, so this oracle takes the plain definition of a bf16
 * GEMM with fp32 accumulation:
 *
 *   R32[i][j] = fl32( ... fl32( fl32(0 + a(i,0)*b(0,j)) + a(i,1)*b(1,j) ) ...
 *                     + a(i,K-1)*b(K-1,j) )        k increasing, one fp32 add
 *   C[i][j]   = bf16 round-to-nearest-even of R32[i][j]
 *
 * with a(i,k), b(k,j) the bf16 inputs widened to fp32.  A product of two bf16
 * values has at most 16 significant bits, so it is exact in fp32 and only the
 * k-ordered additions round.
 *
 * Storage:  A is [M][lda] row-major (element (i,k) at A[i*lda+k]).
 *           b_layout 0 ("NK"): B is stored as its transpose, [N][ldb] row-major,
 *           logical b(k,j) at B[j*ldb+k] (the K-contiguous weight layout).
 *           b_layout 1 ("KN"): B is [K][ldb] row-major, b(k,j) at B[k*ldb+j].
 *           R32 and Cbf16 are dense [M][N] row-major; either may be NULL.
 *
 * Parity pinned by: brute force in exact rationals on tiny shapes, the exact
 * integer regime, identity/zero/transpose invariants, an fp64 library product
 * within Higham's summation bound, a constructed case where the k order alone
 * decides the answer, and the bf16 rounding against torch's conversion.
 *
 * Deliberately plain: no blocking, no BLAS, no fast-math; parallel only over
 * output rows, so the result does not depend on the thread count.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* bf16 -> fp32: the bf16 bit pattern is the top half of the fp32 pattern. */
static float oracle_bf16_to_f32(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* fp32 -> bf16, round to nearest, ties to even, on the bit pattern.
 * Adding 0x7FFF plus the lowest kept bit and truncating rounds the discarded
 * 16 bits to nearest with ties going to the even kept value; an overflow of
 * the mantissa carries into the exponent, which is the correct rounding too.
 * NaN is kept a (quiet) NaN. */
uint16_t oracle_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0u)
    return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7FFFu + lsb;
  return (uint16_t)(u >> 16);
}

void oracle_f32_to_bf16_array(const float* x, uint16_t* y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) y[i] = oracle_f32_to_bf16(x[i]);
}

/* Returns 0 on success, -1 on a bad argument. */
int oracle_gemm_bf16(int M, int N, int K, const uint16_t* A, int lda,
                     const uint16_t* B, int ldb, int b_layout, float* R32,
                     uint16_t* Cbf16) {
  if (M < 0 || N < 0 || K < 0) return -1;
  if (b_layout != 0 && b_layout != 1) return -1;
  if (M == 0 || N == 0) return 0;
  if (K > 0 && (A == NULL || B == NULL)) return -1;
  if (lda < K || (b_layout == 0 ? ldb < K : ldb < N)) return -1;

  /* Widen B once into a [K][N] fp32 copy, b(k,j) at Bt[k*N+j], so that the
   * inner loop below runs over j for fixed k: that keeps k strictly ordered
   * per output while letting the compiler vectorise across outputs. */
  float* Bt = NULL;
  if (K > 0) {
    Bt = (float*)malloc(sizeof(float) * (size_t)K * (size_t)N);
    if (Bt == NULL) return -1;
    for (int k = 0; k < K; ++k)
      for (int j = 0; j < N; ++j)
        Bt[(size_t)k * N + j] = oracle_bf16_to_f32(
            b_layout == 0 ? B[(size_t)j * ldb + k] : B[(size_t)k * ldb + j]);
  }

  int fail = 0;
#pragma omp parallel
  {
    float* acc = (float*)malloc(sizeof(float) * (size_t)N);
    if (acc == NULL) {
#pragma omp atomic write
      fail = 1;
    } else {
#pragma omp for schedule(dynamic, 1)
      for (int i = 0; i < M; ++i) {
        for (int j = 0; j < N; ++j) acc[j] = 0.0f;
        for (int k = 0; k < K; ++k) {
          const float a = oracle_bf16_to_f32(A[(size_t)i * lda + k]);
          const float* brow = Bt + (size_t)k * N;
          for (int j = 0; j < N; ++j) acc[j] = acc[j] + a * brow[j];
        }
        for (int j = 0; j < N; ++j) {
          if (R32) R32[(size_t)i * N + j] = acc[j];
          if (Cbf16) Cbf16[(size_t)i * N + j] = oracle_f32_to_bf16(acc[j]);
        }
      }
      free(acc);
    }
  }
  free(Bt);
  return fail ? -1 : 0;
}

/* Number of OpenMP threads a parallel region will use (reported beside the
 * CPU timing). */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    {
#ifdef _OPENMP
      extern int omp_get_num_threads(void);
      n = omp_get_num_threads();
#endif
    }
  }
  return n;
}
