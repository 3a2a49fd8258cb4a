/* CPU oracle for the skew-symmetric LTL^T factorization and the Pfaffian.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is plain, slow, scalar C that follows
 * the textbook definitions (Parlett & Reid's partially pivoted reduction of a
 * skew-symmetric matrix to tridiagonal form, and the Pfaffian identity
 * Pf(B X B^T) = det(B) Pf(X)).  It shares no code, header or constant with
 * the GPU library; only the tests, the smoke check and the benchmark's CPU
 * baseline may load it.
 *
 * Complex matrices (complex skew-symmetric, X^T = -X) use the same steps
 * with written-out complex arithmetic (ltlt_oracle_complex.h).
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC
 * (no contraction into FMA, no reassociation: every operation rounds once,
 * in the order written).  OpenMP only splits the columns of the real rank-2
 * update between threads; results do not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define CAT_(a, b) a##b
#define CAT(a, b) CAT_(a, b)
#define AT(i, j) A[(int64_t)(i) + (int64_t)(j) * lda]

#define REAL double
#define SFX _f64
#define FABS fabs
#include "ltlt_oracle_body.h"
#undef REAL
#undef SFX
#undef FABS

#define REAL float
#define SFX _f32
#define FABS fabsf
#include "ltlt_oracle_body.h"
#undef REAL
#undef SFX
#undef FABS

#define REAL double
#define CSFX _c128
#define FABS fabs
#include "ltlt_oracle_complex.h"
#undef REAL
#undef CSFX
#undef FABS

#define REAL float
#define CSFX _c64
#define FABS fabsf
#include "ltlt_oracle_complex.h"
#undef REAL
#undef CSFX
#undef FABS

/* Exported entry points (ctypes). */
void oracle_set_threads(int32_t t)
{
#ifdef _OPENMP
    omp_set_num_threads(t > 0 ? t : 1);
#else
    (void)t;
#endif
}

int32_t oracle_get_threads(void)
{
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_ltlt_f64(int64_t n, double* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{ ltlt_f64(n, A, lda, ipiv, nsteps, NULL, NULL, NULL); }

void oracle_ltlt_f32(int64_t n, float* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{ ltlt_f32(n, A, lda, ipiv, nsteps, NULL, NULL, NULL); }

/* The same, recording each step's pivot magnitude and runner-up. */
void oracle_ltlt_trace_f64(int64_t n, double* A, int64_t lda, int32_t* ipiv, int64_t nsteps,
                           double* best_mag, int32_t* runner, double* runner_mag)
{ ltlt_f64(n, A, lda, ipiv, nsteps, best_mag, runner, runner_mag); }

void oracle_ltlt_trace_f32(int64_t n, float* A, int64_t lda, int32_t* ipiv, int64_t nsteps,
                           float* best_mag, int32_t* runner, float* runner_mag)
{ ltlt_f32(n, A, lda, ipiv, nsteps, best_mag, runner, runner_mag); }

void oracle_swap_f64(int64_t n, double* A, int64_t lda, int64_t r, int64_t p)
{ swap_indices_f64(n, A, lda, r, p); }

void oracle_pfaffian_f64(int64_t n, const double* A, int64_t lda, const int32_t* ipiv,
                         double* logabs, int32_t* sign)
{ pfaffian_f64(n, A, lda, ipiv, logabs, sign); }

void oracle_pfaffian_f32(int64_t n, const float* A, int64_t lda, const int32_t* ipiv,
                         double* logabs, int32_t* sign)
{ pfaffian_f32(n, A, lda, ipiv, logabs, sign); }

void oracle_pfaffian_direct_f64(int64_t n, double* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{ pfaffian_direct_f64(n, A, lda, ipiv, nsteps); }

void oracle_pfaffian_direct_f32(int64_t n, float* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{ pfaffian_direct_f32(n, A, lda, ipiv, nsteps); }

/* Batched: `batch` matrices, matrix b at A + b*strideA, pivots at
 * ipiv + b*strideIpiv, one after the other. */
void oracle_ltlt_batched_f64(int64_t n, int64_t batch, double* A, int64_t lda, int64_t strideA,
                             int32_t* ipiv, int64_t strideIpiv, double* logabs, int32_t* sign)
{
    int64_t b;
    for (b = 0; b < batch; ++b) {
        ltlt_f64(n, A + b * strideA, lda, ipiv + b * strideIpiv, -1, NULL, NULL, NULL);
        pfaffian_f64(n, A + b * strideA, lda, ipiv + b * strideIpiv, logabs + b, sign + b);
    }
}

void oracle_ltlt_batched_f32(int64_t n, int64_t batch, float* A, int64_t lda, int64_t strideA,
                             int32_t* ipiv, int64_t strideIpiv, double* logabs, int32_t* sign)
{
    int64_t b;
    for (b = 0; b < batch; ++b) {
        ltlt_f32(n, A + b * strideA, lda, ipiv + b * strideIpiv, -1, NULL, NULL, NULL);
        pfaffian_f32(n, A + b * strideA, lda, ipiv + b * strideIpiv, logabs + b, sign + b);
    }
}

/* Complex: A holds (re, im) pairs, lda in complex elements. */
void oracle_ltlt_c128(int64_t n, void* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{ ltlt_c128(n, (cplx_c128*)A, lda, ipiv, nsteps); }

void oracle_ltlt_c64(int64_t n, void* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{ ltlt_c64(n, (cplx_c64*)A, lda, ipiv, nsteps); }

void oracle_swap_c128(int64_t n, void* A, int64_t lda, int64_t r, int64_t p)
{ cswap_indices_c128(n, (cplx_c128*)A, lda, r, p); }

void oracle_pfaffian_c128(int64_t n, const void* A, int64_t lda, const int32_t* ipiv,
                          double* logabs, double* phase)
{ pfaffian_c128(n, (const cplx_c128*)A, lda, ipiv, logabs, phase); }

void oracle_pfaffian_c64(int64_t n, const void* A, int64_t lda, const int32_t* ipiv,
                         double* logabs, double* phase)
{ pfaffian_c64(n, (const cplx_c64*)A, lda, ipiv, logabs, phase); }
