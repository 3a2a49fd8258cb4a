/* Driver for the sanitizer build of the CPU oracle (AddressSanitizer and
 * UndefinedBehaviorSanitizer, host code only): every exported oracle entry
 * point on small and edge-case inputs -- orders 0..5 and a few larger ones,
 * lda > n with guard bands, zero and NaN matrices, several threads for the
 * rank-2 update.  Inputs come from a xorshift generator here; nothing is
 * checked but memory safety and defined behaviour (the numerical pins live in
 * the Python tests). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void oracle_set_threads(int32_t t);
void oracle_ltlt_f64(int64_t n, double* A, int64_t lda, int32_t* ipiv, int64_t nsteps);
void oracle_ltlt_f32(int64_t n, float* A, int64_t lda, int32_t* ipiv, int64_t nsteps);
void oracle_ltlt_trace_f64(int64_t n, double* A, int64_t lda, int32_t* ipiv, int64_t nsteps,
                           double* best, int32_t* runner, double* rmag);
void oracle_swap_f64(int64_t n, double* A, int64_t lda, int64_t r, int64_t p);
void oracle_pfaffian_f64(int64_t n, const double* A, int64_t lda, const int32_t* ipiv,
                         double* logabs, int32_t* sign);
void oracle_pfaffian_f32(int64_t n, const float* A, int64_t lda, const int32_t* ipiv,
                         double* logabs, int32_t* sign);
void oracle_pfaffian_direct_f64(int64_t n, double* A, int64_t lda, int32_t* ipiv, int64_t nsteps);
void oracle_pfaffian_direct_f32(int64_t n, float* A, int64_t lda, int32_t* ipiv, int64_t nsteps);
void oracle_ltlt_batched_f64(int64_t n, int64_t batch, double* A, int64_t lda, int64_t strideA,
                             int32_t* ipiv, int64_t strideIpiv, double* logabs, int32_t* sign);
void oracle_ltlt_c128(int64_t n, void* A, int64_t lda, int32_t* ipiv, int64_t nsteps);
void oracle_ltlt_c64(int64_t n, void* A, int64_t lda, int32_t* ipiv, int64_t nsteps);
void oracle_pfaffian_c128(int64_t n, const void* A, int64_t lda, const int32_t* ipiv,
                          double* logabs, double* phase);
void oracle_swap_c128(int64_t n, void* A, int64_t lda, int64_t r, int64_t p);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform(void)
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return (double)(rng_state >> 11) * (1.0 / 9007199254740992.0) * 2.0 - 1.0;
}

/* kind 0: random, 1: zero, 2: NaN and Inf sprinkled, 3: small integers */
static void fill(double* A, int64_t n, int64_t lda, int kind)
{
    int64_t i, j;
    for (j = 0; j < n; ++j)
        for (i = 0; i < lda; ++i) {
            double v = uniform();
            if (kind == 1) v = 0.0;
            if (kind == 3) v = floor(2.5 * v);
            if (kind == 2 && ((i * 7 + j) % 11 == 0)) v = (i & 1) ? NAN : INFINITY;
            A[i + j * lda] = v;
        }
}

int main(void)
{
    static const int64_t orders[] = {0, 1, 2, 3, 4, 5, 7, 16, 33, 64, 100};
    size_t o;
    int kind, threads;
    for (threads = 1; threads <= 3; threads += 2) {
        oracle_set_threads(threads);
        for (o = 0; o < sizeof(orders) / sizeof(orders[0]); ++o) {
            const int64_t n = orders[o];
            const int64_t lda = n + 3;
            const int64_t cells = lda * (n > 0 ? n : 1);
            for (kind = 0; kind < 4; ++kind) {
                double* A = (double*)malloc((size_t)cells * sizeof(double));
                double* B = (double*)malloc((size_t)cells * sizeof(double));
                float* F = (float*)malloc((size_t)cells * sizeof(float));
                double* C = (double*)malloc((size_t)cells * 2 * sizeof(double));
                int32_t* ipiv = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
                int64_t ns = n > 2 ? n - 2 : 1;
                double* best = (double*)malloc((size_t)ns * sizeof(double));
                double* rmag = (double*)malloc((size_t)ns * sizeof(double));
                int32_t* runner = (int32_t*)malloc((size_t)ns * sizeof(int32_t));
                double logabs, phase[2];
                int32_t sign;
                int64_t i;
                fill(A, n, lda, kind);
                memcpy(B, A, (size_t)cells * sizeof(double));
                for (i = 0; i < cells; ++i) F[i] = (float)A[i];
                for (i = 0; i < cells; ++i) { C[2 * i] = A[i]; C[2 * i + 1] = 0.5 * A[(i * 5) % cells]; }

                oracle_ltlt_f64(n, A, lda, ipiv, -1);
                oracle_pfaffian_f64(n, A, lda, ipiv, &logabs, &sign);
                memcpy(A, B, (size_t)cells * sizeof(double));
                oracle_ltlt_trace_f64(n, A, lda, ipiv, -1, best, runner, rmag);
                memcpy(A, B, (size_t)cells * sizeof(double));
                oracle_ltlt_f64(n, A, lda, ipiv, n / 2);
                memcpy(A, B, (size_t)cells * sizeof(double));
                if (n >= 2) oracle_swap_f64(n, A, lda, 0, n - 1);
                memcpy(A, B, (size_t)cells * sizeof(double));
                oracle_pfaffian_direct_f64(n, A, lda, ipiv, -1);
                oracle_pfaffian_f64(n, A, lda, ipiv, &logabs, &sign);
                oracle_ltlt_f32(n, F, lda, ipiv, -1);
                oracle_pfaffian_f32(n, F, lda, ipiv, &logabs, &sign);
                for (i = 0; i < cells; ++i) F[i] = (float)B[i];
                oracle_pfaffian_direct_f32(n, F, lda, ipiv, -1);
                oracle_ltlt_c128(n, C, lda, ipiv, -1);
                oracle_pfaffian_c128(n, C, lda, ipiv, &logabs, phase);
                if (n >= 2) oracle_swap_c128(n, C, lda, 0, n - 1);
                for (i = 0; i < cells; ++i) { C[2 * i] = (float)B[i]; C[2 * i + 1] = 0.0; }
                /* complex64: reinterpret the first half of C as (float re, float im) pairs */
                {
                    float* C32 = (float*)C;
                    for (i = 0; i < cells; ++i) { C32[2 * i] = (float)B[i]; C32[2 * i + 1] = (float)B[(i * 3) % cells]; }
                    oracle_ltlt_c64(n, C32, lda, ipiv, -1);
                }
                free(A); free(B); free(F); free(C); free(ipiv); free(best); free(rmag); free(runner);
            }
            /* batched: three matrices with strides beyond lda*n */
            {
                const int64_t batch = 3, stride = (n + 1) * (n > 0 ? n : 1) + 5;
                double* Ab = (double*)malloc((size_t)(stride * batch) * sizeof(double));
                int32_t* ib = (int32_t*)malloc((size_t)((n + 2) * batch) * sizeof(int32_t));
                double lb[3];
                int32_t sb[3];
                int64_t b;
                for (b = 0; b < batch; ++b) fill(Ab + b * stride, n, n > 0 ? n : 1, (int)b);
                oracle_ltlt_batched_f64(n, batch, Ab, n > 0 ? n : 1, stride, ib, n + 2, lb, sb);
                free(Ab); free(ib);
            }
        }
    }
    printf("sanitized oracle run complete\n");
    return 0;
}
