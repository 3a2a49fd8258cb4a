/*
 * ltlt.h -- C ABI of the MI355X (gfx950) skew-symmetric LTL^T / Pfaffian library.
 *
 * The operation.  For a dense real skew-symmetric X (X^T = -X), the pivoted
 * triangular tridiagonalization (Parlett & Reid's reduction with partial
 * pivoting) computes
 *
 *        P X P^T = L T L^T
 *
 * with L unit lower triangular and L(:,0) = e_0, T skew-symmetric tridiagonal
 * and P a permutation built from one row/column exchange per column step.
 * Step k (k = 0 .. n-3) takes as pivot the first index r >= k+1 of largest
 * |X(r,k)| in the partially reduced matrix, exchanges indices k+1 and r,
 * sets alpha_k = X(k+1,k) = T(k+1,k) and eliminates column k below row k+1
 * with multipliers L(r,k+1) = X(r,k)/alpha_k (0 when alpha_k = 0).  The
 * Pfaffian follows from Pf(B X B^T) = det(B) Pf(X):
 *        Pf(X) = det(P) * prod_j T(2j, 2j+1) = det(P) * prod_j (-alpha_{2j}).
 * The paper behind this library gives no interface for the method; these
 * entry points follow the problem statement, and matrix storage follows the
 * Fortran column-major convention the paper adopts (section 2, "Data
 * storage"): element (i, j) of A is A[i + j*lda].
 *
 * Common rules for every entry point
 *   - All pointers are DEVICE pointers (memory of the current HIP device)
 *     unless stated otherwise.  Calls are stream-ordered and asynchronous:
 *     they enqueue work on `stream` (0 = legacy default stream) and return.
 *   - The caller owns every buffer it passes; nothing is retained after the
 *     call returns.  The library owns a per-device workspace that it grows on
 *     demand (hipMalloc) and keeps until ltlt_release_workspace().
 *   - Calls that overlap in time on one device (e.g. on two streams) share
 *     that workspace and race; serialize them.
 *   - Return value: 0 on success; -i when argument i (1-based) is invalid
 *     (nothing is enqueued); LTLT_ERR_HIP_BASE - e for a HIP runtime error e;
 *     LTLT_ERR_UNSUPPORTED when the size cannot be run (e.g. the panel would
 *     need more co-resident workgroups than the device holds).
 *   - Non-finite input gives unspecified factors but every call terminates.
 *   - Device-side waits.  The panels of ltlt_factor and
 *     ltlt_pfaffian_direct, and ltlt_solve, run workgroups that wait on each
 *     other; every wait is bounded (2 s).  When one gives up (a grid that
 *     could not become resident), the call still runs to its end with every
 *     access in bounds, but its results are poisoned: the factor columns
 *     committed after the failure are NaN and ltlt_pfaffian /
 *     ltlt_pfaffian_direct / ltlt_pfaffian_complex return logabs = NaN with
 *     sign 0 (phase 0).  The failure is recorded in a sticky per-device flag
 *     that ltlt_device_status reports (and clears); the return code of an
 *     asynchronous call cannot carry it.
 */
#ifndef LTLT_H
#define LTLT_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element types (argument `dtype`).  The complex types hold (re, im) pairs
 * (the layout of C99 / numpy / torch complex numbers); lda counts complex
 * elements.  Only ltlt_factor, ltlt_factor_nb and ltlt_pfaffian_complex take
 * them. */
#define LTLT_F64 0
#define LTLT_F32 1
#define LTLT_C128 2
#define LTLT_C64 3

#define LTLT_OK 0
#define LTLT_ERR_HIP_BASE (-1000)      /* returned as LTLT_ERR_HIP_BASE - (int)hipError_t */
#define LTLT_ERR_UNSUPPORTED (-2000)
#define LTLT_ERR_DEVICE_TIMEOUT (-3000) /* a device-side wait exceeded its bound (see ltlt_device_status) */
#define LTLT_ERR_SINGULAR (-4000)       /* ltlt_solve: odd order, X is singular */
#define LTLT_ERR_SCRATCH (-5000)        /* ltlt_factor_noalloc: the order needs more than its fixed array */

/* Largest n accepted by ltlt_factor_batched. */
#define LTLT_BATCHED_MAX_N 64

/*
 * ltlt_factor -- P X P^T = L T L^T of one n x n skew-symmetric matrix, in place.
 *   n      (1) order, 0 <= n < 2^21 - 1 (larger orders return
 *              LTLT_ERR_UNSUPPORTED; an fp64 matrix of that order is 32 TiB).
 *   A      (2) device, column-major, leading dimension lda.  On entry the
 *              STRICT LOWER triangle defines X (X(i,j) = A(i,j) for i > j,
 *              X(j,i) = -A(i,j)); the diagonal is taken as 0 and is never
 *              read or written.  On exit A(k+1,k) = alpha_k = T(k+1,k) for
 *              k = 0..n-2 and A(r,k) = L(r,k+1) for r >= k+2, with rows in the
 *              final pivot order.  The strict upper triangle is never read or
 *              written.
 *   lda    (3) lda >= max(1, n).
 *   dtype  (4) LTLT_F64 or LTLT_F32 (element type of A; arithmetic in it),
 *              or LTLT_C128 / LTLT_C64 for a complex skew-symmetric X
 *              (X^T = -X, a transpose without conjugation; the paper does
 *              not treat this case): the same steps in complex
 *              arithmetic, the pivot being the first index of the largest
 *              |Re X(r,k)| + |Im X(r,k)| (the magnitude of the BLAS complex
 *              i_amax) and the multipliers Smith quotients; same storage and
 *              outputs with complex elements.  The library works on a split
 *              copy (real and imaginary planes, 2 n^2 components of
 *              workspace) and writes the strict lower triangle back at the end.
 *   ipiv   (5) device int32[n]: 0-based exchanges in LAPACK laswp order:
 *              ipiv[0] = 0, ipiv[k+1] = the index exchanged with k+1 at step
 *              k (>= k+1), ipiv[n-1] = n-1.  P applies (i, ipiv[i]) for
 *              i = 0..n-1 in increasing order.
 *   stream (6) HIP stream.
 * Uses the default panel width (128), narrowed when it does not fit: the
 * panel keeps every row of a block in registers of workgroups that are all
 * resident at once (one per CU), R rows each, so a width w needs
 * ceil((n-1)/R) <= CUs with R = 512, 256, 128 for w <= 64, 128, 256
 * (complex: w <= 32, 64, 128).  When the default width needs more
 * workgroups than that, ltlt_factor halves it, down to 32: on a 256-CU
 * device the default width serves n <= 65537 (complex: 32769) and the
 * narrowed ones n <= 131073; larger orders return LTLT_ERR_UNSUPPORTED.
 */
int ltlt_factor(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, hipStream_t stream);

/*
 * ltlt_factor_nb -- as ltlt_factor with an explicit panel width.
 *   nb (6) number of column steps per block, 1 <= nb <= 256 (complex:
 *          1 <= nb <= 128); the trailing update of each block is one
 *          rank-(nb+1) lower-triangular product (complex: one real product of
 *          depth 2(nb+1) per plane).
 *   stream is argument 7.
 * Returns LTLT_ERR_UNSUPPORTED (nothing enqueued) when the panel of width nb
 * needs more co-resident workgroups than the device holds (see ltlt_factor);
 * ltlt_factor itself narrows the width instead.
 */
int ltlt_factor_nb(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, int nb,
                   hipStream_t stream);

/*
 * ltlt_factor_noalloc -- ltlt_factor for callers that cannot allocate device
 * memory: code being captured into a HIP graph, tight serving loops, harnesses
 * that forbid hipMalloc.  Same operation, arguments, outputs and kernels as
 * ltlt_factor with the default panel width (128), real types only (dtype
 * LTLT_F64 or LTLT_F32; others return -4).  Its whole workspace is a fixed
 * 16 MiB device array inside the library (one per GPU, held until the process
 * ends), so it serves n <= 4928 in fp64 and n <= 8128 in fp32; a larger order
 * returns LTLT_ERR_SCRATCH with nothing enqueued.  It calls no hipMalloc /
 * hipFree and allocates no host memory; its first call on a device looks up
 * the array's address and enqueues one small kernel that clears the status
 * words kept there.  Every call on one GPU shares that array (and every call
 * of this library shares its status words): calls that overlap in time on one
 * GPU -- on two streams, or with another call of this library -- race.  The
 * array keeps the last call's contents; each call initializes what it reads.
 * No per-kernel profiling events are recorded for it.
 */
int ltlt_factor_noalloc(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, hipStream_t stream);

/*
 * ltlt_pfaffian -- sign and log|Pf(X)| from the output of ltlt_factor.
 *   n, A, lda, dtype, ipiv (1-5) exactly as returned by ltlt_factor (read only).
 *   logabs (6) device double[1]: log|Pf(X)| (natural log), summed in fp64.
 *   sign   (7) device int32[1]: -1, 0 or +1.
 *   stream (8).
 * n = 0 gives sign 1, logabs 0.  Odd n, or any alpha_{2j} = 0, gives sign 0
 * and logabs = -inf (Pf(X) = 0).
 */
int ltlt_pfaffian(int64_t n, const void* A, int64_t lda, int dtype, const int32_t* ipiv,
                  double* logabs, int32_t* sign, hipStream_t stream);

/*
 * ltlt_pfaffian_complex -- log|Pf(X)| and the phase Pf(X)/|Pf(X)| from the
 * output of ltlt_factor for a complex X:
 *        Pf(X) = det(P) * prod_j (-alpha_{2j}),  det(P) = (-1)^(#exchanges).
 *   n, A, lda, dtype, ipiv (1-5) as returned by ltlt_factor with dtype
 *              LTLT_C128 or LTLT_C64 (read only; other dtypes: -4).
 *   logabs (6) device double[1]: sum_j log|alpha_{2j}| in fp64.
 *   phase  (7) device double[2]: (re, im) of the unit complex number
 *              det(P) prod_j (-alpha_{2j})/|alpha_{2j}|, in fp64.
 *   stream (8).
 * n = 0 gives logabs 0, phase 1.  Odd n, or any alpha_{2j} = 0, gives
 * logabs = -inf and phase 0.
 */
int ltlt_pfaffian_complex(int64_t n, const void* A, int64_t lda, int dtype, const int32_t* ipiv,
                          double* logabs, double* phase, hipStream_t stream);

/*
 * ltlt_pfaffian_direct -- Pf(X) without the factors: the pivoted reduction
 * run on the even column steps only.  After column k is eliminated with
 * pivot row k+1, row k of the transformed matrix has the single entry
 * T(k, k+1) = -alpha_k, so the Pfaffian expands along it into -alpha_k times
 * the Pfaffian of the matrix without indices k and k+1; column k+1 is never
 * eliminated.  With Pf(B X B^T) = det(B) Pf(X) for the unit lower
 * elimination matrices and the exchanges,
 *   Pf(X) = (-1)^(#exchanges) prod_{k even} (-alpha_k),
 * from half the pivot searches of ltlt_factor (the paper does not treat
 * Pfaffians; this follows from the two identities above).
 *   n, A, lda, dtype: as ltlt_factor.  A is used as workspace: on exit
 *       A(k+1, k) = alpha_k for even k; every other entry of the strict lower
 *       triangle is unspecified; diagonal and upper triangle untouched.
 *   ipiv (device int32[n]): ipiv[k+1] = pivot of even step k (first index of
 *       the largest magnitude in the current column k, rows >= k+1),
 *       ipiv[i] = i elsewhere.
 *   nb: columns per block, even, 2 .. 256; 0 selects the default (128),
 *       halved down to 32 when its panel does not fit on the device (the
 *       pair panel holds 448, 224, 112 rows per workgroup, one workgroup
 *       per CU, for nb <= 64, 128, 256: on 256 CUs the default serves
 *       n <= 57345 and the narrowed widths n <= 114689); an explicit nb that
 *       does not fit returns LTLT_ERR_UNSUPPORTED.
 *   logabs, sign: DEVICE double / int32 outputs as in ltlt_pfaffian (odd n:
 *       sign 0, logabs -inf; n = 0: sign 1, logabs 0).
 * Returns 0, -i when argument i is invalid (nb odd or out of range: -6), or
 * a runtime / device-wait error as ltlt_factor.  Stream-ordered.
 */
int ltlt_pfaffian_direct(int64_t n, void* A, int64_t lda, int dtype, int32_t* ipiv, int nb,
                         double* logabs, int32_t* sign, hipStream_t stream);

/*
 * ltlt_solve -- X x = b for each column b of B, from the output of
 * ltlt_factor (packed A and ipiv).  With P X P^T = L T L^T:
 *   x = P^T L^{-T} T^{-1} L^{-1} P b,
 * a permutation, a forward substitution with the unit lower L (read from the
 * packed columns: L(r, c) = A(r, c-1), r >= c+1; L(:,0) = e_0), the two
 * recurrences of the skew tridiagonal T (T(k+1,k) = A(k+1,k)), a backward
 * substitution with L^T and the inverse permutation (the paper does not
 * treat solves; this is the factorization's defining identity).
 *   n, A, lda, dtype, ipiv: as left by ltlt_factor (A and ipiv are read only).
 *   nrhs: number of right-hand sides (>= 0).
 *   B (device, dtype): n x nrhs column-major, leading dimension ldb >= n;
 *       overwritten with the solutions.
 * Returns 0; -i when argument i is invalid; LTLT_ERR_SINGULAR for odd n
 * (a skew-symmetric matrix of odd order is singular); a runtime or
 * device-wait error as ltlt_factor.  When some alpha_{2j} is 0 (Pf(X) = 0)
 * the solutions are not finite.  Stream-ordered; uses the library's cached
 * workspace.
 */
int ltlt_solve(int64_t n, const void* A, int64_t lda, int dtype, const int32_t* ipiv, int64_t nrhs, void* B,
               int64_t ldb, hipStream_t stream);

/*
 * ltlt_factor_batched -- independent factorizations and Pfaffians of `batch`
 * matrices of order n <= LTLT_BATCHED_MAX_N, one wave per matrix (four per
 * workgroup).  The pivot rule, storage and Pfaffian are those of
 * ltlt_factor and ltlt_pfaffian; the column updates are applied in blocks of
 * 16 steps (a different rounding order, same tolerance).
 *   n          (1) order, 0 <= n <= LTLT_BATCHED_MAX_N.
 *   batch      (2) number of matrices, >= 0.
 *   A          (3) device; matrix b is column-major at A + b*strideA
 *                  (elements), leading dimension lda; strict lower triangle
 *                  in, factors out exactly as ltlt_factor (upper triangle and
 *                  diagonal neither read nor written).
 *   lda        (4) lda >= max(1, n).
 *   strideA    (5) >= lda*n (matrices must not overlap).
 *   dtype      (6) LTLT_F64 or LTLT_F32.
 *   ipiv       (7) device int32; pivots of matrix b at ipiv + b*strideIpiv.
 *   strideIpiv (8) >= n.
 *   logabs     (9) device double[batch]: log|Pf| per matrix.
 *   sign      (10) device int32[batch]: sign of Pf per matrix.
 *   stream    (11).
 */
int ltlt_factor_batched(int64_t n, int64_t batch, void* A, int64_t lda, int64_t strideA,
                        int dtype, int32_t* ipiv, int64_t strideIpiv, double* logabs,
                        int32_t* sign, hipStream_t stream);

/*
 * ltlt_skew_update -- the trailing update of one block on its own:
 *   for m x m indices i > c:
 *     C(i,c) <- S(perm[i], perm[c]) + sum_{u<K} Lx(i,u) * Bt(c,u),
 *   where S(a,b) = C(a,b) for a > b and -C(b,a) for a < b (the skew matrix
 *   held in the strict lower triangle).
 *   C      (2) device, column-major, ldc; only the strict lower triangle of
 *              the m x m block is written; the diagonal and the upper
 *              triangle are never written.
 *   perm   (4) device int32[m] or NULL (identity).  Entries must form a
 *              permutation and, for every pair i > c with perm[i] != i or
 *              perm[c] != c, the element C(perm[i], perm[c]) must lie outside
 *              the m x m block being written -- i.e. callers pass a C that is a
 *              sub-block of a larger matrix and offsets in perm that point
 *              into the surrounding rows/columns (read through the same
 *              strict-lower-triangle rule); with perm == NULL this is a plain
 *              skew-symmetric rank-K update.  perm entries are relative to C
 *              (may be negative, reaching rows/columns before C).
 *   Lx, Bt (6, 8) device, column-major m x K with leading dims ldl, ldb.
 *   In the factorization, K = nb + 1, Lx = [L(:, j+1..j+nb), carry column]
 *   and Bt = Lx Tx^T with Tx skew tridiagonal (Tx[u,u+1] = alpha_{j+u+1},
 *   Tx[nb-1,nb] = 1), so Lx Bt^T = Lx Tx Lx^T.
 * Arguments: (1) m, (2) C, (3) ldc, (4) perm, (5) K, (6) Lx, (7) ldl,
 * (8) Bt, (9) ldb, (10) dtype, (11) stream.
 */
int ltlt_skew_update(int64_t m, void* C, int64_t ldc, const int32_t* perm, int64_t K,
                     const void* Lx, int64_t ldl, const void* Bt, int64_t ldb, int dtype,
                     hipStream_t stream);

/*
 * ltlt_device_status -- synchronizes `stream` and reports whether a
 * device-side bounded wait of any call on the current device gave up since
 * the last ltlt_device_status (LTLT_ERR_DEVICE_TIMEOUT: the results of that
 * call are poisoned, see the common rules) and clears that sticky flag.
 * Returns 0 when no wait gave up, or a HIP runtime error.
 */
int ltlt_device_status(hipStream_t stream);

/*
 * ltlt_test_force_timeout -- for tests of the failure path only (host call,
 * process-wide).  on = 1: every following ltlt_factor, ltlt_pfaffian_direct
 * and ltlt_solve starts as if one of its device-side waits had already given
 * up (waits end at their first poll, outputs are poisoned, the sticky flag
 * is raised), without any kernel waiting for long; on = 0 (the default)
 * restores normal operation.  Returns 0, or -1 for another value.
 */
int ltlt_test_force_timeout(int on);

/*
 * Per-kernel timing of ltlt_factor, measured with HIP events recorded on the
 * stream each kernel runs on.
 *   ltlt_profile_enable(1) starts recording every launch (and clears earlier
 *   records), ltlt_profile_enable(2) the trailing-update launches only (each
 *   recorded launch adds two event records, about 2 us each, to the
 *   stream), ltlt_profile_enable(0) stops; other values return -1.
 *   ltlt_profile_read synchronizes the recorded events and writes, for each
 *   kernel kind k < nkinds (0 = panel, 1 = trailing update, 2 = commit,
 *   3 = other), the launch count, the summed milliseconds and the summed
 *   nominal flops (trailing update: m2^2 * nb per launch; others 0) into the
 *   HOST arrays launches[k], ms[k], flops[k].  Returns the number of kinds
 *   written.
 */
int ltlt_profile_enable(int on);
int ltlt_profile_read(int nkinds, int64_t* launches, double* ms, double* flops);

/* Frees the cached workspace of every device (host call; synchronizes). */
int ltlt_release_workspace(void);

/*
 * ltlt_set_cooperative_panels -- how the grids whose workgroups wait on
 * each other are launched: the panels of ltlt_factor and
 * ltlt_pfaffian_direct and the substitutions of ltlt_solve (host call,
 * process-wide; returns 0, or -1 for a value other than 0 or 1).  Such a
 * grid (a panel: at most one workgroup per CU; a substitution: at most what
 * the device holds at once) must be resident all at once.  on = 0 (the
 * default): ordinary launches.  Issued in
 * stream order onto a device that runs nothing else, every workgroup is
 * dispatched at once; when other streams or processes hold CUs during a
 * call, the panel waits for them, and if it cannot become resident within
 * its bounded wait (2 s) the call reports LTLT_ERR_DEVICE_TIMEOUT through
 * ltlt_device_status instead of hanging.  on = 1: the runtime's cooperative
 * launch, which guarantees co-residency on a shared device at about 20 us
 * per panel launch (2-3 % of an n = 16384 factorization).
 */
int ltlt_set_cooperative_panels(int on);

/*
 * ltlt_mfma_probe -- measured matrix-core rate of the current device.  A
 * diagnostic, not part of the factorization: it runs, on `stream`, one
 * kernel in which every wave executes `iters` iterations of 16 independent
 * 16x16x4 MFMAs (fp64 for LTLT_F64, fp32 for LTLT_F32) from registers, two
 * workgroups of four waves per CU, times it with HIP events and writes the
 * sustained TFLOP/s into the HOST double *tflops.  This is the ceiling an
 * MFMA kernel can reach on the device, used to state a kernel's rate as a
 * fraction of it next to the published peak.  Allocates and frees a small
 * device buffer; synchronizes the stream.
 * Returns 0, -1 (bad dtype), -2 (iters outside [1, 1e8]), -3 (tflops NULL)
 * or a runtime error.
 */
int ltlt_mfma_probe(int dtype, int64_t iters, double* tflops, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LTLT_H */
