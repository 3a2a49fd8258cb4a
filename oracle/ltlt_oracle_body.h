/* Body of the CPU oracle, instantiated once per floating-point type by
 * ltlt_oracle.c (REAL = double or float, SFX = _f64 or _f32, FABS = fabs or
 * fabsf).  Test infrastructure only: nothing in the library links this.
 *
 * Storage: column-major with leading dimension lda; element (i, j) is
 * A[i + j*lda].  Only the strict lower triangle is read or written; the
 * skew-symmetric matrix is X(i,j) = A(i,j) for i > j, X(j,i) = -A(i,j),
 * X(i,i) = 0.
 */

/* Swap indices r < p of the skew matrix held in the strict lower triangle,
 * i.e. replace X by Q X Q^T where Q exchanges rows/columns r and p.
 * Every stored entry (a, b), a > b, of the new matrix is X(s(a), s(b)) with s
 * the transposition (r p); read off case by case:
 *   b <  r          : rows r and p exchange                (a in {r, p})
 *   b == r, r<a<p   : X(a, p) = -X(p, a)  (upper entry of X read from lower)
 *   b == r, a == p  : X(r, p) = -X(p, r)
 *   b == r, a >  p  : X(a, p)
 *   r<b<p,  a == p  : X(r, b) = -X(b, r)
 *   b == p, a >  p  : X(a, r)
 * and nothing else changes. */
static void CAT(swap_indices, SFX)(int64_t n, REAL* A, int64_t lda, int64_t r, int64_t p)
{
    int64_t b, a;
    REAL t;
    for (b = 0; b < r; ++b) {               /* rows r and p, columns left of r */
        t = AT(r, b); AT(r, b) = AT(p, b); AT(p, b) = t;
    }
    for (a = r + 1; a < p; ++a) {           /* column r against row p */
        t = AT(a, r);
        AT(a, r) = -AT(p, a);
        AT(p, a) = -t;
    }
    AT(p, r) = -AT(p, r);
    for (a = p + 1; a < n; ++a) {           /* columns r and p below row p */
        t = AT(a, r); AT(a, r) = AT(a, p); AT(a, p) = t;
    }
}

/* Skew rank-2 update of the trailing strict lower triangle after column k
 * is eliminated: X(i, j) += l_i v_j - v_i l_j for i > j >= k+2, with the
 * multipliers l in column k of A and v = X(k+2:, k+1) copied beforehand.
 * Columns j are independent (each writes only its own column and reads
 * column k and v), so they may run on several threads: every entry is still
 * formed by the same two products and two additions in the same order, and
 * the result is bitwise the same for any thread count. */
static void CAT(rank2_update, SFX)(int64_t n, REAL* A, int64_t lda, int64_t k, const REAL* v)
{
    int64_t j;
#pragma omp parallel for schedule(dynamic, 16)
    for (j = k + 2; j < n; ++j) {
        const REAL lj = AT(j, k), vj = v[j];
        int64_t i;
        for (i = j + 1; i < n; ++i) {
            AT(i, j) = AT(i, j) + (AT(i, k) * vj - v[i] * lj);
        }
    }
}

/* Unblocked Parlett-Reid reduction with partial pivoting,
 * P X P^T = L T L^T, run for `nsteps` column steps (all n-2 steps when
 * nsteps < 0 or nsteps > n-2).
 *
 * Step k (k = 0 .. n-3) eliminates column k below row k+1:
 *   1. p = first index r >= k+1 maximising |X(r, k)|            (pivot)
 *   2. ipiv[k+1] = p; exchange indices k+1 and p                 (Q_k)
 *   3. alpha_k = X(k+1, k); l_r = X(r, k) / alpha_k for r >= k+2
 *      (l = 0 when alpha_k = 0: the column is already eliminated)
 *   4. X <- M X M^T with M = I - l e_{k+1}^T, which on the trailing
 *      strict lower triangle (i > j >= k+2) is the skew rank-2 update
 *      X(i, j) += l_i v_j - v_i l_j,  v = X(k+2:, k+1)
 *      (column k+1 itself is unchanged because X(k+1, k+1) = 0).
 * On exit A(k+1, k) = alpha_k = T(k+1, k) and A(r, k) = l_r = L(r, k+1) for
 * r >= k+2, with rows of earlier columns carried through later exchanges.
 * When best_mag is not NULL, step k also records |X(p, k)| in best_mag[k] and
 * the runner-up row and magnitude in runner[k], runner_mag[k] (arrays of
 * n-2 entries); the factorization itself is the same either way. */
static void CAT(ltlt, SFX)(int64_t n, REAL* A, int64_t lda, int32_t* ipiv, int64_t nsteps,
                          REAL* best_mag, int32_t* runner, REAL* runner_mag)
{
    int64_t i, k, r, p, q, last;
    REAL best, second, alpha;
    REAL* v;

    for (i = 0; i < n; ++i) ipiv[i] = (int32_t)i;
    last = n - 2;                                 /* number of column steps */
    if (nsteps >= 0 && nsteps < last) last = nsteps;
    if (last <= 0) return;
    v = (REAL*)malloc((size_t)n * sizeof(REAL));
    if (!v) return;

    for (k = 0; k < last; ++k) {
        /* 1. pivot: strict '>' keeps the first of equal magnitudes */
        p = k + 1;
        best = FABS(AT(k + 1, k));
        for (r = k + 2; r < n; ++r) {
            if (FABS(AT(r, k)) > best) { best = FABS(AT(r, k)); p = r; }
        }
        /* optional record of the decision: the pivot's magnitude and the
         * runner-up (first index of the largest magnitude among the other
         * rows; -1 when there is none) */
        if (best_mag) {
            q = -1;
            second = (REAL)0;
            for (r = k + 1; r < n; ++r) {
                if (r != p && (q < 0 || FABS(AT(r, k)) > second)) { second = FABS(AT(r, k)); q = r; }
            }
            best_mag[k] = best;
            runner[k] = (int32_t)q;
            runner_mag[k] = second;
        }
        /* 2. exchange */
        ipiv[k + 1] = (int32_t)p;
        if (p != k + 1) CAT(swap_indices, SFX)(n, A, lda, k + 1, p);
        /* 3. multipliers */
        alpha = AT(k + 1, k);
        for (r = k + 2; r < n; ++r) AT(r, k) = (alpha != (REAL)0) ? AT(r, k) / alpha : (REAL)0;
        /* 4. skew rank-2 update of the trailing strict lower triangle */
        for (r = k + 2; r < n; ++r) v[r] = AT(r, k + 1);
        CAT(rank2_update, SFX)(n, A, lda, k, v);
    }
    free(v);
}

/* Pfaffian from the factors.  Pf(B X B^T) = det(B) Pf(X) gives
 * Pf(X) = det(P) det(L) Pf(T) with det(L) = 1, det(P) = (-1)^(#exchanges),
 * and for the skew tridiagonal T with T(2j+1, 2j) = alpha_{2j}:
 * Pf(T) = prod_j T(2j, 2j+1) = prod_j (-alpha_{2j}).
 * Returned as sign in {-1, 0, +1} and log|Pf| (fp64, summed in index order);
 * odd n or a zero alpha_{2j} gives sign 0 and logabs = -inf. */
static void CAT(pfaffian, SFX)(int64_t n, const REAL* A, int64_t lda, const int32_t* ipiv,
                               double* logabs, int32_t* sign)
{
    int64_t j, i;
    int s = 1;
    double acc = 0.0;
    if (n % 2 != 0) { *logabs = -INFINITY; *sign = 0; return; }
    for (j = 0; 2 * j < n; ++j) {
        double a = (double)A[(2 * j + 1) + (2 * j) * lda];
        if (a == 0.0) { *logabs = -INFINITY; *sign = 0; return; }
        acc += log(fabs(a));
        if (-a < 0.0) s = -s;                    /* factor T(2j,2j+1) = -alpha */
    }
    for (i = 0; i < n; ++i)
        if (ipiv[i] != i) s = -s;                /* each exchange flips det(P) */
    *logabs = acc;
    *sign = s;
}

/* Pfaffian by the even column steps only (no factorization output).
 * Step k = 0, 2, 4, ..., n-2 on the current matrix:
 *   1. p = first index r >= k+1 maximising |X(r, k)|; ipiv[k+1] = p;
 *      exchange indices k+1 and p
 *   2. alpha_k = X(k+1, k); l_r = X(r, k) / alpha_k for r >= k+2
 *      (l = 0 when alpha_k = 0)
 *   3. X <- M X M^T, M = I - l e_{k+1}^T: the same skew rank-2 update of the
 *      trailing strict lower triangle as a full step,
 *      X(i, j) += l_i v_j - v_i l_j (i > j >= k+2),  v = X(k+2:, k+1).
 * After step 3, row k of X has the single nonzero X(k, k+1) = -alpha_k, so
 * expanding the Pfaffian along row k gives Pf = X(k, k+1) Pf(X without k and
 * k+1): column k+1 is never eliminated and the next step is k+2.  With
 * det(M) = 1 and one sign flip per exchange,
 *   Pf(X) = (-1)^(#exchanges) prod_{k even} (-alpha_k).
 * On exit A(k+1, k) = alpha_k for even k (other entries hold intermediate
 * values), ipiv[k+1] = p_k for even k and ipiv[i] = i otherwise; the
 * Pfaffian of the result is read by `pfaffian` above.  Odd n: no steps
 * (Pf = 0). */
static void CAT(pfaffian_direct, SFX)(int64_t n, REAL* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{
    int64_t i, k, r, p, done;
    REAL best, alpha;
    REAL* v;

    for (i = 0; i < n; ++i) ipiv[i] = (int32_t)i;
    if (n % 2 != 0 || n < 2) return;
    v = (REAL*)malloc((size_t)n * sizeof(REAL));
    if (!v) return;
    /* nsteps >= 0 stops after that many even steps (a timing sample) */
    for (k = 0, done = 0; k + 1 < n && (nsteps < 0 || done < nsteps); k += 2, ++done) {
        p = k + 1;
        best = FABS(AT(k + 1, k));
        for (r = k + 2; r < n; ++r) {
            if (FABS(AT(r, k)) > best) { best = FABS(AT(r, k)); p = r; }
        }
        ipiv[k + 1] = (int32_t)p;
        if (p != k + 1) CAT(swap_indices, SFX)(n, A, lda, k + 1, p);
        alpha = AT(k + 1, k);
        for (r = k + 2; r < n; ++r) AT(r, k) = (alpha != (REAL)0) ? AT(r, k) / alpha : (REAL)0;
        for (r = k + 2; r < n; ++r) v[r] = AT(r, k + 1);
        CAT(rank2_update, SFX)(n, A, lda, k, v);
    }
    free(v);
}
