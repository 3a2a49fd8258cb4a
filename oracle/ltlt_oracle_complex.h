/* Complex body of the CPU oracle, instantiated once per component type by
 * ltlt_oracle.c (REAL = double or float, CSFX = _c128 or _c64, FABS = fabs
 * or fabsf).  Test infrastructure only: nothing in the library links this.
 *
 * The same reduction as the real body for a complex skew-symmetric X
 * (X^T = -X; a transpose, no conjugation), in the same storage: column-major,
 * element (i, j) at A[i + j*lda], complex elements as (re, im) pairs
 * (the layout of C99 / numpy complex), strict lower triangle only.
 *
 * Complex arithmetic is written out so that every operation rounds once, in
 * the order written:
 *   product   (a + bi)(c + di) = (ac - bd) + (ad + bc) i
 *   quotient  Smith's algorithm (Smith, CACM 5(8), 1962): for |c| >= |d|,
 *             r = d/c, den = c + d r, ((a + b r) + (b - a r) i) / den, and
 *             symmetrically for |d| > |c|
 *   magnitude for the pivot search: |re| + |im| (the magnitude the BLAS
 *             complex i_amax uses)
 * With zero imaginary parts every one of these reduces exactly to its real
 * counterpart, so a real matrix stored as complex gives the real body's
 * results bit for bit. */

typedef struct { REAL re, im; } CAT(cplx, CSFX);
#define CT CAT(cplx, CSFX)
#define CAT_C(i, j) A[(int64_t)(i) + (int64_t)(j) * lda]

static CT CAT(cmul, CSFX)(CT x, CT y)
{
    CT z;
    z.re = x.re * y.re - x.im * y.im;
    z.im = x.re * y.im + x.im * y.re;
    return z;
}

static CT CAT(csub, CSFX)(CT x, CT y)
{
    CT z;
    z.re = x.re - y.re;
    z.im = x.im - y.im;
    return z;
}

static CT CAT(cadd, CSFX)(CT x, CT y)
{
    CT z;
    z.re = x.re + y.re;
    z.im = x.im + y.im;
    return z;
}

static CT CAT(cneg, CSFX)(CT x)
{
    CT z;
    z.re = -x.re;
    z.im = -x.im;
    return z;
}

static CT CAT(cdiv, CSFX)(CT x, CT y)
{
    CT z;
    REAL r, den;
    if (FABS(y.re) >= FABS(y.im)) {
        r = y.im / y.re;
        den = y.re + y.im * r;
        z.re = (x.re + x.im * r) / den;
        z.im = (x.im - x.re * r) / den;
    } else {
        r = y.re / y.im;
        den = y.im + y.re * r;
        z.re = (x.re * r + x.im) / den;
        z.im = (x.im * r - x.re) / den;
    }
    return z;
}

static REAL CAT(cabs1, CSFX)(CT x) { return FABS(x.re) + FABS(x.im); }

static int CAT(cnonzero, CSFX)(CT x) { return x.re != (REAL)0 || x.im != (REAL)0; }

/* Q X Q^T for the transposition (r p), r < p: the case list of the real
 * body's swap_indices, with complex negation. */
static void CAT(cswap_indices, CSFX)(int64_t n, CT* A, int64_t lda, int64_t r, int64_t p)
{
    int64_t b, a;
    CT t;
    for (b = 0; b < r; ++b) {
        t = CAT_C(r, b); CAT_C(r, b) = CAT_C(p, b); CAT_C(p, b) = t;
    }
    for (a = r + 1; a < p; ++a) {
        t = CAT_C(a, r);
        CAT_C(a, r) = CAT(cneg, CSFX)(CAT_C(p, a));
        CAT_C(p, a) = CAT(cneg, CSFX)(t);
    }
    CAT_C(p, r) = CAT(cneg, CSFX)(CAT_C(p, r));
    for (a = p + 1; a < n; ++a) {
        t = CAT_C(a, r); CAT_C(a, r) = CAT_C(a, p); CAT_C(a, p) = t;
    }
}

/* The unblocked pivoted reduction (steps 1-4 of the real body's ltlt), with
 * the pivot chosen by |re| + |im| (first maximum) and complex multipliers
 * and rank-2 update X(i, j) += l_i v_j - v_i l_j. */
static void CAT(ltlt, CSFX)(int64_t n, CT* A, int64_t lda, int32_t* ipiv, int64_t nsteps)
{
    int64_t i, j, k, r, p, last;
    REAL best, m;
    CT alpha;
    CT* v;

    for (i = 0; i < n; ++i) ipiv[i] = (int32_t)i;
    last = n - 2;
    if (nsteps >= 0 && nsteps < last) last = nsteps;
    if (last <= 0) return;
    v = (CT*)malloc((size_t)n * sizeof(CT));
    if (!v) return;

    for (k = 0; k < last; ++k) {
        p = k + 1;
        best = CAT(cabs1, CSFX)(CAT_C(k + 1, k));
        for (r = k + 2; r < n; ++r) {
            m = CAT(cabs1, CSFX)(CAT_C(r, k));
            if (m > best) { best = m; p = r; }
        }
        ipiv[k + 1] = (int32_t)p;
        if (p != k + 1) CAT(cswap_indices, CSFX)(n, A, lda, k + 1, p);
        alpha = CAT_C(k + 1, k);
        for (r = k + 2; r < n; ++r) {
            if (CAT(cnonzero, CSFX)(alpha)) {
                CAT_C(r, k) = CAT(cdiv, CSFX)(CAT_C(r, k), alpha);
            } else {
                CAT_C(r, k).re = (REAL)0;
                CAT_C(r, k).im = (REAL)0;
            }
        }
        for (r = k + 2; r < n; ++r) v[r] = CAT_C(r, k + 1);
        for (j = k + 2; j < n; ++j) {
            CT lj = CAT_C(j, k), vj = v[j];
            for (i = j + 1; i < n; ++i) {
                CT t = CAT(csub, CSFX)(CAT(cmul, CSFX)(CAT_C(i, k), vj), CAT(cmul, CSFX)(v[i], lj));
                CAT_C(i, j) = CAT(cadd, CSFX)(CAT_C(i, j), t);
            }
        }
    }
    free(v);
}

/* Pfaffian from the factors, Pf(X) = det(P) prod_j (-alpha_{2j}), returned
 * as log|Pf| (fp64, sum of log|alpha_{2j}| in index order, |z| by hypot) and
 * the phase Pf / |Pf| (fp64, the running product of the unit factors
 * -alpha_{2j} / |alpha_{2j}| in index order, times det(P)).  Odd n or a zero
 * alpha_{2j}: logabs = -inf, phase 0. */
static void CAT(pfaffian, CSFX)(int64_t n, const CT* A, int64_t lda, const int32_t* ipiv,
                                double* logabs, double* phase)
{
    int64_t j, i;
    double acc = 0.0, pr = 1.0, pi = 0.0;
    if (n % 2 != 0) { *logabs = -INFINITY; phase[0] = 0.0; phase[1] = 0.0; return; }
    for (j = 0; 2 * j < n; ++j) {
        double ar = (double)A[(2 * j + 1) + (2 * j) * lda].re;
        double ai = (double)A[(2 * j + 1) + (2 * j) * lda].im;
        double mag = hypot(ar, ai);
        double ur, ui, tr;
        if (mag == 0.0) { *logabs = -INFINITY; phase[0] = 0.0; phase[1] = 0.0; return; }
        acc += log(mag);
        ur = -ar / mag;                           /* factor T(2j,2j+1) = -alpha, made unit */
        ui = -ai / mag;
        tr = pr * ur - pi * ui;
        pi = pr * ui + pi * ur;
        pr = tr;
    }
    for (i = 0; i < n; ++i)
        if (ipiv[i] != i) { pr = -pr; pi = -pi; }
    *logabs = acc;
    phase[0] = pr;
    phase[1] = pi;
}

#undef CAT_C
#undef CT
