/* CPU oracle for the convolution operator O = conv(F, I) and its im2col
 * transform.
 *
 * TEST INFRASTRUCTURE ONLY.  Plain, slow, scalar C that writes out the
 * definitions of the paper's section 3: the direct seven-loop convolution of
 * Figure 4 and the explicit im2col transform of Figure 5.  It shares no code,
 * header or constant with the GPU library; only the tests, the smoke check and
 * the benchmark's CPU baseline may load it.
 *
 * Storage (section 3, "Tensor data storage"): every tensor is a linear array
 * whose leftmost index runs fastest,
 *   I[h][w][c][b]   -> I[h + hi*(w + wi*(c + ci*b))]        (hi x wi x ci x b)
 *   F[k][y][x][c]   -> F[k + kn*(y + kh*(x + kw*c))]        (kn x kh x kw x ci)
 *   O[k][oh][ow][b] -> O[k + kn*(oh + ho*(ow + wo*b))]      (kn x ho x wo x b)
 * with ho = floor((hi - kh + 2p)/s) + 1 and wo likewise (section 3).
 *
 * Padding: the figures index the input as I[s*i_h + i_kh][s*i_w + i_kw] with no
 * padding term.  With padding p the input is read as if p zero rows and
 * columns surrounded it: the entry used is I[s*i_h + i_kh - p][s*i_w + i_kw - p],
 * and a position outside 0..hi-1 or 0..wi-1 contributes zero.  For p = 0 this
 * is exactly the figures' indexing.
 *
 * Precision: inputs are fp32 (the paper's experiments use single precision);
 * every product of two fp32 values is exact in fp64 and the sums run in fp64,
 * in the loop order of Figure 4.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC.
 * OpenMP splits only the outermost loop over the batch index i_b; each thread
 * owns whole output samples, so the results do not depend on the thread count.
 */
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int g_threads = 0;

void oracle_conv_set_threads(int32_t t) { g_threads = t; }

int32_t oracle_conv_get_threads(void)
{
#ifdef _OPENMP
    return g_threads > 0 ? g_threads : omp_get_max_threads();
#else
    return 1;
#endif
}

/* Direct realization of O = conv(F, I) (section 3, Figure 4).  O (fp64,
 * kn x ho x wo x b) is overwritten. */
void oracle_conv_direct(int64_t kn, int64_t kh, int64_t kw, int64_t ci, int64_t hi, int64_t wi,
                        int64_t b, int64_t s, int64_t p, const float* F, const float* I, double* O)
{
    const int64_t ho = (hi - kh + 2 * p) / s + 1;
    const int64_t wo = (wi - kw + 2 * p) / s + 1;
    memset(O, 0, sizeof(double) * (size_t)(kn * ho * wo * b));
    int64_t ib;
#ifdef _OPENMP
#pragma omp parallel for schedule(static) num_threads(oracle_conv_get_threads())
#endif
    for (ib = 0; ib < b; ++ib)                                      /* L1 */
        for (int64_t ic = 0; ic < ci; ++ic)                         /* L2 */
            for (int64_t iw = 0; iw < wo; ++iw)                     /* L3 */
                for (int64_t ih = 0; ih < ho; ++ih)                 /* L4 */
                    for (int64_t ikw = 0; ikw < kw; ++ikw) {        /* L5 */
                        const int64_t x = s * iw + ikw - p;
                        if (x < 0 || x >= wi) continue;
                        for (int64_t ikh = 0; ikh < kh; ++ikh) {    /* L6 */
                            const int64_t y = s * ih + ikh - p;
                            if (y < 0 || y >= hi) continue;
                            const double v = (double)I[y + hi * (x + wi * (ic + ci * ib))];
                            const float* f = F + kn * (ikh + kh * (ikw + kw * ic));
                            double* o = O + kn * (ih + ho * (iw + wo * ib));
                            for (int64_t ik = 0; ik < kn; ++ik)     /* L7 */
                                o[ik] += (double)f[ik] * v;
                        }
                    }
}

/* Explicit im2col transform (section 3, Figure 5): the augmented matrix
 * B (K x N, column-major, K = kh*kw*ci, N = ho*wo*b) with
 *   row    r = i_kh + i_kw*kh + i_c*kw*kh,
 *   column c = i_h + i_w*ho + i_b*ho*wo,
 *   B[r][c] = I[s*i_h + i_kh - p][s*i_w + i_kw - p][i_c][i_b]  (zero outside).
 * The figure's column formula prints hi, wi where the output sizes belong; the
 * columns of B are the ho*wo*b output positions. */
void oracle_im2col(int64_t kh, int64_t kw, int64_t ci, int64_t hi, int64_t wi, int64_t b, int64_t s,
                   int64_t p, const float* I, float* B)
{
    const int64_t ho = (hi - kh + 2 * p) / s + 1;
    const int64_t wo = (wi - kw + 2 * p) / s + 1;
    const int64_t K = kh * kw * ci;
    int64_t ib;
#ifdef _OPENMP
#pragma omp parallel for schedule(static) num_threads(oracle_conv_get_threads())
#endif
    for (ib = 0; ib < b; ++ib)
        for (int64_t ic = 0; ic < ci; ++ic)
            for (int64_t iw = 0; iw < wo; ++iw)
                for (int64_t ih = 0; ih < ho; ++ih) {
                    const int64_t c = ih + iw * ho + ib * ho * wo;
                    for (int64_t ikw = 0; ikw < kw; ++ikw)
                        for (int64_t ikh = 0; ikh < kh; ++ikh) {
                            const int64_t r = ikh + ikw * kh + ic * kw * kh;
                            const int64_t y = s * ih + ikh - p;
                            const int64_t x = s * iw + ikw - p;
                            B[r + K * c] = (y < 0 || y >= hi || x < 0 || x >= wi)
                                               ? 0.0f
                                               : I[y + hi * (x + wi * (ic + ci * ib))];
                        }
                }
}

/* Selected entries of O = conv(F, I), each from its definition (the sum of
 * Figure 4 over i_c, i_kw, i_kh for one (i_k, i_h, i_w, i_b)), for checking
 * sampled outputs of problems too large for the full direct loops.
 * pts holds npts quadruples (i_k, i_h, i_w, i_b); out[t] receives the sum. */
void oracle_conv_points(int64_t kn, int64_t kh, int64_t kw, int64_t ci, int64_t hi, int64_t wi,
                        int64_t b, int64_t s, int64_t p, const float* F, const float* I,
                        int64_t npts, const int64_t* pts, double* out)
{
    (void)b;
    int64_t t;
#ifdef _OPENMP
#pragma omp parallel for schedule(static) num_threads(oracle_conv_get_threads())
#endif
    for (t = 0; t < npts; ++t) {
        const int64_t ik = pts[4 * t], ih = pts[4 * t + 1], iw = pts[4 * t + 2], ib = pts[4 * t + 3];
        double acc = 0.0;
        for (int64_t ic = 0; ic < ci; ++ic)
            for (int64_t ikw = 0; ikw < kw; ++ikw) {
                const int64_t x = s * iw + ikw - p;
                if (x < 0 || x >= wi) continue;
                for (int64_t ikh = 0; ikh < kh; ++ikh) {
                    const int64_t y = s * ih + ikh - p;
                    if (y < 0 || y >= hi) continue;
                    acc += (double)F[ik + kn * (ikh + kh * (ikw + kw * ic))] *
                           (double)I[y + hi * (x + wi * (ic + ci * ib))];
                }
            }
        out[t] = acc;
    }
}
