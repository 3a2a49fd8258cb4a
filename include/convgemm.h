/*
 * convgemm.h -- C ABI of the MI355X (gfx950) CONVGEMM convolution: the
 * convolution operator computed as one matrix product whose second operand,
 * the im2col matrix, is assembled from the input tensor while it is staged
 * into on-chip memory and never exists in device memory.
 *
 * The operation (the paper's section 3, Figure 4; the GEMM form of section 4).
 * A convolution layer with kn filters of size kh x kw x ci, applied with
 * stride s and zero padding p to b inputs of size hi x wi x ci, gives b outputs
 * of size ho x wo x kn with
 *        ho = floor((hi - kh + 2p)/s) + 1,   wo = floor((wi - kw + 2p)/s) + 1,
 *        O[k][oh][ow][n] = sum over c, y, x of
 *                          F[k][y][x][c] * I[s*oh + y - p][s*ow + x - p][c][n]
 * where an input position outside 0..hi-1 / 0..wi-1 reads zero (for p = 0
 * this is exactly Figure 4's indexing).  Equivalently (section 4)
 *        O = F^ . im2col(I),   F^ : kn x (kh kw ci),   im2col(I) : (kh kw ci) x (ho wo b),
 * with im2col row r = y + x*kh + c*kh*kw and column j = oh + ow*ho + n*ho*wo
 * (Figures 5 and 6).
 *
 * Storage (section 3, "Tensor data storage"): the leftmost index runs
 * fastest, with no padding between dimensions:
 *        I[h][w][c][n]   at I[h + hi*(w + wi*(c + ci*n))]
 *        F[k][y][x][c]   at F[k + kn*(y + kh*(x + kw*c))]   (= F^ column-major, ld kn)
 *        O[k][oh][ow][n] at O[k + kn*(oh + ho*(ow + wo*n))]  (= O^ column-major, ld kn)
 *
 * Rules (as in ltlt.h): pointers are DEVICE pointers of the current HIP
 * device; the call is stream-ordered and asynchronous; the caller owns every
 * buffer and nothing is retained; the library allocates nothing for this call.
 * Return value: 0 on success (also when b = 0: nothing to do); -i when argument
 * i (1-based) is invalid, with nothing enqueued; CONVGEMM_ERR_HIP_BASE - e for
 * a HIP runtime error e.  Arithmetic is IEEE fp32 (the paper's experiments use
 * single precision), products and sums on the fp32 matrix cores; the order of
 * the sums is unspecified, so results agree with an exact evaluation within
 * the usual fp32 bound |error| <= gamma_K * sum |F| |I| (K = kh kw ci), and are
 * exact whenever every partial sum is an integer below 2^24.  For short
 * grids with long contractions the automatic choice splits a tile's
 * contraction over several workgroups that add into O atomically, so the
 * last bits of such a call may differ from one run to the next.  O may not
 * overlap F or I.
 */
#ifndef CONVGEMM_H
#define CONVGEMM_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CONVGEMM_OK 0
#define CONVGEMM_ERR_HIP_BASE (-1000) /* returned as CONVGEMM_ERR_HIP_BASE - (int)hipError_t */

/* Output extent floor((h - k + 2 pad)/stride) + 1 of one spatial dimension
 * (section 3), or -1 when the window does not fit the padded input or an
 * argument is out of range (k < 1, stride < 1, pad < 0).  Host only. */
int convgemm_out_size(int h, int k, int stride, int pad);

/* O = conv(F, I) (accumulate = 0) or O += conv(F, I) (accumulate = 1), as one
 * implicit-im2col GEMM on the fp32 matrix cores (section 4, Figure 6).
 *   kn, kh, kw, ci : filter count and size (all >= 1);
 *   hi, wi         : input height and width (>= 1, with hi + 2 pad >= kh and
 *                    wi + 2 pad >= kw);
 *   b              : batch size (>= 0);
 *   stride >= 1, pad >= 0;
 *   F, I, O        : tensors in the storage above (O: kn*ho*wo*b floats);
 *   path           : 0 = chosen from the sizes (then mt = nt = 0);
 *                    1 = LDS-staged gather (any stride and padding), tile
 *                        (mt, nt) one of (64, 64), (64, 128), (64, 256),
 *                        (128, 128), (192, 128), or (0, 0) = chosen;
 *                    2 = register-direct (no LDS staging; pad must be 0 and
 *                        kh*kw*ci <= 16384), tile one of (64, 64), (64, 128),
 *                        (128, 64), (128, 128), or (0, 0) = chosen.
 *                    Paths and tiles are for tests and tuning: every choice
 *                    gives results within the bound above.  An invalid path
 *                    or path/padding/size combination is argument 14, an
 *                    invalid tile argument 15.
 * Limits (else the argument named is reported invalid): hi*wi*ci and
 * kh*kw*ci below 2^31 (hi, kh); ho*wo*b below 2^31 and the whole input
 * hi*wi*ci*b below 2^30 elements, 4 GiB (b); kn below 2^24 and the filter
 * tensor kn*kh*kw*ci below 2^30 elements (kn). */
int convgemm_f32(int kn, int kh, int kw, int ci, int hi, int wi, int b, int stride, int pad,
                 const float* F, const float* I, float* O, int accumulate, int path, int mt, int nt,
                 hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* CONVGEMM_H */
