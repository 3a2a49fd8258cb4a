// Batched small-n path: one 256-thread workgroup factors one matrix of order
// n <= 64 entirely in LDS (full skew storage, both triangles, padded rows),
// runs every column step of the pivoted reduction (pivot search by one wave,
// symmetric exchange of two rows and two columns, multipliers, skew rank-2
// update of the trailing lower triangle with its mirror), then writes the
// strict lower triangle back and computes the Pfaffian.  Global traffic is one
// read and one write of each matrix's strict lower triangle, coalesced per
// column, which is what bounds this path (HBM).

#include "ltlt_device.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int kBN = 64;            // largest order handled
constexpr int kBP = kBN + 1;       // padded LDS row length

template <typename T>
__global__ void __launch_bounds__(256) batched_kernel(int n, T* Aall, int64_t lda, int64_t strideA, int* ipiv_all,
                                                      int64_t strideIpiv, double* logabs, int* sign) {
  __shared__ T S[kBN * kBP];       // S[i*kBP + c] = X(i, c)
  __shared__ int s_p;
  __shared__ int s_piv[kBN];
  const int tid = threadIdx.x;
  const int64_t bidx = blockIdx.x;
  T* A = Aall + bidx * strideA;
  int* ipiv = ipiv_all + bidx * strideIpiv;

  // load strict lower triangle (column c, rows c+1..n-1 contiguous) and mirror
  for (int e = tid; e < n * n; e += 256) {
    const int c = e / n, i = e % n;
    if (i > c) {
      const T v = A[(int64_t)i + (int64_t)c * lda];
      S[i * kBP + c] = v;
      S[c * kBP + i] = -v;
    } else if (i == c) {
      S[i * kBP + i] = T(0);
    }
  }
  for (int i = tid; i < n; i += 256) s_piv[i] = i;
  __syncthreads();

  for (int k = 0; k + 2 < n; ++k) {
    // pivot: first maximum of |X(r,k)|, r >= k+1 (at most 63 candidates)
    if (tid < kWave) {
      const int r = k + 1 + tid;
      double bv = -1.0;
      int bi = INT32_MAX;
      if (r < n) { bv = (double)fabs(S[r * kBP + k]); bi = r; }
      wave_argmax(bv, bi);
      if (tid == 0) s_p = (bi == INT32_MAX) ? k + 1 : bi;
    }
    __syncthreads();
    const int p = s_p;
    if (p != k + 1) {
      // rows k+1 <-> p over all columns, then columns k+1 <-> p over all rows
      for (int c = tid; c < n; c += 256) {
        const T t0 = S[(k + 1) * kBP + c];
        S[(k + 1) * kBP + c] = S[p * kBP + c];
        S[p * kBP + c] = t0;
      }
      __syncthreads();
      for (int r = tid; r < n; r += 256) {
        const T t0 = S[r * kBP + (k + 1)];
        S[r * kBP + (k + 1)] = S[r * kBP + p];
        S[r * kBP + p] = t0;
      }
      if (tid == 0) s_piv[k + 1] = p;
      __syncthreads();
    }
    const T alpha = S[(k + 1) * kBP + k];
    // multipliers
    for (int r = k + 2 + tid; r < n; r += 256)
      S[r * kBP + k] = (alpha != T(0)) ? S[r * kBP + k] / alpha : T(0);
    __syncthreads();
    // skew rank-2 update of the trailing strict lower triangle (+ mirror)
    const int m = n - (k + 2);
    for (int e = tid; e < m * m; e += 256) {
      const int i = k + 2 + e / m, c = k + 2 + e % m;
      if (i > c) {
        const T li = S[i * kBP + k], lc = S[c * kBP + k];
        const T vi = S[i * kBP + k + 1], vc = S[c * kBP + k + 1];
        const T val = S[i * kBP + c] + (li * vc - vi * lc);
        S[i * kBP + c] = val;
        S[c * kBP + i] = -val;
      }
    }
    __syncthreads();
  }

  // write back strict lower triangle and pivots
  for (int e = tid; e < n * n; e += 256) {
    const int c = e / n, i = e % n;
    if (i > c) A[(int64_t)i + (int64_t)c * lda] = S[i * kBP + c];
  }
  for (int i = tid; i < n; i += 256) ipiv[i] = s_piv[i];
  // Pfaffian (one wave, fixed order)
  if (tid < kWave) {
    double lg = 0.0;
    int neg = 0, zero = 0;
    if ((n & 1) == 0) {
      for (int jj = tid; jj < n / 2; jj += kWave) {
        const double al = (double)S[(2 * jj + 1) * kBP + 2 * jj];
        if (al == 0.0) zero = 1;
        else { lg += log(fabs(al)); if (-al < 0.0) neg ^= 1; }
      }
      for (int i = tid; i < n; i += kWave)
        if (s_piv[i] != i) neg ^= 1;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      lg += __shfl_xor(lg, off, kWave);
      neg ^= __shfl_xor(neg, off, kWave);
      zero |= __shfl_xor(zero, off, kWave);
    }
    if (tid == 0) {
      if ((n & 1) || zero) { logabs[bidx] = -INFINITY; sign[bidx] = 0; }
      else { logabs[bidx] = lg; sign[bidx] = neg ? -1 : 1; }
    }
  }
}

template <typename T>
hipError_t launch_batched(int n, int batch, T* A, int64_t lda, int64_t strideA, int* ipiv, int64_t strideIpiv,
                          double* logabs, int* sign, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(batched_kernel<T>, dim3(batch), dim3(256), 0, s, n, A, lda, strideA, ipiv, strideIpiv, logabs,
                     sign);
  return hipGetLastError();
}

template hipError_t launch_batched<double>(int, int, double*, int64_t, int64_t, int*, int64_t, double*, int*,
                                           hipStream_t);
template hipError_t launch_batched<float>(int, int, float*, int64_t, int64_t, int*, int64_t, double*, int*,
                                          hipStream_t);

}  // namespace ltlt
