// Bandwidth-bound helper kernels of the blocked factorization and the
// Pfaffian reduction.
//
//  init        ipiv = identity, status cleared.
//  commit      after a block's trailing update: alphas, the block's
//              multiplier columns and the carry column go into A.
//  perm_chain  composition of the per-block row orders.  A block's
//              exchanges reorder the rows of every earlier multiplier column;
//              instead of swapping those rows once per block, the final row
//              order of block J's columns is G_J = T_{J+1} o T_{J+2} o ... ,
//              computed per row with one dependent lookup per later block.
//  perm_apply  gathers every multiplier column into its final row order: one
//              workgroup per column stages the column in LDS (or, for columns
//              longer than LDS holds, in a per-workgroup global slot) and
//              writes it back through G_J.
//  pfaffian    log|Pf| = sum_j log|alpha_{2j}| in fp64 and the sign
//              (-1)^(n/2) * prod sign(alpha_{2j}) * (-1)^(#exchanges),
//              one fixed-order tree reduction.

#include <algorithm>

#include "ltlt_device.h"
#include "ltlt_internal.h"

namespace ltlt {

// status[0] (this call's abort flag) starts cleared; with `force` both words
// are raised instead, as if a wait had already given up (the host-side switch
// that tests the failure path without any kernel waiting for long).
__global__ void init_kernel(int* ipiv, int n, int* status, int force) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = t; i < n; i += stride) ipiv[i] = (int)i;
  if (t == 0) {
    status[0] = force;
    if (force) status[1] = 1;
  }
}

hipError_t launch_init(int* ipiv, int n, int* status, hipStream_t s) {
  int blocks = (int)((n + 255) / 256);
  if (blocks < 1) blocks = 1;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(init_kernel, dim3(blocks), dim3(256), 0, s, ipiv, n, status, forced_timeout() ? 1 : 0);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// After a panel whose wait gave up (status[0] raised) the block's outputs were
// never formed: NaN is committed instead, so that no aborted call leaves
// plausible factors behind.
template <typename T>
__global__ void commit_kernel(T* A, int64_t lda, int n, int j, int bw, const T* PO, int64_t ldw, const T* alpha,
                              const int* status) {
  const int u = blockIdx.y;                   // 0..bw (bw = carry column)
  const int col = j + u;
  const bool failed = status[0] != 0;
  for (int i = col + 1 + blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    T v;
    if (u < bw && i == col + 1) v = alpha[u];
    else v = PO[(int64_t)(i - (j + 1)) + (int64_t)u * ldw];
    A[(int64_t)i + (int64_t)col * lda] = failed ? T(NAN) : v;
  }
}

template <typename T>
hipError_t launch_commit(T* A, int64_t lda, int n, int j, int bw, const T* PO, int64_t ldw, const T* alpha,
                         const int* status, hipStream_t s) {
  const int rows = n - (j + 1);
  if (rows <= 0) return hipSuccess;
  int bx = (rows + 255) / 256;
  if (bx > 64) bx = 64;
  hipLaunchKernelGGL(commit_kernel<T>, dim3(bx, bw + 1), dim3(256), 0, s, A, lda, n, j, bw, PO, ldw, alpha,
                     status);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Blocks are uniform: block J starts at column J*nb.
// Tblk[J*n + i] = index held at the start of block J by position i (i > J*nb);
// G[J*n + i] = source row of position i for the columns of block J (J < nblk-1).
// Every looked-up index is clamped into the positions of its block,
// [nxt*nb + 1, n): a complete block order is unchanged by that, and an order
// left unfinished by a panel that gave up (status raised) cannot send a later
// lookup, or perm_apply's gather, out of bounds.
__global__ void perm_chain_kernel(const int* Tblk, int nb, int nblk, int n, int* G) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int g = i;
  for (int J = nblk - 2; J >= 0; --J) {
    const int nxt = J + 1;
    if (g > nxt * nb) g = min(max(Tblk[(int64_t)nxt * n + g], nxt * nb + 1), n - 1);
    G[(int64_t)J * n + i] = g;
  }
}

hipError_t launch_perm_chain(const int* Tblk, int nb, int nblk, int n, int* G, hipStream_t s) {
  if (nblk < 2 || n <= 0) return hipSuccess;
  hipLaunchKernelGGL(perm_chain_kernel, dim3((n + 255) / 256), dim3(256), 0, s, Tblk, nb, nblk, n, G);
  return hipGetLastError();
}

constexpr size_t kPermLds = 150 * 1024;      // column staging in LDS up to this size
constexpr int kPermGlobalWgs = 256;          // workgroups when staging in global memory

// Column c belongs to block J = c / nb; rows below that block (from
// r0 = J*nb + nb + 1 on) are reordered: A(i, c) <- A(G_J[i], c).
template <typename T, bool IN_LDS>
__global__ void __launch_bounds__(256) perm_apply_kernel(T* A, int64_t lda, int n, const int* G, int nb, int c_end,
                                                         T* stage) {
  extern __shared__ __align__(16) unsigned char smem[];
  T* buf = IN_LDS ? reinterpret_cast<T*>(smem) : stage + (int64_t)blockIdx.x * n;
  for (int c = blockIdx.x; c < c_end; c += gridDim.x) {
    const int J = c / nb;
    const int r0 = J * nb + nb + 1;
    const int len = n - r0;
    if (len <= 0) continue;                    // uniform across the workgroup
    T* col = A + (int64_t)c * lda + r0;
    // 8 independent loads in flight per thread per round
    constexpr int kU = 8;
    for (int i0 = threadIdx.x; i0 < len; i0 += kU * blockDim.x) {
      T v[kU];
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const int i = i0 + e * blockDim.x;
        v[e] = col[i < len ? i : 0];
      }
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const int i = i0 + e * blockDim.x;
        if (i < len) buf[i] = v[e];
      }
    }
    __syncthreads();
    const int* g = G + (int64_t)J * n + r0;
    for (int i0 = threadIdx.x; i0 < len; i0 += kU * blockDim.x) {
      int src[kU];
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const int i = i0 + e * blockDim.x;
        src[e] = min(max(g[i < len ? i : 0] - r0, 0), len - 1);   // in the column whatever G holds
      }
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const int i = i0 + e * blockDim.x;
        if (i < len) col[i] = buf[src[e]];
      }
    }
    __syncthreads();
  }
}

template <typename T>
size_t perm_stage_elems(int n, int c_end) {
  if ((size_t)n * sizeof(T) <= kPermLds || c_end <= 0) return 0;
  return (size_t)std::min(c_end, kPermGlobalWgs) * (size_t)n;
}

template <typename T>
hipError_t launch_perm_apply(T* A, int64_t lda, int n, const int* G, int nb, int c_end, T* stage, hipStream_t s) {
  if (c_end <= 0) return hipSuccess;
  const size_t bytes = (size_t)n * sizeof(T);
  if (bytes <= kPermLds) {
    const hipError_t e = ensure_dynamic_lds((const void*)perm_apply_kernel<T, true>, (int)kPermLds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((perm_apply_kernel<T, true>), dim3(c_end), dim3(256), bytes, s, A, lda, n, G, nb, c_end,
                       (T*)nullptr);
  } else {
    const int wgs = std::min(c_end, kPermGlobalWgs);
    hipLaunchKernelGGL((perm_apply_kernel<T, false>), dim3(wgs), dim3(256), 0, s, A, lda, n, G, nb, c_end, stage);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// A raised abort flag (status[0]: a wait of the last factorization gave up)
// gives log|Pf| = NaN and sign 0.
template <typename T>
__global__ void __launch_bounds__(1024) pfaffian_kernel(int n, const T* A, int64_t lda, const int* ipiv,
                                                        double* logabs, int* sign, const int* status) {
  __shared__ double s_log[1024];
  __shared__ int s_neg[1024], s_zero[1024];
  const int tid = threadIdx.x;
  double lg = 0.0;
  int neg = 0, zero = 0;
  const int half = n / 2;
  if ((n & 1) == 0) {
    for (int jj = tid; jj < half; jj += 1024) {
      const double al = (double)A[(int64_t)(2 * jj + 1) + (int64_t)(2 * jj) * lda];
      if (al == 0.0) zero = 1;
      else {
        lg += log(fabs(al));
        if (-al < 0.0) neg ^= 1;             // factor T(2j,2j+1) = -alpha_{2j}
      }
    }
    for (int i = tid; i < n; i += 1024)
      if (ipiv[i] != i) neg ^= 1;
  }
  s_log[tid] = lg; s_neg[tid] = neg; s_zero[tid] = zero;
  __syncthreads();
  for (int st = 512; st >= 1; st >>= 1) {
    if (tid < st) {
      s_log[tid] += s_log[tid + st];
      s_neg[tid] ^= s_neg[tid + st];
      s_zero[tid] |= s_zero[tid + st];
    }
    __syncthreads();
  }
  if (tid == 0) {
    if (status[0] != 0) { *logabs = NAN; *sign = 0; }
    else if (n & 1 || s_zero[0]) { *logabs = -INFINITY; *sign = 0; }
    else { *logabs = s_log[0]; *sign = s_neg[0] ? -1 : 1; }
  }
}

template <typename T>
hipError_t launch_pfaffian(int n, const T* A, int64_t lda, const int* ipiv, double* logabs, int* sign,
                           const int* status, hipStream_t s) {
  hipLaunchKernelGGL(pfaffian_kernel<T>, dim3(1), dim3(1024), 0, s, n, A, lda, ipiv, logabs, sign, status);
  return hipGetLastError();
}

#define LTLT_INST(T)                                                                                         \
  template hipError_t launch_commit<T>(T*, int64_t, int, int, int, const T*, int64_t, const T*, const int*,   \
                                      hipStream_t);                                                         \
  template hipError_t launch_perm_apply<T>(T*, int64_t, int, const int*, int, int, T*, hipStream_t);        \
  template size_t perm_stage_elems<T>(int, int);                                                            \
  template hipError_t launch_pfaffian<T>(int, const T*, int64_t, const int*, double*, int*, const int*,     \
                                         hipStream_t);
LTLT_INST(double)
LTLT_INST(float)
#undef LTLT_INST

}  // namespace ltlt
