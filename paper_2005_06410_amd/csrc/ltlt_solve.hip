// Solve X x = b with the factors of ltlt_factor.  With P X P^T = L T L^T,
// X x = b is L T L^T (P x) = P b, so (per right-hand side)
//   y = P b            y[i] = b[perm[i]], perm = the exchanges (i, ipiv[i])
//                      applied in order to the identity ordering;
//   z = L^{-1} y       forward substitution, L unit lower with L(:,0) = e_0
//                      and L(r, c) = A(r, c-1) for r >= c+1 (packed storage);
//   w = T^{-1} z       T skew tridiagonal, T(k+1,k) = alpha_k = A(k+1,k): row 0
//                      and the even rows give the odd unknowns forward, row
//                      n-1 and the odd rows the even unknowns backward;
//   u = L^{-T} w       backward substitution;
//   x = P^T u          x[perm[i]] = u[i].
//
// gfx950 mapping:
//  * perm: one thread applies the n exchanges to an index array in LDS
//    (ipiv[i] >= i, so position i is final once step i is done);
//  * the triangular solves are persistent cooperative kernels over 64-row
//    blocks, left-looking: the workgroup of block b streams the 64x64 tiles
//    of L to the left of its diagonal block (forward) or below it (backward)
//    through LDS, waiting for the flag of the block each tile multiplies,
//    then solves its diagonal block (one wave per right-hand side, the
//    unknown broadcast by readlane) and raises its own flag.  A workgroup
//    takes its blocks in dependency order, so the earliest unfinished block
//    always has its inputs and the grid cannot deadlock; every wait is
//    bounded.  Each solve reads the lower triangle of L once: HBM-bound for
//    few right-hand sides;
//  * the recurrences of T run one lane per (right-hand side, chain), with
//    the reciprocals of alpha formed in parallel beforehand.
// Right-hand sides are taken kSolveRhs at a time.

#include "ltlt_device.h"
#include "ltlt_exchange.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int kSB = 64;                // rows per block
constexpr int kSLd = kSB + 1;          // LDS stride of a tile column (bank spread)
constexpr int kSThreads = 256;         // 4 waves
constexpr int kSGroups = kSThreads / kSB;   // column (or row) groups of a tile
constexpr int kSCols = kSB / kSGroups;      // 16 columns per group

// ---- permutation ----------------------------------------------------------
// at[i] = index of the row at position i after the exchanges (i, ipiv[i]),
// i = 0 .. n-1, in order.  With use_lds the index array and a copy of ipiv
// sit in LDS (8 n bytes); otherwise the index array is in global scratch and
// ipiv is read from global memory (slow: one dependent access per step).
__global__ void __launch_bounds__(256) solve_perm_kernel(int n, const int* ipiv, int* perm, int* gscratch,
                                                         int use_lds) {
  extern __shared__ int slds[];
  int* at = use_lds ? slds : gscratch;
  const int* piv = ipiv;
  if (use_lds) {
    int* sp = slds + n;
    for (int i = threadIdx.x; i < n; i += blockDim.x) sp[i] = ipiv[i];
    piv = sp;
  }
  for (int i = threadIdx.x; i < n; i += blockDim.x) at[i] = i;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 0; i < n; ++i) {
      const int p = piv[i];
      const int x = at[i], y = at[p];
      at[i] = y;
      at[p] = x;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) perm[i] = at[i];
}

template <typename T>
__global__ void solve_gather_kernel(int n, int nr, const int* perm, const T* B, int64_t ldb, T* Y, int64_t ldy) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int q = blockIdx.y;
  if (i < n && q < nr) Y[(int64_t)i + (int64_t)q * ldy] = B[(int64_t)perm[i] + (int64_t)q * ldb];
}

template <typename T>
__global__ void solve_scatter_kernel(int n, int nr, const int* perm, const T* Y, int64_t ldy, T* B, int64_t ldb) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int q = blockIdx.y;
  if (i < n && q < nr) B[(int64_t)perm[i] + (int64_t)q * ldb] = Y[(int64_t)i + (int64_t)q * ldy];
}

// alpha_k = A(k+1, k) and its reciprocal, k < n-1
template <typename T>
__global__ void solve_alpha_kernel(int n, const T* A, int64_t lda, T* alpha, T* ralpha) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k + 1 < n) {
    const T a = A[(int64_t)(k + 1) + (int64_t)k * lda];
    alpha[k] = a;
    ralpha[k] = T(1) / a;
  }
}

__global__ void solve_flags_kernel(int* flags, int count) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) flags[i] = 0;
}

// ---- skew tridiagonal recurrences -----------------------------------------
// lane l < nr: odd unknowns of right-hand side l, forward; lane 32 + l: even
// unknowns, backward.  Each chain reads the inputs of the other chain's
// parity, so the result goes to a separate buffer W.
template <typename T>
__global__ void __launch_bounds__(64) solve_tridiag_kernel(int n, int nr, const T* alpha, const T* ralpha,
                                                           const T* Y, T* W, int64_t ldy) {
  const int lane = threadIdx.x;
  const int q = lane & 31;
  if (q >= nr) return;
  const T* y = Y + (int64_t)q * ldy;
  T* wv = W + (int64_t)q * ldy;
  if (lane < 32) {
    // W[1] = -R[0] / alpha_0;  W[i+1] = (alpha_{i-1} W[i-1] - R[i]) / alpha_i, i even
    T wprev = -y[0] * ralpha[0];
    wv[1] = wprev;
    for (int i = 2; i + 1 < n; i += 2) {
      const T w = (alpha[i - 1] * wprev - y[i]) * ralpha[i];
      wv[i + 1] = w;
      wprev = w;
    }
  } else {
    // W[n-2] = R[n-1] / alpha_{n-2};  W[i-1] = (R[i] + alpha_i W[i+1]) / alpha_{i-1}, i odd
    T wnext = y[n - 1] * ralpha[n - 2];
    wv[n - 2] = wnext;
    for (int i = n - 3; i >= 1; i -= 2) {
      const T w = (y[i] + alpha[i] * wnext) * ralpha[i - 1];
      wv[i - 1] = w;
      wnext = w;
    }
  }
}

// ---- triangular solves ----------------------------------------------------
struct SolveTriArgs {
  const void* A;
  int64_t lda;
  int n;
  int nblk;
  void* Y;
  int64_t ldy;
  int nr;             // right-hand sides of this pass (<= kSolveRhs)
  int* flag;          // [nblk], 0 = not yet solved
  int* status;
};

// L(r, c) for global row r and column c: unit lower, L(:,0) = e_0,
// L(r, c) = A(r, c-1) below the diagonal.
template <typename T>
__device__ __forceinline__ T l_entry(const T* A, int64_t lda, int n, int r, int c) {
  if (r >= n || c >= n || r <= c || c == 0) return T(0);
  return A[(int64_t)r + (int64_t)(c - 1) * lda];
}

// Tile of L: rows r0 .. r0+63, columns c0 .. c0+63, into LDS column by column
// (tile[cc * kSLd + r]); thread t loads column (t / 64) + 4 j, row t % 64, so
// every wave instruction reads 64 consecutive rows of one column.
template <typename T>
__device__ __forceinline__ void load_l_tile(const T* A, int64_t lda, int n, int r0, int c0, T* tile, int tid) {
  const int r = tid & (kSB - 1);
  const int g = tid / kSB;
#pragma unroll
  for (int jj = 0; jj < kSCols; ++jj) {
    const int cc = g + kSGroups * jj;
    tile[cc * kSLd + r] = l_entry(A, lda, n, r0 + r, c0 + cc);
  }
}

template <typename T>
__device__ __forceinline__ bool wait_flag(int* flag, int* status, int& s_abort) {
  if (threadIdx.x == 0) {
    const uint64_t t0 = wall_ticks();
    while (ld_coh(flag) == 0) {
      if (ld_coh(status) != 0 || wall_ticks() - t0 > kWaitLimitTicks) {
        atomicOr(status, 1);
        s_abort = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
  return s_abort == 0;
}

// Forward: z_b = y_b - sum_{c<b} L_bc z_c, then z_b = L_bb^{-1} z_b.
template <typename T>
__global__ void __launch_bounds__(kSThreads, 1) solve_lower_kernel(SolveTriArgs a) {
  __shared__ T tile[kSB * kSLd];
  __shared__ T yc[kSB * kSolveRhs];                // z of the block a tile multiplies
  __shared__ T part[kSGroups * kSB * kSolveRhs];   // partial sums of the four column groups
  __shared__ int s_abort;
  const T* A = static_cast<const T*>(a.A);
  T* Y = static_cast<T*>(a.Y);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int r = tid & (kSB - 1), g = tid / kSB;
  const int n = a.n, nr = a.nr;
  if (tid == 0) s_abort = 0;
  __syncthreads();
  for (int b = blockIdx.x; b < a.nblk; b += gridDim.x) {
    const int r0 = b * kSB;
    T acc[kSolveRhs];
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) acc[q] = T(0);
    for (int c = 0; c < b; ++c) {
      const int c0 = c * kSB;
      load_l_tile(A, a.lda, n, r0, c0, tile, tid);
      if (!wait_flag<T>(&a.flag[c], a.status, s_abort)) return;
      for (int e = tid; e < kSB * nr; e += kSThreads) {
        const int rr = e % kSB, q = e / kSB;
        yc[rr * kSolveRhs + q] = (c0 + rr < n) ? ld_coh_t(&Y[(int64_t)(c0 + rr) + (int64_t)q * a.ldy]) : T(0);
      }
      __syncthreads();
#pragma unroll 4
      for (int jj = 0; jj < kSCols; ++jj) {
        const int cc = g * kSCols + jj;
        const T lv = tile[cc * kSLd + r];
#pragma unroll
        for (int q = 0; q < kSolveRhs; ++q)
          if (q < nr) acc[q] = fma(lv, yc[cc * kSolveRhs + q], acc[q]);
      }
      __syncthreads();
    }
    // sum the four groups, subtract from y_b
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) part[(g * kSB + r) * kSolveRhs + q] = acc[q];
    load_l_tile(A, a.lda, n, r0, r0, tile, tid);
    __syncthreads();
    // diagonal block: wave w solves right-hand sides w, w+4; lane = row
    for (int q = wave; q < nr; q += kSThreads / kWave) {
      T x = T(0);
      if (r0 + lane < n) {
        x = ld_coh_t(&Y[(int64_t)(r0 + lane) + (int64_t)q * a.ldy]);
        T s = T(0);
#pragma unroll
        for (int gg = 0; gg < kSGroups; ++gg) s += part[(gg * kSB + lane) * kSolveRhs + q];
        x -= s;
      }
#pragma unroll 8
      for (int cc = 0; cc < kSB; ++cc) {
        const T xc = __shfl(x, cc, kWave);
        if (lane > cc) x = fma(-tile[cc * kSLd + lane], xc, x);
      }
      if (r0 + lane < n) st_coh_t(&Y[(int64_t)(r0 + lane) + (int64_t)q * a.ldy], x);
    }
    wait_stores();
    __syncthreads();
    if (tid == 0) st_coh(&a.flag[b], 1);
  }
}

// Backward: u_b = w_b - sum_{b'>b} L_{b'b}^T u_{b'}, then u_b = L_bb^{-T} u_b.
// Blocks are taken from the last one down.
template <typename T>
__global__ void __launch_bounds__(kSThreads, 1) solve_upper_kernel(SolveTriArgs a) {
  __shared__ T tile[kSB * kSLd];
  __shared__ T yc[kSB * kSolveRhs];
  __shared__ T part[kSGroups * kSB * kSolveRhs];
  __shared__ int s_abort;
  const T* A = static_cast<const T*>(a.A);
  T* Y = static_cast<T*>(a.Y);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int cl = tid & (kSB - 1), g = tid / kSB;   // this thread's column of the block, row group
  const int n = a.n, nr = a.nr;
  if (tid == 0) s_abort = 0;
  __syncthreads();
  for (int i = blockIdx.x; i < a.nblk; i += gridDim.x) {
    const int b = a.nblk - 1 - i;
    const int c0 = b * kSB;
    T acc[kSolveRhs];
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) acc[q] = T(0);
    for (int bp = a.nblk - 1; bp > b; --bp) {
      const int r0 = bp * kSB;
      load_l_tile(A, a.lda, n, r0, c0, tile, tid);   // tile[cc][rr] = L(r0 + rr, c0 + cc)
      if (!wait_flag<T>(&a.flag[bp], a.status, s_abort)) return;
      for (int e = tid; e < kSB * nr; e += kSThreads) {
        const int rr = e % kSB, q = e / kSB;
        yc[rr * kSolveRhs + q] = (r0 + rr < n) ? ld_coh_t(&Y[(int64_t)(r0 + rr) + (int64_t)q * a.ldy]) : T(0);
      }
      __syncthreads();
#pragma unroll 4
      for (int jj = 0; jj < kSCols; ++jj) {
        const int rr = g * kSCols + jj;
        const T lv = tile[cl * kSLd + rr];
#pragma unroll
        for (int q = 0; q < kSolveRhs; ++q)
          if (q < nr) acc[q] = fma(lv, yc[rr * kSolveRhs + q], acc[q]);
      }
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) part[(g * kSB + cl) * kSolveRhs + q] = acc[q];
    load_l_tile(A, a.lda, n, c0, c0, tile, tid);
    __syncthreads();
    // diagonal block, backward: lane = column c of the block
    for (int q = wave; q < nr; q += kSThreads / kWave) {
      T x = T(0);
      if (c0 + lane < n) {
        x = ld_coh_t(&Y[(int64_t)(c0 + lane) + (int64_t)q * a.ldy]);
        T s = T(0);
#pragma unroll
        for (int gg = 0; gg < kSGroups; ++gg) s += part[(gg * kSB + lane) * kSolveRhs + q];
        x -= s;
      }
#pragma unroll 8
      for (int rr = kSB - 1; rr >= 0; --rr) {
        const T xr = __shfl(x, rr, kWave);
        if (lane < rr) x = fma(-tile[lane * kSLd + rr], xr, x);   // L(c0+rr, c0+lane)
      }
      if (c0 + lane < n) st_coh_t(&Y[(int64_t)(c0 + lane) + (int64_t)q * a.ldy], x);
    }
    wait_stores();
    __syncthreads();
    if (tid == 0) st_coh(&a.flag[b], 1);
  }
}

template <typename T, bool UPPER>
int solve_tri_max_blocks() {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const void* k;
  if constexpr (UPPER) k = (const void*)solve_upper_kernel<T>;
  else k = (const void*)solve_lower_kernel<T>;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kSThreads, 0) != hipSuccess) return 0;
  return per_cu * cus;
}

template <typename T, bool UPPER>
hipError_t launch_solve_tri(const SolveTriArgs& a, hipStream_t s) {
  const int cap = solve_tri_max_blocks<T, UPPER>();
  if (cap <= 0) return hipErrorInvalidValue;
  const int grid = a.nblk < cap ? a.nblk : cap;
  SolveTriArgs copy = a;
  void* args[] = {&copy};
  const void* k;
  if constexpr (UPPER) k = (const void*)solve_upper_kernel<T>;
  else k = (const void*)solve_lower_kernel<T>;
  return hipLaunchCooperativeKernel(k, dim3(grid), dim3(kSThreads), args, 0, s);
}

size_t solve_perm_lds_bytes(int n) { return 2 * (size_t)n * sizeof(int); }

template <typename T>
hipError_t launch_solve(int n, const T* A, int64_t lda, const int* ipiv, int nrhs, T* B, int64_t ldb,
                        const SolveWork& w, hipStream_t s) {
  hipError_t e;
  {
    const size_t lds = solve_perm_lds_bytes(n);
    const int use_lds = lds <= kSolvePermLds ? 1 : 0;
    if (use_lds) {
      static bool attr_set = false;
      if (!attr_set) {
        e = hipFuncSetAttribute((const void*)solve_perm_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)kSolvePermLds);
        if (e != hipSuccess) return e;
        attr_set = true;
      }
    }
    hipLaunchKernelGGL(solve_perm_kernel, dim3(1), dim3(256), use_lds ? lds : 0, s, n, ipiv, w.perm, w.scratch,
                       use_lds);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  T* alpha = static_cast<T*>(w.alpha);
  T* ralpha = static_cast<T*>(w.ralpha);
  T* Y = static_cast<T*>(w.Y);
  T* W = static_cast<T*>(w.W);
  hipLaunchKernelGGL(solve_alpha_kernel<T>, dim3((n + 255) / 256), dim3(256), 0, s, n, A, lda, alpha, ralpha);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int nblk = (n + kSB - 1) / kSB;
  for (int q0 = 0; q0 < nrhs; q0 += kSolveRhs) {
    const int nr = nrhs - q0 < kSolveRhs ? nrhs - q0 : kSolveRhs;
    T* Bq = B + (int64_t)q0 * ldb;
    hipLaunchKernelGGL(solve_gather_kernel<T>, dim3((n + 255) / 256, nr), dim3(256), 0, s, n, nr, w.perm, Bq, ldb,
                       Y, w.ldy);
    hipLaunchKernelGGL(solve_flags_kernel, dim3((2 * nblk + 255) / 256), dim3(256), 0, s, w.flags, 2 * nblk);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SolveTriArgs ta{};
    ta.A = A; ta.lda = lda; ta.n = n; ta.nblk = nblk; ta.Y = Y; ta.ldy = w.ldy; ta.nr = nr;
    ta.flag = w.flags; ta.status = w.status;
    if ((e = launch_solve_tri<T, false>(ta, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(solve_tridiag_kernel<T>, dim3(1), dim3(64), 0, s, n, nr, alpha, ralpha, Y, W, w.ldy);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    ta.Y = W;
    ta.flag = w.flags + nblk;
    if ((e = launch_solve_tri<T, true>(ta, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(solve_scatter_kernel<T>, dim3((n + 255) / 256, nr), dim3(256), 0, s, n, nr, w.perm, W, w.ldy,
                       Bq, ldb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

template hipError_t launch_solve<double>(int, const double*, int64_t, const int*, int, double*, int64_t,
                                         const SolveWork&, hipStream_t);
template hipError_t launch_solve<float>(int, const float*, int64_t, const int*, int, float*, int64_t,
                                        const SolveWork&, hipStream_t);

}  // namespace ltlt
