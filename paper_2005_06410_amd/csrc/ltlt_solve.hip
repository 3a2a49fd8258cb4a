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
//  * perm: every row follows its own moves through the exchanges, in
//    parallel (the steps bucketed by the position they target);
//  * the triangular solves are persistent cooperative kernels over 64-row
//    blocks, left-looking: the workgroup of block b streams the 64x64 tiles
//    of L to the left of its diagonal block (forward) or below it (backward)
//    through LDS, waiting for the stamped solution words of the block each
//    tile multiplies, then solves its diagonal block (one wave per
//    right-hand side, the unknown broadcast by readlane) and publishes its
//    own solution as stamped words.  A workgroup
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

#include <atomic>

namespace ltlt {

constexpr int kSB = 64;                // rows per block
constexpr int kSLd = kSB + 1;          // LDS stride of a tile column (bank spread)
constexpr int kSThreads = 256;         // 4 waves
constexpr int kSGroups = kSThreads / kSB;   // column (or row) groups of a tile
constexpr int kSCols = kSB / kSGroups;      // 16 columns per group

// ---- permutation ----------------------------------------------------------
// perm[i] = index of the row at position i after the exchanges (i, ipiv[i]),
// i = 0 .. n-1 in order, with ipiv[i] >= i, so position i is final once step
// i is done.  Computed per row, in parallel: a row at position x at step t
// is moved next either by the first step s in [t, x) with ipiv[s] = x (it
// then lands at s, final), or, failing that, by step x itself (to ipiv[x],
// or it stays at x when ipiv[x] = x).  The steps are bucketed by the position
// they target (count, scan, scatter), then every row walks its positions.
__global__ void perm_count_kernel(int n, const int* ipiv, int* cnt) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s < n) {
    const int x = ipiv[s];
    if (x > s && x < n) atomicAdd(&cnt[x], 1);
  }
}

// exclusive prefix sum of cnt[0..n) into off[0..n] (one workgroup)
__global__ void __launch_bounds__(1024) perm_scan_kernel(int n, const int* cnt, int* off) {
  __shared__ int part[1024];
  const int t = threadIdx.x;
  const int per = (n + 1023) / 1024;
  const int lo = min(n, t * per), hi = min(n, lo + per);
  int sum = 0;
  for (int i = lo; i < hi; ++i) sum += cnt[i];
  part[t] = sum;
  __syncthreads();
  for (int d = 1; d < 1024; d <<= 1) {            // inclusive scan of the per-thread sums
    const int v = t >= d ? part[t - d] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int run = part[t] - sum;
  for (int i = lo; i < hi; ++i) { off[i] = run; run += cnt[i]; }
  if (t == 1023) off[n] = part[1023];
}

__global__ void perm_scatter_kernel(int n, const int* ipiv, const int* off, int* fill, int* list) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s < n) {
    const int x = ipiv[s];
    if (x > s && x < n) list[off[x] + atomicAdd(&fill[x], 1)] = s;
  }
}

__global__ void perm_walk_kernel(int n, const int* ipiv, const int* off, const int* list, int* perm) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  int x = r, t = 0;
  for (;;) {
    int first = INT32_MAX;                         // first step s in [t, x) targeting x
    for (int e = off[x]; e < off[x + 1]; ++e) {
      const int s = list[e];
      if (s >= t && s < first) first = s;
    }
    if (first != INT32_MAX) { x = first; break; }
    const int p = ipiv[x];
    if (p <= x || p >= n) break;                   // no move (ipiv[x] = x)
    t = x + 1;
    x = p;
  }
  perm[x] = r;
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

__global__ void zero_ints_kernel(int* v, int count) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) v[i] = 0;
}

// ---- skew tridiagonal recurrences -----------------------------------------
// Wave 0 runs the odd unknowns forward, wave 1 the even unknowns backward;
// lane q < nr takes right-hand side q.  Each chain reads the inputs of the
// other chain's parity, so the result goes to a separate buffer W.  The
// inputs of kTriChunk steps at a time are staged in LDS by the whole wave, so
// that the chain itself waits only on its own arithmetic.
constexpr int kTriChunk = 512;
template <typename T>
__global__ void __launch_bounds__(128) solve_tridiag_kernel(int n, int nr, const T* alpha, const T* ralpha,
                                                            const T* Y, T* W, int64_t ldy) {
  __shared__ T sbuf[2][kTriChunk * (2 + kSolveRhs)];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  T* sa = sbuf[wave];                              // multiplier alpha of each step
  T* sr = sa + kTriChunk;                          // reciprocal alpha of each step
  T* sy = sr + kTriChunk;                          // [step][rhs] right-hand side entry
  const int half = n / 2;                          // unknowns per chain
  if (wave == 0) {
    // W[1] = -R[0] / alpha_0;  step s >= 1, i = 2s:  W[i+1] = (alpha_{i-1} W[i-1] - R[i]) / alpha_i
    T wprev = T(0);
    if (lane < nr) {
      wprev = -Y[(int64_t)lane * ldy] * ralpha[0];
      W[1 + (int64_t)lane * ldy] = wprev;
    }
    for (int s0 = 1; s0 < half; s0 += kTriChunk) {
      const int cnt = min(kTriChunk, half - s0);
      for (int e = lane; e < cnt; e += kWave) {
        const int i = 2 * (s0 + e);
        sa[e] = alpha[i - 1];
        sr[e] = ralpha[i];
        for (int q = 0; q < nr; ++q) sy[e * kSolveRhs + q] = Y[(int64_t)i + (int64_t)q * ldy];
      }
      wave_lds_sync();
      if (lane < nr) {
        for (int e = 0; e < cnt; ++e) {
          const T w = (sa[e] * wprev - sy[e * kSolveRhs + lane]) * sr[e];
          W[(int64_t)(2 * (s0 + e) + 1) + (int64_t)lane * ldy] = w;
          wprev = w;
        }
      }
      wave_lds_sync();
    }
  } else {
    // W[n-2] = R[n-1] / alpha_{n-2};  step s >= 1, i = n-1-2s:  W[i-1] = (R[i] + alpha_i W[i+1]) / alpha_{i-1}
    T wnext = T(0);
    if (lane < nr) {
      wnext = Y[(int64_t)(n - 1) + (int64_t)lane * ldy] * ralpha[n - 2];
      W[(int64_t)(n - 2) + (int64_t)lane * ldy] = wnext;
    }
    for (int s0 = 1; s0 < half; s0 += kTriChunk) {
      const int cnt = min(kTriChunk, half - s0);
      for (int e = lane; e < cnt; e += kWave) {
        const int i = n - 1 - 2 * (s0 + e);
        sa[e] = alpha[i];
        sr[e] = ralpha[i - 1];
        for (int q = 0; q < nr; ++q) sy[e * kSolveRhs + q] = Y[(int64_t)i + (int64_t)q * ldy];
      }
      wave_lds_sync();
      if (lane < nr) {
        for (int e = 0; e < cnt; ++e) {
          const T w = (sy[e * kSolveRhs + lane] + sa[e] * wnext) * sr[e];
          W[(int64_t)(n - 2 - 2 * (s0 + e)) + (int64_t)lane * ldy] = w;
          wnext = w;
        }
      }
      wave_lds_sync();
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
  uint64_t* box;      // [nblk][kSolveRhs][kSB][2] stamped solution words
  unsigned stamp;     // stamp of this launch (never 0)
  int* status;
};

// A solution value crosses workgroups as two 64-bit words, each holding one
// 32-bit half of the value above the 32-bit stamp of the launch: naturally
// aligned 64-bit stores are single-copy atomic, so a reader that sees the
// stamp in both words has the value, without a separate flag (and the writer
// does not wait for its stores before signalling).  Words of an earlier
// launch carry an older stamp and never validate.
template <typename T>
__device__ __forceinline__ void box_put(uint64_t* w, T x, unsigned stamp) {
  unsigned hi, lo;
  if constexpr (sizeof(T) == 8) {
    hi = (unsigned)__double2hiint(x);
    lo = (unsigned)__double2loint(x);
  } else {
    hi = __float_as_uint(x);
    lo = 0u;
  }
  st_coh64(&w[0], ((uint64_t)hi << 32) | stamp);
  st_coh64(&w[1], ((uint64_t)lo << 32) | stamp);
}
template <typename T>
__device__ __forceinline__ bool box_get(const uint64_t* w, unsigned stamp, T& x) {
  const uint64_t w0 = ld_coh64(&w[0]), w1 = ld_coh64(&w[1]);
  if ((unsigned)w0 != stamp || (unsigned)w1 != stamp) return false;
  if constexpr (sizeof(T) == 8) x = __hiloint2double((int)(w0 >> 32), (int)(w1 >> 32));
  else x = __uint_as_float((unsigned)(w0 >> 32));
  return true;
}

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

// Poll the solution of block sb until every (row, right-hand side) entry
// carries this launch's stamp; the values land in yc[row][rhs].  Bounded.
template <typename T>
__device__ __forceinline__ bool wait_box(const SolveTriArgs& a, int sb, T* yc, int tid) {
  const uint64_t* bx = a.box + (size_t)sb * kSolveRhs * kSB * 2;
  const uint64_t t0 = wall_ticks();
  for (;;) {
    bool ok = true;
    for (int e = tid; e < kSB * a.nr; e += kSThreads) {
      const int rr = e % kSB, q = e / kSB;
      T v;
      if (box_get(&bx[((size_t)q * kSB + rr) * 2], a.stamp, v)) yc[rr * kSolveRhs + q] = v;
      else ok = false;
    }
    if (__syncthreads_and(ok)) return true;
    const bool late = tid == 0 && (ld_coh(a.status) != 0 || wall_ticks() - t0 > kWaitLimitTicks);
    if (__syncthreads_or(late)) {
      if (tid == 0) atomicOr(a.status, 1);
      return false;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Broadcast lane l's value (l wave-uniform) through scalar registers.
template <typename T>
__device__ __forceinline__ T lane_bcast(T x, int l) {
  if constexpr (sizeof(T) == 8) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(x), l);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(x), l);
    return __hiloint2double(hi, lo);
  } else {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
  }
}

// Forward (UPPER = false): z_b = L_bb^{-1} (y_b - sum_{c<b} L_bc z_c).
// Backward (UPPER = true), blocks from the last one down:
//   u_b = L_bb^{-T} (w_b - sum_{b'>b} L_{b'b}^T u_{b'}).
// The off-diagonal tiles of a block are streamed through LDS with the next
// tile's values already in registers (they do not depend on any flag); the
// diagonal tile has its own buffer, loaded at the start of the block.
template <typename T, bool UPPER>
__global__ void __launch_bounds__(kSThreads, 1) solve_tri_kernel(SolveTriArgs a) {
  __shared__ T tile[kSB * kSLd];
  __shared__ T dtile[kSB * kSLd];
  __shared__ T yc[kSB * kSolveRhs];                // solution of the block a tile multiplies
  __shared__ T part[kSGroups * kSB * kSolveRhs];   // partial sums of the four groups
  const T* A = static_cast<const T*>(a.A);
  T* Y = static_cast<T*>(a.Y);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int r = tid & (kSB - 1), g = tid / kSB;
  const int n = a.n, nr = a.nr, nblk = a.nblk;
  const int64_t lda = a.lda, ldy = a.ldy;
  for (int i = blockIdx.x; i < nblk; i += gridDim.x) {
    const int b = UPPER ? nblk - 1 - i : i;
    const int d0 = b * kSB;
    const int ntile = UPPER ? nblk - 1 - b : b;
    // tile t multiplies the solution of block src(t): forward t, backward nblk-1-t
    auto src = [&](int t) { return UPPER ? nblk - 1 - t : t; };
    T regs[kSCols];
    auto fetch = [&](int t) {
      const int s0 = src(t) * kSB;
      const int rr0 = UPPER ? s0 : d0, cc0 = UPPER ? d0 : s0;
#pragma unroll
      for (int jj = 0; jj < kSCols; ++jj) regs[jj] = l_entry(A, lda, n, rr0 + r, cc0 + g + kSGroups * jj);
    };
    load_l_tile(A, lda, n, d0, d0, dtile, tid);
    // this wave's right-hand side entries of the block (rhs wave, wave + 4),
    // read now: they are needed only at the diagonal step, which is on the
    // chain from block to block
    constexpr int kQW = kSolveRhs / (kSThreads / kWave);
    T ypre[kQW];
#pragma unroll
    for (int k = 0; k < kQW; ++k) {
      const int q = wave + (kSThreads / kWave) * k;
      ypre[k] = (q < nr && d0 + lane < n) ? Y[(int64_t)(d0 + lane) + (int64_t)q * ldy] : T(0);
    }
    T acc[kSolveRhs];
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) acc[q] = T(0);
    if (ntile > 0) fetch(0);
    for (int t = 0; t < ntile; ++t) {
#pragma unroll
      for (int jj = 0; jj < kSCols; ++jj) tile[(g + kSGroups * jj) * kSLd + r] = regs[jj];
      if (t + 1 < ntile) fetch(t + 1);
      if (!wait_box<T>(a, src(t), yc, tid)) return;
      // forward: thread (row r, column group g); backward: (column r, row group g)
#pragma unroll 4
      for (int jj = 0; jj < kSCols; ++jj) {
        const int k = g * kSCols + jj;
        const T lv = UPPER ? tile[r * kSLd + k] : tile[k * kSLd + r];
#pragma unroll
        for (int q = 0; q < kSolveRhs; ++q)
          if (q < nr) acc[q] = fma(lv, yc[k * kSolveRhs + q], acc[q]);
      }
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) part[(g * kSB + r) * kSolveRhs + q] = acc[q];
    __syncthreads();
    // diagonal block: wave w solves right-hand sides w, w+4; lane = row
    // (forward) or column (backward) of the block.  The lane's entries of
    // the diagonal tile go to registers first, so that the 64 dependent steps
    // wait only on the scalar broadcast and the FMA.
#pragma unroll
    for (int k = 0; k < kQW; ++k) {
      const int q = wave + (kSThreads / kWave) * k;
      if (q >= nr) break;
      T dl[kSB];
#pragma unroll
      for (int cc = 0; cc < kSB; ++cc) dl[cc] = UPPER ? dtile[lane * kSLd + cc] : dtile[cc * kSLd + lane];
      T x = T(0);
      if (d0 + lane < n) {
        T sum = T(0);
#pragma unroll
        for (int gg = 0; gg < kSGroups; ++gg) sum += part[(gg * kSB + lane) * kSolveRhs + q];
        x = ypre[k] - sum;
      }
      if constexpr (!UPPER) {
#pragma unroll
        for (int cc = 0; cc < kSB; ++cc) {
          const T xc = lane_bcast(x, cc);
          if (lane > cc) x = fma(-dl[cc], xc, x);                    // L(d0+lane, d0+cc)
        }
      } else {
#pragma unroll
        for (int rr = kSB - 1; rr >= 0; --rr) {
          const T xr = lane_bcast(x, rr);
          if (lane < rr) x = fma(-dl[rr], xr, x);                    // L(d0+rr, d0+lane)
        }
      }
      if (d0 + lane < n) Y[(int64_t)(d0 + lane) + (int64_t)q * ldy] = x;
      box_put(&a.box[(((size_t)b * kSolveRhs + q) * kSB + lane) * 2], d0 + lane < n ? x : T(0), a.stamp);
    }
    __syncthreads();                               // part and dtile are reused by the next block
  }
}

template <typename T, bool UPPER>
int solve_tri_max_blocks() {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const void* k = (const void*)solve_tri_kernel<T, UPPER>;
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
  const void* k = (const void*)solve_tri_kernel<T, UPPER>;
  return hipLaunchCooperativeKernel(k, dim3(grid), dim3(kSThreads), args, 0, s);
}

// Stamps of the mailbox words: a process-wide counter that skips 0 (zeroed
// memory never validates).
unsigned next_stamp() {
  static std::atomic<unsigned> counter{0};
  unsigned v;
  do { v = counter.fetch_add(1) + 1; } while (v == 0);
  return v;
}

template <typename T>
hipError_t launch_solve(int n, const T* A, int64_t lda, const int* ipiv, int nrhs, T* B, int64_t ldb,
                        const SolveWork& w, hipStream_t s) {
  hipError_t e;
  {
    const int gb = (n + 255) / 256;
    hipLaunchKernelGGL(zero_ints_kernel, dim3((2 * n + 255) / 256), dim3(256), 0, s, w.cnt, 2 * n);
    hipLaunchKernelGGL(perm_count_kernel, dim3(gb), dim3(256), 0, s, n, ipiv, w.cnt);
    hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(1024), 0, s, n, w.cnt, w.off);
    hipLaunchKernelGGL(perm_scatter_kernel, dim3(gb), dim3(256), 0, s, n, ipiv, w.off, w.cnt + n, w.list);
    hipLaunchKernelGGL(perm_walk_kernel, dim3(gb), dim3(256), 0, s, n, ipiv, w.off, w.list, w.perm);
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
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SolveTriArgs ta{};
    ta.A = A; ta.lda = lda; ta.n = n; ta.nblk = nblk; ta.Y = Y; ta.ldy = w.ldy; ta.nr = nr;
    ta.box = w.box; ta.status = w.status;
    ta.stamp = next_stamp();
    if ((e = launch_solve_tri<T, false>(ta, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(solve_tridiag_kernel<T>, dim3(1), dim3(128), 0, s, n, nr, alpha, ralpha, Y, W, w.ldy);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    ta.Y = W;
    ta.stamp = next_stamp();
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
