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
//  * the inverses of the 64x64 unit lower diagonal blocks of L, and their
//    products with the two nearest off-diagonal tiles, are formed first,
//    all blocks at once (off the dependency chain);
//  * the triangular solves are persistent cooperative kernels over 64-row
//    blocks, left-looking: the workgroup of block b streams the 64x64 tiles
//    of L to the left of its diagonal block (forward) or below it (backward)
//    through LDS, waiting for the stamped solution words of the block each
//    tile multiplies, except the two nearest ones; then each wave takes one
//    right-hand side alone: the residual times the inverse of the diagonal
//    block (its transpose, backward), minus the precomputed products with
//    the two nearest blocks' solutions, waiting for each only then (one
//    64-term product on the chain from block to block instead of a tile
//    and a 64-step substitution), and publishes its solution as stamped
//    words.  A workgroup
//    takes its blocks in dependency order, so the earliest unfinished block
//    always has its inputs and the grid cannot deadlock; every wait is
//    bounded.  Each solve reads the lower triangle of L once: HBM-bound for
//    few right-hand sides;
//  * each recurrence of T (w_s = a_s w_{s-1} + b_s along one parity) runs
//    as a chunked scan: every lane of a wave composes the affine maps of its
//    chunk of steps, the wave scans the 64 compositions, and every lane then
//    re-runs its chunk from its exact starting value with the recurrence as
//    written; one wave per (right-hand side, chain), the reciprocals of alpha
//    formed in parallel beforehand.
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
// One wave per (right-hand side q, chain): waves 2q run the odd unknowns
// forward, waves 2q+1 the even unknowns backward.  Both chains are
// w_s = a_s w_{s-1} + b_s over s = 1 .. n/2 - 1 after a first value w_0:
//   odd:  i = 2s,        W[i+1] = (alpha_{i-1} W[i-1] - R[i]) / alpha_i,  w_0 = W[1] = -R[0] / alpha_0
//   even: i = n-1-2s,    W[i-1] = (R[i] + alpha_i W[i+1]) / alpha_{i-1},  w_0 = W[n-2] = R[n-1] / alpha_{n-2}
// Lane j takes the steps of chunk j (C consecutive steps): it composes their
// maps (A, B) with w_end = A w_start + B, the wave forms the exclusive prefix
// compositions by a shuffle scan, and each lane re-runs its chunk from
// w_start = A_prefix w_0 + B_prefix, writing every unknown with the
// recurrence as written above.  Each chain reads the other parity's inputs,
// so the result goes to a separate buffer W.
template <typename T>
__device__ __forceinline__ void tri_step_coeffs(bool odd, int n, int s, const T* alpha, const T* ralpha, const T* R,
                                                T& ca, T& cb, T& cr, int& out) {
  if (odd) {                                       // i = 2s: W[i+1] = (alpha_{i-1} w - R[i]) * ralpha[i]
    const int i = 2 * s;
    ca = alpha[i - 1]; cb = R[i]; cr = ralpha[i]; out = i + 1;
  } else {                                         // i = n-1-2s: W[i-1] = (R[i] + alpha_i w) * ralpha[i-1]
    const int i = n - 1 - 2 * s;
    ca = alpha[i]; cb = R[i]; cr = ralpha[i - 1]; out = i - 1;
  }
}

template <typename T>
__global__ void __launch_bounds__(1024) solve_tridiag_kernel(int n, int nr, const T* alpha, const T* ralpha,
                                                             const T* Y, T* W, int64_t ldy) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int q = wave >> 1;
  if (q >= nr) return;                             // whole wave
  const bool odd = (wave & 1) == 0;
  const T* R = Y + (int64_t)q * ldy;
  T* Wq = W + (int64_t)q * ldy;
  const int half = n / 2;                          // unknowns per chain
  const T w0 = odd ? -R[0] * ralpha[0] : R[n - 1] * ralpha[n - 2];
  if (lane == 0) Wq[odd ? 1 : n - 2] = w0;
  const int steps = half - 1;                      // s = 1 .. half-1
  const int C = (steps + kWave - 1) / kWave;       // steps per lane
  const int s_lo = 1 + lane * C, s_hi = min(half, s_lo + C);
  // composition of this chunk's maps: w -> a w + b, a = ca cr (odd) / ca cr,
  // b = -cb cr (odd) / cb cr (even)
  T Ac = T(1), Bc = T(0);
#pragma unroll 8
  for (int s = s_lo; s < s_hi; ++s) {
    T ca, cb, cr;
    int out;
    tri_step_coeffs(odd, n, s, alpha, ralpha, R, ca, cb, cr, out);
    const T a = ca * cr, b = odd ? -cb * cr : cb * cr;
    Ac = a * Ac;
    Bc = fma(a, Bc, b);
  }
  // inclusive scan of the compositions in lane order (later maps applied
  // after earlier ones: (A2, B2) o (A1, B1) = (A2 A1, A2 B1 + B2))
  T Ai = Ac, Bi = Bc;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const T Ap = __shfl_up(Ai, off, kWave), Bp = __shfl_up(Bi, off, kWave);
    if (lane >= off) {
      Bi = fma(Ai, Bp, Bi);
      Ai = Ai * Ap;
    }
  }
  // exclusive prefix: the inclusive one of the previous lane
  T Ae = __shfl_up(Ai, 1, kWave), Be = __shfl_up(Bi, 1, kWave);
  if (lane == 0) { Ae = T(1); Be = T(0); }
  T w = fma(Ae, w0, Be);                           // value entering this chunk
#pragma unroll 8
  for (int s = s_lo; s < s_hi; ++s) {
    T ca, cb, cr;
    int out;
    tri_step_coeffs(odd, n, s, alpha, ralpha, R, ca, cb, cr, out);
    w = odd ? (ca * w - cb) * cr : (cb + ca * w) * cr;
    Wq[out] = w;
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
  const void* Dinv;   // inverses of the diagonal blocks of L: [nblk][64 * 64], column-major
  const void* Mf;     // D_b^{-1} L_{b,b-d}: [kLook][nblk][64 * 64], column-major
  const void* Mb;     // D_b^{-T} L_{b+d,b}^T: [kLook][nblk][64 * 64], column-major
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

// Per 64-row block b: the inverse of its unit lower diagonal block D_b of L
// and the matrices that carry the last kLook dependencies of each
// substitution, for d = 1 .. kLook,
//   Mf_{b,d} = D_b^{-1} L_{b,b-d}        (forward, b >= d),
//   Mb_{b,d} = D_b^{-T} L_{b+d,b}^T      (backward, b + d < nblk),
// so that z_b = D_b^{-1} r_b - sum_d Mf_{b,d} z_{b-d} and
// u_b = D_b^{-T} r_b - sum_d Mb_{b,d} u_{b+d}, where r_b is the block's
// right-hand side less the contributions of every farther block.  All are
// stored column-major per block, X[b*64*64 + k*64 + r] = X(r, k); rows and
// columns past n give the identity (D_b^{-1}) or zeros (M), which the solves
// never use.
constexpr int kLook = 1;                          // dependencies carried by the waves

// D_b^{-1}, one wave per block: lane c forms column c by forward
// substitution, X(c,c) = 1, X(r,c) = -sum_{c<=k<r} D(r,k) X(k,c), D read from
// LDS by broadcast.
template <typename T>
__global__ void __launch_bounds__(kWave) solve_dinv_kernel(const T* A, int64_t lda, int n, T* Dinv) {
  __shared__ T d[kSB * kSLd];                      // D(r, c), then D^{-1}(r, c), at d[c * kSLd + r]
  const int b = blockIdx.x, lane = threadIdx.x;
  const int d0 = b * kSB;
#pragma unroll 4
  for (int cc = 0; cc < kSB; ++cc) d[cc * kSLd + lane] = l_entry(A, lda, n, d0 + lane, d0 + cc);
  wave_lds_sync();
  T x[kSB];
#pragma unroll
  for (int r = 0; r < kSB; ++r) {
    T acc = T(0);
#pragma unroll
    for (int k = 0; k < r; ++k) acc = fma(d[k * kSLd + r], x[k], acc);
    x[r] = r < lane ? T(0) : (r == lane ? T(1) : -acc);
  }
  wave_lds_sync();                                 // every read of D is done
#pragma unroll
  for (int r = 0; r < kSB; ++r) d[lane * kSLd + r] = x[r];
  wave_lds_sync();
  T* out = Dinv + (size_t)b * kSB * kSB;
#pragma unroll 4
  for (int cc = 0; cc < kSB; ++cc) out[cc * kSB + lane] = d[cc * kSLd + lane];
}

// Mf_{b,d} and Mb_{b,d}, 2 kLook waves per block: D_b^{-1} into LDS; wave
// 2(d-1) + e (e = 0 forward, 1 backward), lane k, loads column k of L_{b,b-d}
// or row k of L_{b+d,b} and forms column k of its matrix with D_b^{-1} read
// by broadcast.
template <typename T>
__global__ void __launch_bounds__(2 * kLook * kWave) solve_mmat_kernel(const T* A, int64_t lda, int n, int nblk,
                                                                       const T* Dinv, T* Mf, T* Mb) {
  __shared__ T d[kSB * kSLd];                      // D^{-1}(r, c) at d[c * kSLd + r]
  const int b = blockIdx.x, tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int d0 = b * kSB;
  const size_t blk = (size_t)b * kSB * kSB;
  for (int e = tid; e < kSB * kSB; e += blockDim.x) d[(e / kSB) * kSLd + e % kSB] = Dinv[blk + e];
  const int dist = 1 + wave / 2;
  const bool fwd = (wave & 1) == 0;
  const bool has = fwd ? b >= dist : b + dist < nblk;
  T lv[kSB];
#pragma unroll 8
  for (int j = 0; j < kSB; ++j)
    lv[j] = !has ? T(0)
                 : (fwd ? l_entry(A, lda, n, d0 + j, d0 - dist * kSB + lane)
                        : l_entry(A, lda, n, d0 + dist * kSB + lane, d0 + j));
  __syncthreads();
  if (!has) return;                                // no barrier follows
  T* out = (fwd ? Mf : Mb) + (size_t)(dist - 1) * nblk * kSB * kSB + blk + (size_t)lane * kSB;
  // forward:  Mf(r, k) = sum_j D^{-1}(r, j) L_{b,b-d}(j, k)
  // backward: Mb(r, k) = sum_j D^{-1}(j, r) L_{b+d,b}(k, j)
  const int sj = fwd ? kSLd : 1, sr = fwd ? 1 : kSLd;   // LDS strides of j and r
  for (int r = 0; r < kSB; ++r) {
    T acc = T(0);
#pragma unroll
    for (int j = 0; j < kSB; ++j) acc = fma(d[j * sj + r * sr], lv[j], acc);
    out[r] = acc;
  }
}

// Workgroup barrier for LDS only: it waits for this wave's LDS operations
// but not for its outstanding global loads (__syncthreads does, and with
// them every tile and solution prefetch in flight).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Workgroup-wide AND of v over an LDS-only barrier: each wave's vote goes to
// one of two flag sets, alternating per call (a set is rewritten two votes
// later, after every wave has passed the barrier of the vote in between).
struct Vote {
  int* flags;        // LDS [2][waves]
  int k;
  __device__ bool all(bool v, int wave, int lane) {
    int* f = flags + (k & 1) * (kSThreads / kWave);
    ++k;
    const int w = __ballot(!v) == 0;
    if (lane == 0) f[wave] = w;
    lds_barrier();
    bool r = true;
#pragma unroll
    for (int i = 0; i < kSThreads / kWave; ++i) r = r && f[i] != 0;
    return r;
  }
};

// Poll the solution of block sb until every (row, right-hand side) entry
// carries this launch's stamp; the values land in yc[row][rhs].  Bounded;
// the whole workgroup returns false together when the wait gives up.  The
// status word is read in the same round trip as the solution words, so an
// unsuccessful poll costs one round trip, not two.
template <typename T>
__device__ __forceinline__ bool wait_box(const SolveTriArgs& a, int sb, T* yc, int tid, Vote& vote) {
  const int wave = tid / kWave, lane = tid & (kWave - 1);
  const uint64_t* bx = a.box + (size_t)sb * kSolveRhs * kSB * 2;
  const uint64_t t0 = wall_ticks();
  for (;;) {
    bool ok = true;
    const int st = tid == 0 ? ld_coh(a.status) : 0;
    for (int e = tid; e < kSB * a.nr; e += kSThreads) {
      const int rr = e % kSB, q = e / kSB;
      T v;
      if (box_get(&bx[((size_t)q * kSB + rr) * 2], a.stamp, v)) yc[rr * kSolveRhs + q] = v;
      else ok = false;
    }
    if (vote.all(ok, wave, lane)) return true;
    const bool late = tid == 0 && (st != 0 || wall_ticks() - t0 > kWaitLimitTicks);
    if (!vote.all(!late, wave, lane)) {
      if (tid == 0) raise_wait_status(a.status);
      return false;
    }
  }
}

// One wave polls the 64 solution entries of block sb for right-hand side q
// (lane = row), reading the status word in the same round trip.  Bounded:
// when the wait gives up (or an earlier wait already has) the status flag is
// set and false is returned; the wave carries on with an unspecified value,
// so that no wave leaves its workgroup's barriers.
template <typename T>
__device__ __forceinline__ bool wait_words(const SolveTriArgs& a, int sb, int q, int lane, T& v) {
  const uint64_t* w = a.box + (((size_t)sb * kSolveRhs + q) * kSB + lane) * 2;
  const uint64_t t0 = wall_ticks();
  for (;;) {
    const int st = ld_coh(a.status);
    const bool ok = box_get(w, a.stamp, v);
    if (__ballot(!ok) == 0) return true;
    const int late = __builtin_amdgcn_readfirstlane((st != 0 || wall_ticks() - t0 > kWaitLimitTicks) ? 1 : 0);
    if (late) {
      if (lane == 0) raise_wait_status(a.status);
      return false;
    }
  }
}

// Forward (UPPER = false): z_b = D_b^{-1} r_b - sum_{d<=kLook} Mf_{b,d} z_{b-d},
//   r_b = y_b - sum_{c<b-kLook} L_bc z_c.
// Backward (UPPER = true), blocks from the last one down:
//   u_b = D_b^{-T} r_b - sum_{d<=kLook} Mb_{b,d} u_{b+d},
//   r_b = w_b - sum_{b'>b+kLook} L_{b'b}^T u_{b'}.
// The workgroup multiplies the farther off-diagonal tiles of r_b straight
// from registers (two tiles in flight, the next block's solution words
// requested during the current tile, so that a tile whose inputs are long
// published costs no round trip); then every wave takes its
// right-hand sides alone: c = D_b^{-1} r_b (resp. D_b^{-T} r_b) with its row
// of the inverse in registers and r broadcast from LDS, then, nearest block
// last, waits for each of the kLook neighbouring blocks' solutions and
// subtracts M times it.  Only the last of those products is on the chain
// from block to block; the workgroup's own tiles have kLook blocks of slack.
template <typename T, bool UPPER>
__global__ void __launch_bounds__(kSThreads, 1) solve_tri_kernel(SolveTriArgs a) {
  __shared__ T dtile[kSB * kSLd];                  // D_b^{-1}, column-major
  __shared__ T mtile[kLook][kSB * kSLd];           // Mf_{b,d} (forward) or Mb_{b,d} (backward), column-major
  __shared__ T yc[kSB * kSolveRhs];                // solution of the block a tile multiplies
  __shared__ T part[kSGroups * kSB * kSolveRhs];   // partial sums of the four groups
  __shared__ T xs[kSThreads / kWave][kSB];         // vector broadcast to the lanes of a wave
  __shared__ int vflags[2 * (kSThreads / kWave)];
  Vote vote{vflags, 0};
  const T* A = static_cast<const T*>(a.A);
  T* Y = static_cast<T*>(a.Y);
  const T* Dinv = static_cast<const T*>(a.Dinv);
  const T* Mx = static_cast<const T*>(UPPER ? a.Mb : a.Mf);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int r = tid & (kSB - 1), g = tid / kSB;
  const int n = a.n, nr = a.nr, nblk = a.nblk;
  const int64_t lda = a.lda, ldy = a.ldy;
  for (int i = blockIdx.x; i < nblk; i += gridDim.x) {
    const int b = UPPER ? nblk - 1 - i : i;
    const int d0 = b * kSB;
    const int ntile = UPPER ? nblk - 1 - b : b;   // tiles of r_b and the chain's tile
    const int nfull = ntile > kLook ? ntile - kLook : 0;   // tiles the workgroup multiplies itself
    const int nlook = ntile - nfull;               // tiles the waves carry (nearest last)
    // tile t multiplies the solution of block src(t): forward t, backward nblk-1-t
    auto src = [&](int t) { return UPPER ? nblk - 1 - t : t; };
    // thread (r, g) holds, jj < 16, forward L(d0 + r, s0 + g + 4 jj) (row r of
    // the tile, coalesced), backward L(s0 + g + 4 jj, d0 + r) (column r of the
    // tile: one row per instruction, each thread's 16 rows from a few lines);
    // either way the thread's sum is over its own registers
    auto fetch = [&](int t, T(&regs)[kSCols]) {
      const int s0 = src(t) * kSB;
#pragma unroll
      for (int jj = 0; jj < kSCols; ++jj)
        regs[jj] = UPPER ? l_entry(A, lda, n, s0 + g + kSGroups * jj, d0 + r)
                         : l_entry(A, lda, n, d0 + r, s0 + g + kSGroups * jj);
    };
    // the solution words of a tile's block, loaded one tile ahead: entry
    // e = q * 64 + row of the block's words, kYE entries per thread
    constexpr int kYE = kSB * kSolveRhs / kSThreads;
    uint64_t yw[kYE][2];
    auto ypf = [&](int t) {
      const uint64_t* bx = a.box + (size_t)src(t) * kSolveRhs * kSB * 2;
#pragma unroll
      for (int e = 0; e < kYE; ++e) {
        const int idx = tid + e * kSThreads;
        if (idx < kSB * nr) {
          yw[e][0] = ld_coh64(&bx[(size_t)idx * 2]);
          yw[e][1] = ld_coh64(&bx[(size_t)idx * 2 + 1]);
        }
      }
    };
    // the prefetched words into yc when every one carries this launch's
    // stamp (true for the whole workgroup), else false
    auto ytake = [&]() {
      bool ok = true;
#pragma unroll
      for (int e = 0; e < kYE; ++e) {
        const int idx = tid + e * kSThreads;
        if (idx < kSB * nr) {
          const uint64_t w0 = yw[e][0], w1 = yw[e][1];
          if ((unsigned)w0 != a.stamp || (unsigned)w1 != a.stamp) {
            ok = false;
          } else {
            T v;
            if constexpr (sizeof(T) == 8) v = __hiloint2double((int)(w0 >> 32), (int)(w1 >> 32));
            else v = __uint_as_float((unsigned)(w0 >> 32));
            yc[(idx % kSB) * kSolveRhs + idx / kSB] = v;
          }
        }
      }
      return vote.all(ok, wave, lane);
    };
    {
      // every load issued before the first LDS store, so that the block's
      // start costs one memory round trip
      const T* Db = Dinv + (size_t)b * kSB * kSB;
      const size_t mat = (size_t)nblk * kSB * kSB;
      T dv[kSCols], mv[kLook][kSCols];
#pragma unroll
      for (int jj = 0; jj < kSCols; ++jj) {
        const int cc = g + kSGroups * jj;
        dv[jj] = Db[cc * kSB + r];
#pragma unroll
        for (int dd = 0; dd < kLook; ++dd)
          mv[dd][jj] = dd < nlook ? Mx[(size_t)dd * mat + (size_t)b * kSB * kSB + cc * kSB + r] : T(0);
      }
#pragma unroll
      for (int jj = 0; jj < kSCols; ++jj) {
        const int cc = g + kSGroups * jj;
        dtile[cc * kSLd + r] = dv[jj];
#pragma unroll
        for (int dd = 0; dd < kLook; ++dd) mtile[dd][cc * kSLd + r] = mv[dd][jj];
      }
    }
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
    // tile t: its block's solution in yc (prefetched words, else a poll),
    // the next block's words requested, then the product; two tiles are in
    // flight in registers (buffers ra and rb alternate)
    auto step = [&](int t, T(&regs)[kSCols]) {
      if (!ytake() && !wait_box<T>(a, src(t), yc, tid, vote)) return false;
      if (t + 1 < nfull) ypf(t + 1);
      // thread (r, g): output entry r, terms g + 4 jj, straight from registers;
      // every right-hand side slot, branch-free (the sums of slots past nr are
      // never read), so that the tile loads are not all waited for per term
#pragma unroll
      for (int jj = 0; jj < kSCols; ++jj) {
        const int k = g + kSGroups * jj;
#pragma unroll
        for (int q = 0; q < kSolveRhs; ++q) acc[q] = fma(regs[jj], yc[k * kSolveRhs + q], acc[q]);
      }
      lds_barrier();                               // yc is rewritten by the next tile
      return true;
    };
    T ra[kSCols], rb[kSCols];
    if (nfull > 0) { fetch(0, ra); ypf(0); }
    if (nfull > 1) fetch(1, rb);
    for (int t = 0; t < nfull; t += 2) {
      if (!step(t, ra)) return;
      if (t + 2 < nfull) fetch(t + 2, ra);
      if (t + 1 < nfull) {
        if (!step(t + 1, rb)) return;
        if (t + 3 < nfull) fetch(t + 3, rb);
      }
    }
#pragma unroll
    for (int q = 0; q < kSolveRhs; ++q) part[(g * kSB + r) * kSolveRhs + q] = acc[q];
    lds_barrier();
    // wave w takes right-hand sides w, w+4; lane = row (forward) or column
    // (backward) of the block
#pragma unroll
    for (int k = 0; k < kQW; ++k) {
      const int q = wave + (kSThreads / kWave) * k;
      if (q >= nr) break;
      T x = T(0);
      if (d0 + lane < n) {
        T sum = T(0);
#pragma unroll
        for (int gg = 0; gg < kSGroups; ++gg) sum += part[(gg * kSB + lane) * kSolveRhs + q];
        x = ypre[k] - sum;
      }
      xs[wave][lane] = x;
      wave_lds_sync();
      {
        T dl[kSB];
#pragma unroll
        for (int cc = 0; cc < kSB; ++cc) dl[cc] = UPPER ? dtile[lane * kSLd + cc] : dtile[cc * kSLd + lane];
        T s4[4] = {T(0), T(0), T(0), T(0)};
#pragma unroll
        for (int cc = 0; cc < kSB; ++cc) s4[cc & 3] = fma(dl[cc], xs[wave][cc], s4[cc & 3]);
        x = (s4[0] + s4[1]) + (s4[2] + s4[3]);
      }
      wave_lds_sync();                             // xs is rewritten below
      // distance d = nlook .. 1: tile ntile-d multiplies block src(ntile-d)
      for (int dd = nlook - 1; dd >= 0; --dd) {
        T ml[kSB];
#pragma unroll
        for (int kk = 0; kk < kSB; ++kk) ml[kk] = mtile[dd][kk * kSLd + lane];
        T yp;
        wait_words<T>(a, src(ntile - 1 - dd), q, lane, yp);
        xs[wave][lane] = yp;
        wave_lds_sync();
        T s4[4] = {T(0), T(0), T(0), T(0)};
#pragma unroll
        for (int kk = 0; kk < kSB; ++kk) s4[kk & 3] = fma(ml[kk], xs[wave][kk], s4[kk & 3]);
        x -= (s4[0] + s4[1]) + (s4[2] + s4[3]);
        wave_lds_sync();
      }
      if (d0 + lane < n) Y[(int64_t)(d0 + lane) + (int64_t)q * ldy] = x;
      box_put(&a.box[(((size_t)b * kSolveRhs + q) * kSB + lane) * 2], d0 + lane < n ? x : T(0), a.stamp);
    }
    lds_barrier();                                 // part, dtile and mtile are reused by the next block
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

// The substitution's workgroups wait on each other's blocks (bounded waits),
// so the grid never exceeds what the device holds at once; like the panels it
// is an ordinary launch unless ltlt_set_cooperative_panels(1) asks for the
// runtime's cooperative one.
template <typename T, bool UPPER>
hipError_t launch_solve_tri(const SolveTriArgs& a, hipStream_t s) {
  const int cap = solve_tri_max_blocks<T, UPPER>();
  if (cap <= 0) return hipErrorInvalidValue;
  const int grid = a.nblk < cap ? a.nblk : cap;
  return launch_resident_grid(solve_tri_kernel<T, UPPER>, (unsigned)grid, kSThreads, 0, s, a);
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
  {
    // The solution words validate by the stamp of their launch, and stamps are
    // small integers: clear the words first, so that whatever an earlier call
    // left in this part of the workspace can never carry a current stamp.
    const int words = nblk * kSolveRhs * kSB * 2 * 2;   // as 32-bit halves
    hipLaunchKernelGGL(zero_ints_kernel, dim3((words + 255) / 256), dim3(256), 0, s, reinterpret_cast<int*>(w.box),
                       words);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  T* Dinv = static_cast<T*>(w.dinv);
  T* Mf = Dinv + (size_t)nblk * kSB * kSB;
  T* Mb = Mf + (size_t)kLook * nblk * kSB * kSB;
  hipLaunchKernelGGL(solve_dinv_kernel<T>, dim3(nblk), dim3(kWave), 0, s, A, lda, n, Dinv);
  hipLaunchKernelGGL(solve_mmat_kernel<T>, dim3(nblk), dim3(2 * kLook * kWave), 0, s, A, lda, n, nblk, Dinv, Mf, Mb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  for (int q0 = 0; q0 < nrhs; q0 += kSolveRhs) {
    const int nr = nrhs - q0 < kSolveRhs ? nrhs - q0 : kSolveRhs;
    T* Bq = B + (int64_t)q0 * ldb;
    hipLaunchKernelGGL(solve_gather_kernel<T>, dim3((n + 255) / 256, nr), dim3(256), 0, s, n, nr, w.perm, Bq, ldb,
                       Y, w.ldy);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SolveTriArgs ta{};
    ta.A = A; ta.lda = lda; ta.n = n; ta.nblk = nblk; ta.Y = Y; ta.ldy = w.ldy; ta.nr = nr;
    ta.box = w.box; ta.status = w.status; ta.Dinv = Dinv; ta.Mf = Mf; ta.Mb = Mb;
    ta.stamp = next_stamp();
    if ((e = launch_solve_tri<T, false>(ta, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(solve_tridiag_kernel<T>, dim3(1), dim3(2 * nr * kWave), 0, s, n, nr, alpha, ralpha, Y, W,
                       w.ldy);
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
