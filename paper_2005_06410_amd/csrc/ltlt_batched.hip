// Batched small-n path: every matrix (order n <= 64) is factored by ONE wave,
// four matrices per 256-thread workgroup, with no workgroup barrier.
//
// Lane l holds row l+1 of its matrix (positions 1..n-1; row 0 is never
// eliminated, L(:,0) = e_0) and keeps that row's multipliers in registers,
// L[u] = multiplier of step u.  As in the blocked panel, rows never move: an
// exchange of positions k+1 and p swaps the logical positions of two lanes.
// The matrix itself is never updated: the original strict lower triangle
// stays in LDS (packed by column) and column k is refreshed as
//   cv[i] = S(pos[i], pos[k]) + sum_{u<k} g_u L_u[i],
//   g_u = alpha_{u+1} Lrow[u+1] [u <= k-2] - alpha_u Lrow[u-1] [u >= 1],
// Lrow = the multipliers of the row now at position k (Lrow[k-1] = 1), the
// Lx Tx Lx^T form of the accumulated skew rank-2 updates.  g reaches the
// FMAs through DPP row broadcasts (row-broadcast layout, 4 registers).
// Per step: refresh, wave first-maximum, logical exchange, multipliers, the
// pivot row's multipliers staged through LDS, g for the next step.  Global
// traffic is one read and one write of each strict lower triangle, plus
// ipiv and the Pfaffian, which is what bounds this path (HBM).

#include "ltlt_device.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int kBN = 64;                          // largest order handled
constexpr int kBSlots = 64;                      // multiplier slots per lane (steps 0..61)
constexpr int kBPack = kBN * (kBN - 1) / 2;      // packed strict lower triangle
constexpr int kBWaveLds = kBPack + (kBSlots + 1) + (kBSlots + 2) + kBN;   // + alpha history + pivot row + ipiv (kBN ints fit in kBN elements)
constexpr int kBWaves = 4;                       // matrices per workgroup

// Offset of X(i, c), i > c, in the column-packed strict lower triangle.
__device__ __forceinline__ int pack_idx(int n, int i, int c) { return c * (2 * n - c - 1) / 2 + (i - c - 1); }

template <typename T>
__global__ void __launch_bounds__(256, 2) batched_kernel(int n, int batch, T* Aall, int64_t lda, int64_t strideA,
                                                         int* ipiv_all, int64_t strideIpiv, double* logabs,
                                                         int* sign) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int64_t b = (int64_t)blockIdx.x * kBWaves + wave;
  if (b >= batch) return;                          // whole wave leaves together
  T* A = Aall + b * strideA;
  int* ipiv = ipiv_all + b * strideIpiv;
  T* orig = reinterpret_cast<T*>(smem) + (size_t)wave * kBWaveLds;
  T* my_alpha = orig + kBPack;
  T* my_lrowp = my_alpha + (kBSlots + 1);        // my_lrowp[u + 1] = Lrow[u]
  int* my_piv = reinterpret_cast<int*>(my_lrowp + (kBSlots + 2));   // ipiv, written out at the end

  // original strict lower triangle into LDS.  Column c holds n-1-c < 64
  // entries, one per lane (coalesced); the loads of 16 columns are issued
  // before any of them is written, so a matrix costs four memory round trips
  // instead of one per column.
  constexpr int kBFill = 16;
  for (int c0 = 0; c0 + 1 < n; c0 += kBFill) {
    T v[kBFill];
#pragma unroll
    for (int cc = 0; cc < kBFill; ++cc) {
      const int c = c0 + cc;
      v[cc] = (c + 1 < n && lane < n - 1 - c) ? A[(int64_t)(c + 1 + lane) + (int64_t)c * lda] : T(0);
    }
#pragma unroll
    for (int cc = 0; cc < kBFill; ++cc) {
      const int c = c0 + cc;
      if (c + 1 < n && lane < n - 1 - c) orig[pack_idx(n, c + 1, c) + lane] = v[cc];
    }
  }
  if (lane == 0) my_lrowp[0] = T(0);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");

  const bool my_row = lane + 1 < n;
  const int pos = lane + 1;                        // original index of this lane's row
  int lp = pos;                                    // its current position
  T L[kBSlots], gr[4];
#pragma unroll
  for (int c = 0; c < kBSlots; ++c) L[c] = T(0);
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) gr[k4] = T(0);
  T cv = T(0);
  T lv = my_row ? orig[pack_idx(n, pos, 0)] : T(0), lsg = T(1);   // column 0: S(pos, 0)
  int npiv = 0;                                    // exchanges made (Pfaffian sign)

  for (int t = 0; t + 1 < n; ++t) {               // t = k; t = n-2 only forms alpha_{n-2}
    const int k = t;
    const bool active = my_row && lp >= k + 1;
    {
      T acc[4] = {T(0), T(0), T(0), T(0)};
      if (0 < t) refresh16<0>(acc, gr[0], L);
      if (16 < t) refresh16<1>(acc, gr[1], L);
      if (32 < t) refresh16<2>(acc, gr[2], L);
      if (48 < t) refresh16<3>(acc, gr[3], L);
      const T sum = fma(lsg, lv, (acc[0] + acc[1]) + (acc[2] + acc[3]));
      if (active) cv = sum;
    }
    // pivot: first maximum of |cv| by position (NaN never a candidate)
    double av = -1.0;
    if (active) {
      const double mag = (double)fabs(cv);
      if (mag == mag) av = mag;
    }
    double vmax;
    int p;
    const int wl = wave_first_max(av, active ? lp : INT32_MAX, vmax, p);
    T alph;
    int posw;
    if (wl < 0) {                                  // no finite candidate: no exchange
      p = k + 1;
      alph = T(NAN);
      posw = k + 1;
    } else {
      posw = __builtin_amdgcn_readlane(pos, wl);
      alph = (T)vmax;
      if (__builtin_amdgcn_readlane(cv < T(0) ? 1 : 0, wl)) alph = -alph;
    }
    if (lane == 0) my_alpha[t] = alph;
    if (t + 2 == n) break;                         // alpha_{n-2}: last entry of T
    if (lane == 0) my_piv[k + 1] = p;
    if (p != k + 1) {
      ++npiv;
      if (my_row) {
        if (lp == p) lp = k + 1;
        else if (lp == k + 1) lp = p;
      }
    }
    const bool next = my_row && lp >= k + 2;

    // stored column of the pivot row for the next step: S(pos, posw)
    if (next) {
      const int hi = max(pos, posw), lo = min(pos, posw);
      lv = orig[pack_idx(n, hi, lo)];
      lsg = pos > posw ? T(1) : T(-1);
    }
    // the pivot row's multipliers (steps < t) into LDS, from its lane, in
    // groups of 16 slots (entries past t-1 are unused)
    if (wl >= 0 && lane == wl) {
#pragma unroll
      for (int g0 = 0; g0 < kBSlots; g0 += 16) {
        if (g0 < t) {
#pragma unroll
          for (int c = g0; c < g0 + 16; ++c) my_lrowp[c + 1] = L[c];
        }
      }
    }
    // multiplier of step k into slot t
    {
      const T l = next ? ((alph != T(0)) ? cv / alph : T(0)) : T(0);
      const int c = t;
      const bool on = next;
      const T v = l;
#define LTLT_SET_GROUP(G0)                                                                                  \
      if ((c >> 4) == (G0) / 16) {                                                                        \
        _Pragma("unroll") for (int i = 0; i < 16; ++i) L[(G0) + i] = (on && c == (G0) + i) ? v : L[(G0) + i]; \
      }
      LTLT_SET_GROUP(0) LTLT_SET_GROUP(16) LTLT_SET_GROUP(32) LTLT_SET_GROUP(48)
#undef LTLT_SET_GROUP
    }
    if (lane == 0) my_lrowp[t + 1] = T(1);         // Lrow[t] = 1 (unit diagonal)
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // g for step t+1 (t+1 terms), row-broadcast layout
    {
      const int c = lane & 15;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if (kk * 16 <= t) {
          const int u = 16 * kk + c;
          const T a0 = my_alpha[u], a1 = my_alpha[u + 1];
          const T lm = my_lrowp[u], l1 = my_lrowp[u + 2];
          const T up = (u <= t - 1) ? a1 * l1 : T(0);
          const T g = (u >= 1) ? up - a0 * lm : up;
          gr[kk] = (u <= t) ? g : T(0);
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }

  // ---- outputs: A(k+1,k) = alpha_k; the row at final position r holds the
  //      multipliers of the steps before it became final: A(r, u) = L[u],
  //      u <= r-2 ----
  if (my_row) {
    const int r = lp;
#pragma unroll
    for (int u = 0; u < kBSlots; ++u)
      if (u + 2 <= r) A[(int64_t)r + (int64_t)u * lda] = L[u];
  }
  for (int u = lane; u + 1 < n; u += kWave) A[(int64_t)(u + 1) + (int64_t)u * lda] = my_alpha[u];
  if (lane == 0 && n > 0) {
    my_piv[0] = 0;
    my_piv[n - 1] = n - 1;
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  for (int i = lane; i < n; i += kWave) ipiv[i] = my_piv[i];
  // Pfaffian: Pf = det(P) prod_j (-alpha_{2j}), summed in fp64 in a fixed order
  double lg = 0.0;
  int neg = 0, zero = 0;
  if ((n & 1) == 0) {
    for (int jj = lane; jj < n / 2; jj += kWave) {
      const double al = (double)my_alpha[2 * jj];
      if (al == 0.0) zero = 1;
      else { lg += log(fabs(al)); if (-al < 0.0) neg ^= 1; }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    lg += __shfl_xor(lg, off, kWave);
    neg ^= __shfl_xor(neg, off, kWave);
    zero |= __shfl_xor(zero, off, kWave);
  }
  if (lane == 0) {
    neg ^= npiv & 1;
    if (n == 0) { logabs[b] = 0.0; sign[b] = 1; }
    else if ((n & 1) || zero) { logabs[b] = -INFINITY; sign[b] = 0; }
    else { logabs[b] = lg; sign[b] = neg ? -1 : 1; }
  }
}

template <typename T>
hipError_t launch_batched(int n, int batch, T* A, int64_t lda, int64_t strideA, int* ipiv, int64_t strideIpiv,
                          double* logabs, int* sign, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  const size_t lds = (size_t)kBWaves * kBWaveLds * sizeof(T);
  const hipError_t e = ensure_dynamic_lds((const void*)batched_kernel<T>, (int)lds);
  if (e != hipSuccess) return e;
  const int grid = (batch + kBWaves - 1) / kBWaves;
  hipLaunchKernelGGL(batched_kernel<T>, dim3(grid), dim3(256), lds, s, n, batch, A, lda, strideA, ipiv, strideIpiv,
                     logabs, sign);
  return hipGetLastError();
}

template hipError_t launch_batched<double>(int, int, double*, int64_t, int64_t, int*, int64_t, double*, int*,
                                           hipStream_t);
template hipError_t launch_batched<float>(int, int, float*, int64_t, int64_t, int*, int64_t, double*, int*,
                                          hipStream_t);

}  // namespace ltlt
