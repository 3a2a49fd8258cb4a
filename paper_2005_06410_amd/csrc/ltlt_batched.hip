// Batched small-n path: every matrix (order n <= 64) is factored by ONE wave,
// four matrices per 256-thread workgroup, with no workgroup barrier.
//
// Lane l holds row l+1 of its matrix (positions 1..n-1; row 0 is never
// eliminated, L(:,0) = e_0) and keeps that row's multipliers in registers.
// As in the blocked panel, rows never move: an exchange of positions k+1 and
// p swaps the logical positions of two lanes.  The skew matrix S stays in LDS
// as its strict lower triangle (packed by column, indexed by original row),
// and the column steps run in blocks of 16:
//  * inside a block starting at step k0, column k is refreshed from S and the
//    block's own steps only,
//      cv[i] = S(pos[i], pos[k]) + sum_{k0<=u<k} g_u Lb_u[i],
//      g_u = alpha_{u+1} Lrow[u+1] [u <= k-2] - alpha_u Lrow[u-1] [u >= k0+1],
//    Lrow = the in-block multipliers of the row now at position k
//    (Lrow[k-1] = 1), the Lx Tx Lx^T form of the block's skew rank-2
//    updates; g reaches the FMAs through DPP row broadcasts, and only the
//    pivot row's in-block multipliers (at most 15) are staged through LDS;
//  * at the end of a block, the next column (the carry) is refreshed the same
//    way, and the block's update S += Lx Tx Lx^T, Lx = [block multipliers,
//    carry], Tx skew tridiagonal (Tx[u,u+1] = alpha_{k0+u+1}, Tx[15,16] = 1),
//    is applied to the pairs of rows still to be eliminated: each lane forms
//    its row of Bt = Lx Tx^T, the rows still to be eliminated are listed in
//    lane order in a small LDS table, 16 of their Bt rows at a time are
//    spread over the wave with ds_bpermute, and lane a adds
//    sum_u Lx(a,u) Bt(b,u) to S(a,b) for every listed b < a (17
//    DPP-broadcast FMAs per entry).  The 16 steps of a block are unrolled:
//    slot indices are compile-time constants and a step past n-2 simply
//    changes nothing that is read later.
// This is the right-looking skew rank-2k update of the method applied every
// 16 steps inside the wave, with the left-looking refresh confined to the
// block, so a step's refresh, staging and g formation stay short.
// Global traffic is one read and one write of each strict lower triangle,
// plus ipiv and the Pfaffian, which is what bounds this path (HBM).

#include "ltlt_device.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int kBN = 64;                          // largest order handled
constexpr int kBSlots = 64;                      // multiplier slots per lane (steps 0..61)
constexpr int kBBlk = 16;                        // column steps per block
constexpr int kBPack = kBN * (kBN - 1) / 2;      // packed strict lower triangle
constexpr int kBAlpha = kBSlots + 2;             // alpha history (even length keeps the next array 16-byte aligned)
constexpr int kBRow = kBBlk + 2;                 // pivot row's in-block multipliers and its unit
constexpr int kBPiv = kBN + 4;                   // ipiv entries 0..64 (steps past n-2 write up to entry 64)
constexpr int kBWaveLds = kBPack + kBAlpha + kBRow + kBPiv + kBN;   // + ipiv and the trailing-row table (ints)
constexpr int kBWaves = 4;                       // matrices per workgroup

// Offset of X(i, c), i > c, in the column-packed strict lower triangle:
// col_off(n, c) + i.
__device__ __forceinline__ int col_off(int n, int c) { return c * (2 * n - c - 1) / 2 - c - 1; }
__device__ __forceinline__ int pack_idx(int n, int i, int c) { return col_off(n, c) + i; }

// One value from lane addr/4 (ds_bpermute: a cross-lane read, no LDS storage).
__device__ __forceinline__ double bperm(int addr, double v) {
  const int lo = __builtin_amdgcn_ds_bpermute(addr, __double2loint(v));
  const int hi = __builtin_amdgcn_ds_bpermute(addr, __double2hiint(v));
  return __hiloint2double(hi, lo);
}
__device__ __forceinline__ float bperm(int addr, float v) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v)));
}

// In-block refresh, eight slots at a time: acc[c % 4] += g(lane (lane & ~15) + c) * Lb[c]
// for c = 8H .. 8H+7, v_fmac with a DPP row broadcast.  Each asm block starts
// with the two wait states a DPP read needs after a VALU write of its source.
#define LTLT_BF(OP, A, C, X) OP " %" #A ", %4, %" #X " row_newbcast:" #C " row_mask:0xf bank_mask:0xf\n"
#define LTLT_REFRESH8(OP, C0, C1, C2, C3, C4, C5, C6, C7, B)                                                  \
  asm volatile("s_nop 1\n" LTLT_BF(OP, 0, C0, 5) LTLT_BF(OP, 1, C1, 6) LTLT_BF(OP, 2, C2, 7)                 \
                   LTLT_BF(OP, 3, C3, 8) LTLT_BF(OP, 0, C4, 9) LTLT_BF(OP, 1, C5, 10) LTLT_BF(OP, 2, C6, 11) \
                       LTLT_BF(OP, 3, C7, 12)                                                                 \
               : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])                                      \
               : "v"(g), "v"(Lb[B + 0]), "v"(Lb[B + 1]), "v"(Lb[B + 2]), "v"(Lb[B + 3]), "v"(Lb[B + 4]),     \
                 "v"(Lb[B + 5]), "v"(Lb[B + 6]), "v"(Lb[B + 7]))
#define LTLT_REFRESH_FNS(TY, OP)                                                                              \
  template <int H>                                                                                            \
  __device__ __forceinline__ void refresh8(TY (&acc)[4], TY g, const TY (&Lb)[kBBlk]);                        \
  template <>                                                                                                 \
  __device__ __forceinline__ void refresh8<0>(TY (&acc)[4], TY g, const TY (&Lb)[kBBlk]) {                    \
    LTLT_REFRESH8(OP, 0, 1, 2, 3, 4, 5, 6, 7, 0);                                                             \
  }                                                                                                           \
  template <>                                                                                                 \
  __device__ __forceinline__ void refresh8<1>(TY (&acc)[4], TY g, const TY (&Lb)[kBBlk]) {                    \
    LTLT_REFRESH8(OP, 8, 9, 10, 11, 12, 13, 14, 15, 8);                                                       \
  }
LTLT_REFRESH_FNS(double, "v_fmac_f64_dpp")
LTLT_REFRESH_FNS(float, "v_fmac_f32_dpp")
#undef LTLT_REFRESH_FNS
#undef LTLT_REFRESH8
#undef LTLT_BF

// Block update of four columns b = 16q + C0..C0+3 (lanes of one 16-lane row):
// a[j] += sum_u R_u(lane C0+j of each row) * X_u, u = U0..U0+8, where R_u holds
// row 16q + (lane & 15) of Bt and X the lane's own row of Lx.
#define LTLT_BU1(OP, C0, C1, C2, C3, R, X)                                     \
  OP " %0, %" #R ", %" #X " row_newbcast:" #C0 " row_mask:0xf bank_mask:0xf\n" \
  OP " %1, %" #R ", %" #X " row_newbcast:" #C1 " row_mask:0xf bank_mask:0xf\n" \
  OP " %2, %" #R ", %" #X " row_newbcast:" #C2 " row_mask:0xf bank_mask:0xf\n" \
  OP " %3, %" #R ", %" #X " row_newbcast:" #C3 " row_mask:0xf bank_mask:0xf\n"
#define LTLT_BU9(OP, C0, C1, C2, C3, U0)                                                                         \
  asm volatile("s_nop 1\n" LTLT_BU1(OP, C0, C1, C2, C3, 4, 13) LTLT_BU1(OP, C0, C1, C2, C3, 5, 14)              \
                   LTLT_BU1(OP, C0, C1, C2, C3, 6, 15) LTLT_BU1(OP, C0, C1, C2, C3, 7, 16)                       \
                       LTLT_BU1(OP, C0, C1, C2, C3, 8, 17) LTLT_BU1(OP, C0, C1, C2, C3, 9, 18)                   \
                           LTLT_BU1(OP, C0, C1, C2, C3, 10, 19) LTLT_BU1(OP, C0, C1, C2, C3, 11, 20)             \
                               LTLT_BU1(OP, C0, C1, C2, C3, 12, 21)                                              \
               : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3])                                                  \
               : "v"(R[U0 + 0]), "v"(R[U0 + 1]), "v"(R[U0 + 2]), "v"(R[U0 + 3]), "v"(R[U0 + 4]),                 \
                 "v"(R[U0 + 5]), "v"(R[U0 + 6]), "v"(R[U0 + 7]), "v"(R[U0 + 8]), "v"(X[U0 + 0]),                 \
                 "v"(X[U0 + 1]), "v"(X[U0 + 2]), "v"(X[U0 + 3]), "v"(X[U0 + 4]), "v"(X[U0 + 5]),                 \
                 "v"(X[U0 + 6]), "v"(X[U0 + 7]), "v"(X[U0 + 8]))
#define LTLT_UPD_FNS(TY, OP)                                                                              \
  template <int G>                                                                                        \
  __device__ __forceinline__ void upd4(TY (&a)[4], const TY (&R)[18], const TY (&X)[18]);                 \
  template <>                                                                                             \
  __device__ __forceinline__ void upd4<0>(TY (&a)[4], const TY (&R)[18], const TY (&X)[18]) {            \
    LTLT_BU9(OP, 0, 1, 2, 3, 0);                                                                          \
    LTLT_BU9(OP, 0, 1, 2, 3, 9);                                                                          \
  }                                                                                                       \
  template <>                                                                                             \
  __device__ __forceinline__ void upd4<1>(TY (&a)[4], const TY (&R)[18], const TY (&X)[18]) {            \
    LTLT_BU9(OP, 4, 5, 6, 7, 0);                                                                          \
    LTLT_BU9(OP, 4, 5, 6, 7, 9);                                                                          \
  }                                                                                                       \
  template <>                                                                                             \
  __device__ __forceinline__ void upd4<2>(TY (&a)[4], const TY (&R)[18], const TY (&X)[18]) {            \
    LTLT_BU9(OP, 8, 9, 10, 11, 0);                                                                        \
    LTLT_BU9(OP, 8, 9, 10, 11, 9);                                                                        \
  }                                                                                                       \
  template <>                                                                                             \
  __device__ __forceinline__ void upd4<3>(TY (&a)[4], const TY (&R)[18], const TY (&X)[18]) {            \
    LTLT_BU9(OP, 12, 13, 14, 15, 0);                                                                      \
    LTLT_BU9(OP, 12, 13, 14, 15, 9);                                                                      \
  }
LTLT_UPD_FNS(double, "v_fmac_f64_dpp")
LTLT_UPD_FNS(float, "v_fmac_f32_dpp")
#undef LTLT_UPD_FNS
#undef LTLT_BU9
#undef LTLT_BU1

// Columns 16q + 4G .. 16q + 4G + 3 of the trailing rows in lane order (see
// upd4): for the row b of each, S(pos, b) += sum_u Lx(pos,u) Bt(b,u) when
// b < pos and this lane's row is trailing.  pbv holds, in lane c of each
// 16-lane row, the original index of column 16q + c (0 past the last).
template <int G, typename T>
__device__ __forceinline__ void update_group(T* orig, int n, int pos, bool ta, int pbv, const T (&R)[18],
                                             const T (&X)[18]) {
  int pb[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) pb[j] = __builtin_amdgcn_readlane(pbv, 4 * G + j);
  if (pb[0] == 0) return;                        // past the last trailing row
  T a[4];
  int idx[4];
  bool ok[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    ok[j] = ta && pb[j] != 0 && pos > pb[j];
    idx[j] = ok[j] ? col_off(n, pb[j]) + pos : 0;
    a[j] = orig[idx[j]];
  }
  upd4<G>(a, R, X);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (ok[j]) orig[idx[j]] = a[j];
}

// Waves per SIMD: fp64 two (the packed triangle takes 17.8 KB of LDS per
// matrix, and the registers fill 256 VGPRs); fp32 four, by capping it at 128
// VGPRs (a few values then live in scratch, which still beats three waves).
template <typename T>
__global__ void __launch_bounds__(256, sizeof(T) == 4 ? 4 : 2) batched_kernel(int n, int batch, T* Aall, int64_t lda, int64_t strideA,
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
  T* my_lrow = my_alpha + kBAlpha;                 // my_lrow[u] = Lrow[k0 + u]
  int* my_piv = reinterpret_cast<int*>(my_lrow + kBRow);   // ipiv, written out at the end
  int* my_tab = reinterpret_cast<int*>(my_lrow + kBRow + kBPiv);   // lanes of the trailing rows, in lane order

  // strict lower triangle into LDS.  Column c holds n-1-c < 64 entries, one
  // per lane (coalesced); the loads of all columns are issued before any of
  // them is written, so a matrix costs one memory round trip.
  constexpr int kBFill = kBN;
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
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");

  const bool my_row = lane + 1 < n;
  const int pos = lane + 1;                        // original index of this lane's row
  const int cof = col_off(n, pos);                 // its column's offset in the packed triangle
  int lp = pos;                                    // its current position
  T L[kBSlots], Lb[kBBlk];                         // finished blocks' multipliers; the current block's
#pragma unroll
  for (int c = 0; c < kBSlots; ++c) L[c] = T(0);
#pragma unroll
  for (int c = 0; c < kBBlk; ++c) Lb[c] = T(0);
  T gr = T(0);                                     // g of the current block, row-broadcast layout
  T cv = T(0);
  T lv = my_row ? orig[pack_idx(n, pos, 0)] : T(0), lsg = T(1);   // column 0: S(pos, 0)
  int npiv = 0;                                    // exchanges made (Pfaffian sign)

  // Every block runs all 16 steps: a step with k + 2 >= n has at most the
  // row at position n-1 as candidate and no row below it, so it forms alpha_k
  // (k = n-2) or nothing, exchanges nothing and leaves every multiplier 0;
  // its alpha and pivot entries past n-2 are never read.
  int k0 = 0;
  while (k0 + 1 < n) {
#pragma unroll
    for (int tt = 0; tt < kBBlk; ++tt) {          // step k = k0 + tt
      const int k = k0 + tt;
      const bool active = my_row && lp >= k + 1;
      if (tt > 0 || k0 == 0) {                    // a block's first column is the carry of the block before
        T acc[4] = {T(0), T(0), T(0), T(0)};
        if (tt > 0) refresh8<0>(acc, gr, Lb);
        if (tt > 8) refresh8<1>(acc, gr, Lb);
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
      // no finite candidate (wl < 0): no exchange, alpha NaN
      const int wsrc = wl < 0 ? 0 : wl;
      const int posw = wl < 0 ? k + 1 : __builtin_amdgcn_readlane(pos, wsrc);
      const int wneg = __builtin_amdgcn_readlane(cv < T(0) ? 1 : 0, wsrc);
      const T alph = wl < 0 ? T(NAN) : (wneg ? -(T)vmax : (T)vmax);
      if (wl < 0) p = k + 1;
      my_alpha[k] = alph;                          // uniform values, stored by every lane
      my_piv[k + 1] = p;                           // k + 1 <= 64 < kBPiv
      npiv += p != k + 1 ? 1 : 0;
      if (my_row) lp = lp == p ? k + 1 : (lp == k + 1 ? p : lp);
      const bool next = my_row && lp >= k + 2;

      // stored column of the pivot row for the next step: S(pos, posw)
      {
        const int idx = pos > posw ? col_off(n, posw) + pos : cof + posw;
        const T v = orig[next ? idx : 0];
        if (next) {
          lv = v;
          lsg = pos > posw ? T(1) : T(-1);
        }
      }
      // the pivot row's in-block multipliers (steps k0 .. k-1) into LDS
      if (wl >= 0 && lane == wl) {
#pragma unroll
        for (int u = 0; u < tt; ++u) my_lrow[u] = Lb[u];
      }
      my_lrow[tt] = T(1);                          // Lrow[k] = 1 (unit diagonal), every lane
      // multiplier of step k: the division is issued after the LDS stores
      // above and before the wait below, so its latency overlaps theirs
      asm volatile("" : "+v"(cv) : : "memory");
      Lb[tt] = next ? ((alph != T(0)) ? cv / alph : T(0)) : T(0);
      asm volatile("s_waitcnt lgkmcnt(0)" : : "v"(Lb[tt]) : "memory");
      // g for step k+1: in-block terms u = k0 .. k, row-broadcast layout
      {
        const int u = lane & 15;
        T a0 = my_alpha[k0 + u], a1 = my_alpha[k0 + u + 1];
        T lm = my_lrow[u > 0 ? u - 1 : 0], l1 = my_lrow[u + 1];
        asm volatile("" : "+v"(a0), "+v"(a1), "+v"(lm), "+v"(l1));   // all four loads in one round trip
        const T up = (u <= tt - 1) ? a1 * l1 : T(0);
        const T g = (u >= 1) ? up - a0 * lm : up;
        gr = (u <= tt) ? g : T(0);
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    const int kn = k0 + kBBlk;                     // first step of the next block
    if (kn + 1 >= n) break;
    // the carry: column kn refreshed with all of this block's steps
    const bool ta = my_row && lp >= kn + 1;        // rows still to be eliminated
    {
      T acc[4] = {T(0), T(0), T(0), T(0)};
      refresh8<0>(acc, gr, Lb);
      refresh8<1>(acc, gr, Lb);
      const T sum = fma(lsg, lv, (acc[0] + acc[1]) + (acc[2] + acc[3]));
      if (ta) cv = sum;
    }
    // S += Lx Tx Lx^T on the trailing rows: Lx = [Lb, carry], Bt = Lx Tx^T,
    // each entry of this lane's Bt row formed just before it is spread
    {
      T X[18];
#pragma unroll
      for (int u = 0; u < kBBlk; ++u) X[u] = Lb[u];
      X[16] = cv;
      X[17] = T(0);
      const T* al = my_alpha + k0;                 // al[u] = alpha_{k0+u}
      // the trailing rows' lanes in lane order: my_tab[j] = lane of the j-th
      const uint64_t tmask = __ballot(ta);         // bit l: row l+1 trailing
      const int m = __popcll(tmask);
      if (ta) my_tab[__builtin_amdgcn_mbcnt_hi((unsigned)(tmask >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)tmask, 0u))] = lane;
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll 1
      for (int q = 0; 16 * q < m; ++q) {
        const int j = 16 * q + (lane & 15);        // this lane's column of the group
        const int src = j < m ? my_tab[j] : 0;
        const int pbv = j < m ? src + 1 : 0;       // original index of that column's row
        const int addr = src * 4;
        T R[18];
        R[0] = bperm(addr, al[1] * X[1]);
#pragma unroll
        for (int u = 1; u < kBBlk - 1; ++u) R[u] = bperm(addr, al[u + 1] * X[u + 1] - al[u] * X[u - 1]);
        R[15] = bperm(addr, X[16] - al[15] * X[14]);
        R[16] = bperm(addr, -X[15]);
        R[17] = T(0);
        update_group<0>(orig, n, pos, ta, pbv, R, X);
        update_group<1>(orig, n, pos, ta, pbv, R, X);
        update_group<2>(orig, n, pos, ta, pbv, R, X);
        update_group<3>(orig, n, pos, ta, pbv, R, X);
      }
    }
    // archive the block's multipliers
#define LTLT_ARCHIVE(B)                                                   \
    if (k0 == 16 * B) {                                                   \
      _Pragma("unroll") for (int u = 0; u < kBBlk; ++u) L[16 * B + u] = Lb[u]; \
    }
    LTLT_ARCHIVE(0) LTLT_ARCHIVE(1) LTLT_ARCHIVE(2) LTLT_ARCHIVE(3)
#pragma unroll
    for (int u = 0; u < kBBlk; ++u) Lb[u] = T(0);
    gr = T(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    k0 = kn;
  }
  LTLT_ARCHIVE(0) LTLT_ARCHIVE(1) LTLT_ARCHIVE(2) LTLT_ARCHIVE(3)
#undef LTLT_ARCHIVE

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
