// Trailing update of one block: for the m x m trailing block C (skew, held in
// its strict lower triangle) and each pair i > c,
//     C(i,c) <- S(perm[i], perm[c]) + sum_u Lx(i,u) Bt(c,u),
// S(a,b) = C(a,b) for a > b and -C(b,a) for a < b.
// With Bt = Lx Tx^T this is C + Lx Tx Lx^T: the block's 2*nb rank-1 terms
// collapsed into one product of inner dimension nb+1 (the skew rank-2k update
// A22 - (L21 W^T - W L21^T) of the method, with W formed from L21 and the
// alphas, so only the lower triangle is computed, once).
//
// gfx950 mapping:
//  * 256-thread workgroups on 128x128 tiles of the LOWER triangle only
//    (tile row >= tile column), a persistent grid of three workgroups per CU
//    walking an XCD-aware tile order (while one drains its epilogue to HBM,
//    the other two keep the matrix cores busy);
//  * each of the 4 waves owns a 64x64 sub-tile = 4x4 MFMA blocks of 16x16
//    (v_mfma_f64_16x16x4_f64, or v_mfma_f32_16x16x4_f32 for fp32),
//    accumulating in registers;
//  * Lx and Bt are streamed through LDS in K-chunks of 8 columns, double
//    buffered (37 KB of LDS per workgroup).  In fp64 each 128-row column of
//    a chunk goes straight from global memory into LDS with one
//    global_load_lds_dwordx4 per wave (no register staging; the copy of
//    chunk k+1 runs under the MFMAs of chunk k); fp32, and operands whose
//    columns are not 16-byte aligned, take coalesced loads staged through
//    registers;
//  * the epilogue reads the old value through perm (the exchanges of the
//    panel, applied as a gather: every displaced source lies outside the
//    block being written, so tiles never race), adds, and writes the lower
//    entry only; diagonal tiles mask i <= c.  Per block the kernel moves
//    8 m^2 bytes (read + write of the lower triangle) against m^2 (nb+1)
//    flops, about (nb+1)/8 flop/byte in fp64.
// The operand staging follows the paper's packing idea (section 2, packing
// of A_c/B_c amortized over the inner loops), re-shaped for LDS and MFMA.

#include "ltlt_device.h"
#include "ltlt_internal.h"

#include <type_traits>

namespace ltlt {

constexpr int kMT = 128;     // tile edge
constexpr int kKC = 8;       // K chunk
constexpr int kLd = kMT + 16;   // LDS row stride of an operand chunk (bank spread)
constexpr int kUpdateGrid = 768;   // persistent grid: three workgroups on each of 256 CUs
constexpr int kUpdateWgPerCu = 3;

typedef double v4d __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;
template <> struct Mfma<double> {
  typedef v4d acc_t;
  static __device__ __forceinline__ acc_t run(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  // output element v of lane l sits at row (l/16) + 4v, column l%16
  static __device__ __forceinline__ int row(int l, int v) { return (l >> 4) + 4 * v; }
};
template <> struct Mfma<float> {
  typedef v4f acc_t;
  static __device__ __forceinline__ acc_t run(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  // output element v of lane l sits at row 4(l/16) + v, column l%16
  static __device__ __forceinline__ int row(int l, int v) { return 4 * (l >> 4) + v; }
};

// One 128 x kKC chunk of an operand, thread -> column tid / kTpc, rows
// (tid % kTpc) + kTpc e, e < kRpt: each load instruction reads kTpc
// consecutive rows of a column, and each LDS store writes kTpc consecutive
// entries.
constexpr int kTpc = kThreads / kKC;           // threads per chunk column
constexpr int kRpt = kMT / kTpc;                 // rows per thread
template <typename T>
__device__ __forceinline__ void load_chunk(const T* __restrict__ X, int64_t ldx, int m, int K, int r0, int k0,
                                           T (&reg)[kRpt], int tid) {
  const int col = tid / kTpc;
  const int kk = k0 + col;
  const int rbase = r0 + (tid % kTpc);
  if (kk < K && r0 + kMT <= m) {
    const T* p = X + (int64_t)kk * ldx + rbase;
#pragma unroll
    for (int e = 0; e < kRpt; ++e) reg[e] = p[kTpc * e];
  } else {
#pragma unroll
    for (int e = 0; e < kRpt; ++e) {
      const int r = rbase + kTpc * e;
      reg[e] = (kk < K && r < m) ? X[(int64_t)kk * ldx + r] : T(0);
    }
  }
}

// LDS chunk rows are kLd apart (128 + 16): the four k-rows one fragment read
// touches then fall on different banks.
template <typename T>
__device__ __forceinline__ void store_chunk(T* __restrict__ S, const T (&reg)[kRpt], int tid) {
  const int col = tid / kTpc;
  const int rr = tid % kTpc;
#pragma unroll
  for (int e = 0; e < kRpt; ++e) S[col * kLd + rr + kTpc * e] = reg[e];
}

// Direct global -> LDS copy of one 128 x kKC chunk (fp64): wave w moves
// columns w kKC/4 .. (w+1) kKC/4 - 1; one global_load_lds_dwordx4 fills one
// 1 KB LDS column
// (lane l -> rows 2l, 2l+1).  Rows are clamped into [0, mr2) (mr2 = m rounded
// up to even: the caller guarantees that range is readable); rows >= m only
// feed outputs that are masked.  Columns in [K, K4) are zeroed so the last
// 4-wide MFMA step adds nothing.
__device__ __forceinline__ void dma_chunk(const double* __restrict__ X, int64_t ldx, int mr2, int K, int K4, int r0,
                                          int k0, double* S, int wave, int lane) {
  const int r = min(r0 + 2 * lane, mr2 - 2);
#pragma unroll
  for (int j = 0; j < kKC / 4; ++j) {
    const int cl = wave * (kKC / 4) + j;
    const int kk = k0 + cl;
    if (kk < K) {
      __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)(X + (int64_t)kk * ldx + r),
                                       (void __attribute__((address_space(3)))*)(S + cl * kLd), 16, 0, 0);
    } else if (kk < K4) {
      S[cl * kLd + 2 * lane] = 0.0;
      S[cl * kLd + 2 * lane + 1] = 0.0;
    }
  }
}

// Old values S(perm[i], perm[c]) of one 16-column slice for the lane's row i
// (strict lower triangle only; other entries read the valid C(1,0) and are
// discarded).  The sources never change during the update: they are either
// the tile's own entries or lie outside the block being written.
template <typename T>
__device__ __forceinline__ void gather_slice(const T* __restrict__ C, int64_t ldc, int m, int i, int pr,
                                             const int* pcol, int c0, int cl0, T (&out)[16]) {
  // the slice's 16 column sources first (one LDS round trip), then the
  // addresses without branches: S(pr, pc) = C(max, min), negated above the
  // diagonal
  int pcs[16];
#pragma unroll
  for (int cc = 0; cc < 16; ++cc) pcs[cc] = pcol[cl0 + cc];
#pragma unroll
  for (int cc = 0; cc < 16; ++cc) {
    const int c = c0 + cl0 + cc;
    const int pc = pcs[cc];
    const bool in = (i > c) && (i < m);
    const bool low = pr > pc;
    const int hi = low ? pr : pc, lo = low ? pc : pr;
    const int64_t off = in ? (int64_t)hi + (int64_t)lo * ldc : 1;
    const T val = C[off];
    out[cc] = low ? val : -val;
  }
}

// Tile scheduling.  Workgroups are dispatched round-robin over the 8 XCDs
// (block b runs on XCD b % 8) and each XCD has its own L2.  The lower-
// triangular tile set is enumerated in groups of kGrp x kGrp tiles (tiles of
// a group share kGrp row blocks of Lx and kGrp column blocks of Bt), and XCD x
// is given the x-th contiguous eighth of that order, so the workgroups resident
// on one XCD work through the same few groups and their operands stay in
// that XCD's L2.
constexpr int kXcd = 8;
constexpr int kGrp = 8;

__device__ __forceinline__ int tri_index_decode(int b, int& J) {
  int I = (int)((sqrt(8.0 * (double)b + 1.0) - 1.0) * 0.5);
  while ((I + 1) * (I + 2) / 2 <= b) ++I;
  while (I * (I + 1) / 2 > b) --I;
  J = b - I * (I + 1) / 2;
  return I;
}

// The grouped order: groups (GI, GJ), GJ <= GI, row-major; full groups hold
// kGrp*kGrp tiles, diagonal groups hI(hI+1)/2, edge groups fewer.  Group row
// GI holds GI off-diagonal groups of hI x kGrp tiles (hI = row blocks in the
// group row) and one diagonal group.  A workgroup's tile indices only grow,
// so it keeps a cursor on the group row of its last tile: locating the next
// tile moves over a group row or two instead of walking all groups from the
// start (that walk ran on the scalar unit that the CU's waves share).
struct TileCursor { int GI, rowbase; };

__device__ __forceinline__ int group_row_tiles(int GI, int tiles) {
  const int hI = min(kGrp, tiles - GI * kGrp);
  return GI * hI * kGrp + hI * (hI + 1) / 2;
}

__device__ __forceinline__ void grouped_tile(TileCursor& cs, int q, int tiles, int& I, int& J) {
  const int ng = (tiles + kGrp - 1) / kGrp;
  while (cs.GI < ng && q >= cs.rowbase + group_row_tiles(cs.GI, tiles)) {
    cs.rowbase += group_row_tiles(cs.GI, tiles);
    ++cs.GI;
  }
  const int GI = cs.GI;
  const int hI = min(kGrp, tiles - GI * kGrp);
  const int off = q - cs.rowbase;
  const int full = GI * hI * kGrp;               // tiles of the off-diagonal groups
  if (off < full) {
    const int GJ = off / (hI * kGrp), rem = off - GJ * (hI * kGrp);
    I = GI * kGrp + rem / kGrp;
    J = GJ * kGrp + rem % kGrp;
  } else {
    int jj;
    const int ii = tri_index_decode(off - full, jj);
    I = GI * kGrp + ii;
    J = GI * kGrp + jj;
  }
}

// The grid is persistent (at most three workgroups per CU).  XCD x owns the
// x-th contiguous eighth [lo, hi) of the grouped order and its workgroups
// (blocks b with b % 8 == x) take those tiles in turn.  Every tile is covered
// when the grid has at least 8 blocks or one block per tile (the launch uses
// min(tiles, kUpdateGrid) blocks).
struct TileRange { int q, hi, step; };
__device__ __forceinline__ TileRange tiles_of_block(int b, int nblocks, int ntiles) {
  const int x = b % kXcd, l = b / kXcd;
  const int per = ntiles / kXcd, extra = ntiles % kXcd;
  const int lo = x * per + min(x, extra);
  const int hi = lo + per + (x < extra ? 1 : 0);
  const int cx = (nblocks - x + kXcd - 1) / kXcd;  // workgroups on XCD x
  return TileRange{lo + l, hi, cx};
}

template <typename T, bool DMA>
__global__ void __launch_bounds__(kThreads, kUpdateWgPerCu) update_kernel(UpdateArgs a) {
  typedef typename Mfma<T>::acc_t acc_t;
  // operand chunks As[2][kKC*kLd], Bs[2][kKC*kLd]; reused by the epilogue
  __shared__ __align__(16) T lds[4 * kKC * kLd];
  T (*As)[kKC * kLd] = reinterpret_cast<T (*)[kKC * kLd]>(lds);
  T (*Bs)[kKC * kLd] = reinterpret_cast<T (*)[kKC * kLd]>(lds + 2 * kKC * kLd);
  __shared__ int prow[kMT], pcol[kMT];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 1, wc = wave & 1;

  const TileRange tr = tiles_of_block(blockIdx.x, gridDim.x, a.tiles * (a.tiles + 1) / 2);
  TileCursor cursor{0, 0};
  for (int q = tr.q; q < tr.hi; q += tr.step) {
  __syncthreads();                                 // LDS of the previous tile is free
  int I, J;
  grouped_tile(cursor, q, a.tiles, I, J);
  const int r0 = I * kMT, c0 = J * kMT;
  const int m = a.m, K = a.K;

  const T* Lx = static_cast<const T*>(a.Lx);
  const T* Bt = static_cast<const T*>(a.Bt);

  acc_t acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = acc_t{0, 0, 0, 0};

  const int mr2 = (m + 1) & ~1, K4 = (K + 3) & ~3;
  T ra[kRpt], rb[kRpt];
  if constexpr (DMA) {
    dma_chunk((const double*)Lx, a.ldl, mr2, K, K4, r0, 0, (double*)As[0], wave, lane);
    dma_chunk((const double*)Bt, a.ldb, mr2, K, K4, c0, 0, (double*)Bs[0], wave, lane);
  } else {
    load_chunk<T>(Lx, a.ldl, m, K, r0, 0, ra, tid);
    load_chunk<T>(Bt, a.ldb, m, K, c0, 0, rb, tid);
    store_chunk<T>(As[0], ra, tid);
    store_chunk<T>(Bs[0], rb, tid);
  }
  if (tid < kMT) {
    // sources clamped into the caller's range (in the factorization, the
    // positions held since block start): a complete order is unchanged, and
    // one left unfinished by a panel that gave up cannot take the gather
    // outside the matrix
    const int ri = r0 + tid, ci = c0 + tid;
    prow[tid] = (a.perm && ri < m) ? min(max(a.perm[ri] - a.perm_base, a.perm_lo), a.perm_hi) : ri;
    pcol[tid] = (a.perm && ci < m) ? min(max(a.perm[ci] - a.perm_base, a.perm_lo), a.perm_hi) : ci;
  }
  if constexpr (DMA) __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): this wave's chunk copies landed
  __syncthreads();

  // epilogue geometry: lane l of wave (wr, wc) finishes row wr*64 + l of the tile
  T* C = static_cast<T*>(a.C);
  const int64_t ldc = a.ldc;
  const int rl = wr * 64 + lane;
  const int i = r0 + rl;
  const int pr = prow[rl];

  const int nchunk = (K + kKC - 1) / kKC;
  for (int ch = 0; ch < nchunk; ++ch) {
    const int cur = ch & 1;
    const bool more = ch + 1 < nchunk;
    if (more) {
      if constexpr (DMA) {
        dma_chunk((const double*)Lx, a.ldl, mr2, K, K4, r0, (ch + 1) * kKC, (double*)As[cur ^ 1], wave, lane);
        dma_chunk((const double*)Bt, a.ldb, mr2, K, K4, c0, (ch + 1) * kKC, (double*)Bs[cur ^ 1], wave, lane);
      } else {
        load_chunk<T>(Lx, a.ldl, m, K, r0, (ch + 1) * kKC, ra, tid);
        load_chunk<T>(Bt, a.ldb, m, K, c0, (ch + 1) * kKC, rb, tid);
      }
    }
    const T* as = As[cur];
    const T* bs = Bs[cur];
    const int ksteps = min(kKC, K - ch * kKC);
    for (int k4 = 0; k4 < ksteps; k4 += 4) {
      const int kr = k4 + (lane >> 4);
      T af[4], bf[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) af[x] = as[kr * kLd + wr * 64 + x * 16 + (lane & 15)];
#pragma unroll
      for (int y = 0; y < 4; ++y) bf[y] = bs[kr * kLd + wc * 64 + y * 16 + (lane & 15)];
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = Mfma<T>::run(af[x], bf[y], acc[x][y]);
    }
    if constexpr (DMA) {
      __builtin_amdgcn_s_waitcnt(0x0f70);          // vmcnt(0): next chunk landed
    } else if (more) {
      store_chunk<T>(As[cur ^ 1], ra, tid);
      store_chunk<T>(Bs[cur ^ 1], rb, tid);
    }
    __syncthreads();
  }

  // ---- epilogue: stage through LDS, then coalesced add/store ----
  // The MFMA output layout spreads a lane's values over 4 rows x 16 columns,
  // which would make every global access touch 16 partial lines.  Each wave
  // instead writes one 16-column slice of its 64x64 sub-tile to LDS
  // ([column][row], padded), then lane l handles row l of each column: every
  // load/store instruction covers 64 consecutive rows of one column.  The old
  // values of a slice are gathered after it is staged (at 168 VGPRs there is
  // no room to hold them across the K loop); their latency is covered by the
  // other workgroups on the CU.
  constexpr int kEp = 65;                          // padded column stride in LDS
  static_assert(4 * 16 * kEp <= 4 * kKC * kLd, "epilogue staging must fit the operand LDS");
  T* stage = lds + wave * (16 * kEp);              // 16 columns x 65 per wave
#pragma unroll
  for (int y = 0; y < 4; ++y) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        stage[(lane & 15) * kEp + x * 16 + Mfma<T>::row(lane, v)] = acc[x][y][v];
    __builtin_amdgcn_s_waitcnt(0xc07f);            // lgkmcnt(0): this wave's LDS writes done
    T oldv[16];
    gather_slice<T>(C, ldc, m, i, pr, pcol, c0, wc * 64 + y * 16, oldv);
#pragma unroll
    for (int cc = 0; cc < 16; ++cc) {
      const int c = c0 + wc * 64 + y * 16 + cc;
      if ((i > c) && (i < m)) C[(int64_t)i + (int64_t)c * ldc] = oldv[cc] + stage[cc * kEp + lane];
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);            // reads of this slice done before it is overwritten
  }
  }
}

template <typename T>
hipError_t launch_update(const UpdateArgs& a, hipStream_t s) {
  const int tiles = (a.m + kMT - 1) / kMT;
  const int64_t nblk = (int64_t)tiles * (tiles + 1) / 2;
  if (nblk <= 0) return hipSuccess;
  UpdateArgs c = a;
  c.tiles = tiles;
  const int64_t grid = nblk < kUpdateGrid ? nblk : kUpdateGrid;
  // direct-to-LDS operand copies need 16-byte aligned column pairs and one
  // readable row past m when m is odd
  const bool dma = std::is_same<T, double>::value && (reinterpret_cast<uintptr_t>(a.Lx) % 16 == 0) &&
             (reinterpret_cast<uintptr_t>(a.Bt) % 16 == 0) && (a.ldl % 2 == 0) && (a.ldb % 2 == 0) &&
             ((a.m % 2 == 0) || a.pad_row);
  if constexpr (std::is_same<T, double>::value) {
    if (dma) {
      hipLaunchKernelGGL((update_kernel<T, true>), dim3((unsigned)grid), dim3(kThreads), 0, s, c);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((update_kernel<T, false>), dim3((unsigned)grid), dim3(kThreads), 0, s, c);
  return hipGetLastError();
}

template hipError_t launch_update<double>(const UpdateArgs&, hipStream_t);
template hipError_t launch_update<float>(const UpdateArgs&, hipStream_t);

}  // namespace ltlt
