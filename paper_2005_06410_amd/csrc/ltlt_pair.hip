// Pfaffian-only path: the even column steps of the pivoted reduction.
//
// After column k is eliminated with pivot row k+1 (pivot search, exchange,
// multipliers l = column k / alpha_k, skew rank-2 update of the trailing
// matrix with l and v = column k+1), row k of the matrix has the single
// nonzero -alpha_k at column k+1, so the Pfaffian expands along it:
//   Pf(X) = det(P) (-alpha_k) Pf(X without indices k and k+1).
// Column k+1 is therefore never eliminated; the next step is column k+2, and
// Pf(X) = (-1)^(#exchanges) prod_{k even} (-alpha_k).  Half the column steps,
// so half the grid-wide pivot agreements of the full reduction.
//
// Pair panel (one block of bw columns, bw/2 steps, rows at positions >= j+1),
// the register slots and exchange of the full panel; wave 0 of each
// workgroup holds no rows and only publishes and polls, so that the other
// seven waves' work on the next column overlaps its round trip (R = 7*64/S
// rows per workgroup).  Step u
// leaves two slots in every row still in play: slot 2u = l_u (multiplier)
// and slot 2u+1 = w_u (column k+1 below row k+1, refreshed: the v of the
// rank-2 update).  The updates pending within the block are
//   sum_u l_u w_u^T - w_u l_u^T = Lp J Lp^T,   J = diag([[0, 1], [-1, 0]]),
// so column c of the current matrix at row i is
//   S(pos[i], q_c) + sum_s Lp[s][i] g_s,   g_{2u} = w_u(row c), g_{2u+1} = -l_u(row c),
// with q_c the block-start index of the row at position c.  Per step k:
//   1. pivot of column k (rows at positions >= k+1), exchange;
//   2. l = cv / alpha_k (slot 2u);
//   3. loads: S(pos, posw) and S(pos, q) for the stored parts of columns k+1
//      and k+2 (q = row now at position k+2), the slots of rows posw and q;
//   4. the two newest slots of row q (its l_u and w_u), which every lane needs
//      in the g of column k+2, are recomputed by every wave from row q's slots
//      and the g's of columns k and k+1 (two short dot products), so no
//      second agreement per step is needed;
//   5. one pass over the slots forms w (column k+1, slot 2u+1) and the next
//      column k+2.
// Unlike the full reduction, whose next column is the pivot's own, the next
// column here belongs to the row at position k+2, which is known before the
// pivot is (it changes only when the pivot comes from position k+2).  Its
// loads, its dot product with the g of column k and the pass over its slots
// for column k+2 therefore run while wave 0 waits for the other workgroups'
// records -- over the slots older than the previous step only: the previous
// step's two slots of that row are guaranteed visible in G only once every
// record of this step has arrived (each workgroup waits for its G stores
// before publishing), so they are loaded with the pivot row's data and their
// two terms added then (each row keeps its own newest l and w, and the g of
// column k at those two slots, in registers).  After the agreement only the
// pivot row's part remains (its slots, S(pos, posw), the g of column k+1,
// one pass, two scalars); the speculative part is redone in the rare case
// that the row at k+2 changed.
// Outputs of the block for the trailing rows (positions >= j+bw): Lx = Lp in
// slot order and Bt = Lp J^T (Bt column 2u = w_u, 2u+1 = -l_u), one rank-bw
// product for the trailing update; alpha_k and the pivots.

#include "ltlt_device.h"
#include "ltlt_exchange.h"
#include "ltlt_internal.h"

namespace ltlt {

// LDS per wave: the slots of the pivot row (TOT), of row q (TOT) and the g
// of the current column by slot (TOT).
__host__ __device__ constexpr int pair_wave_lds_bytes(int tot, int tsize) { return 3 * tot * tsize; }
template <typename T>
size_t pair_lds_bytes(int bw, int /*R*/) {
  return (size_t)kPanelWaves * pair_wave_lds_bytes(KC * panel_split(bw), (int)sizeof(T));
}

// Row g of the slots held in buf (slot s of a row: s = 2u -> l_u, 2u+1 -> w_u):
// g_{2u} = w_u, g_{2u+1} = -l_u, for slots s < ns; 0 elsewhere.
template <typename T>
__device__ __forceinline__ T g_of(const T* buf, int s, int ns) {
  if (s >= ns) return T(0);
  return (s & 1) ? -buf[s - 1] : buf[s + 1];
}

// Wave-wide sum in a fixed order (every lane gets it): DPP row shifts give
// each 16-lane row's sum in its lane 15, row broadcasts carry rows 0-2 into
// lane 63.  Lanes without a source add 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_add_step(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROW_MASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROW_MASK, 0xF, false);
  return v + __hiloint2double(hi, lo);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add_step(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, false));
}
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  v = dpp_add_step<0x111, 0xF>(v);   // row_shr:1
  v = dpp_add_step<0x112, 0xF>(v);   // row_shr:2
  v = dpp_add_step<0x114, 0xF>(v);   // row_shr:4
  v = dpp_add_step<0x118, 0xF>(v);   // row_shr:8  -> lane 15 of each row: the row's sum
  v = dpp_add_step<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
  v = dpp_add_step<0x143, 0xC>(v);   // row_bcast:31 into rows 2 and 3 -> lane 63: the total
  if constexpr (sizeof(T) == 8) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(v), 63);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(v), 63);
    return __hiloint2double(hi, lo);
  } else {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
  }
}

int pair_panel_rows(int bw) { return (kPanelWaves - 1) * (kWave / panel_split(bw)); }

template <typename T, int S>
__global__ void __launch_bounds__(kPanelThreads, 1) pair_panel_kernel(PanelArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int R = (kPanelWaves - 1) * (kWave / S);
  constexpr int RW = kWave / S;                    // rows per wave
  constexpr int NG = KC / 16;                      // g registers
  constexpr int TOT = KC * S;                      // slots a row can hold
  constexpr int NLQ = TOT / kWave;                 // slot loads per lane and row
  static_assert(NG == 4, "four g registers");
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const bool rowwave = wave != 0;                  // wave 0: exchange only
  const int w = blockIdx.x;
  const int bw = a.bw, n = a.n, j = a.j;
  const int nt = bw / 2;                           // steps of this block
  const int part = lane / RW;
  const int rloc = (wave - 1) * RW + lane % RW;
  const int64_t lda = a.lda, ldw = a.ldw;
  const T* A = static_cast<const T*>(a.A);
  T* G = static_cast<T*>(a.G);

  unsigned char* wl = smem + (size_t)wave * pair_wave_lds_bytes(TOT, (int)sizeof(T));
  T* bufB = reinterpret_cast<T*>(wl);              // slots of the pivot row
  T* bufQ = bufB + TOT;                            // slots of row q
  T* gcol = bufQ + TOT;                            // g of the current column, by slot
  __shared__ int s_p, s_posw, s_abort;
  __shared__ double red_v[kPanelWaves];
  __shared__ uint64_t red_k[kPanelWaves];
  __shared__ T s_alpha;

  const int row0 = j + 1 + w * R;
  const int rows_here = max(0, min(R, n - row0));
  const bool my_row = rowwave && rloc < rows_here;
  const int pos = row0 + rloc;
  int lp = pos;

  T L[KC];
#pragma unroll
  for (int c = 0; c < KC; ++c) L[c] = T(0);
  for (int s = lane; s < TOT; s += kWave) gcol[s] = T(0);
  if (tid == 0) s_abort = 0;
  // Positions that received a displaced row, in registers: entry e (lane e,
  // or lane e-64 of the second pair) = (position, block-start index).  The
  // last entry with position x names the row at x; a position never listed
  // holds the row of its own block-start index.  At most nt <= 128 entries.
  int mpos0 = -1, midx0 = 0, mpos1 = -1, midx1 = 0, nmoved = 0;
  auto lookup = [&](int x) -> int {
    const unsigned long long b1 = __ballot(lane + kWave < nmoved && mpos1 == x);
    const unsigned long long b0 = __ballot(lane < nmoved && mpos0 == x);
    if (b1) return __builtin_amdgcn_readlane(midx1, 63 - __clzll(b1));
    if (b0) return __builtin_amdgcn_readlane(midx0, 63 - __clzll(b0));
    return x;
  };
  int qk = j;                                      // block-start index of the row at position k
  T l_prev = T(0), w_prev = T(0);                  // this row's slots 2t-2, 2t-1
  T gc0 = T(0), gc1 = T(0);                        // g of column k at slots 2t-2, 2t-1
  // column j: S(pos, j) = A(pos, j), every held row is below j
  T cv = T(0);
  {
    T lv = T(0);
    if (my_row && part == 0) lv = A[(int64_t)pos + (int64_t)j * lda];
    cv = part_sum<S>(lv);
  }
  __syncthreads();

  for (int t = 0; t < nt; ++t) {
    const int k = j + 2 * t;
    const int ns = 2 * t;                          // slots filled so far
    const int umax = ns > 0 ? ns - 1 : 0;
    const bool last = t + 1 == nt;
    const bool active = my_row && lp >= k + 1;

    // ---- pivot candidate of column k ----
    {
      double av = -1.0;
      if (active) {
        const double m = (double)fabs(cv);
        if (m == m) av = m;
      }
      double bv;
      int bi;
      const int src = wave_first_max(av, active ? lp : INT32_MAX, bv, bi);
      int wpos = 0, wsg = 0;
      if (src >= 0) {
        wpos = __builtin_amdgcn_readlane(pos, src);
        wsg = __builtin_amdgcn_readlane(cv < T(0) ? 1 : 0, src);
      }
      if (lane == 0) {
        red_v[wave] = src >= 0 ? bv : -1.0;
        red_k[wave] = ((uint64_t)(uint32_t)bi << 32) | ((uint64_t)wpos << 1) | (uint64_t)wsg;
      }
    }
    const int stamp = k / 2 + 1;
    exchange_publish(a, stamp, wave, lane, w, red_v, red_k);

    // ---- column k+2 for the row qq at position k+2 (independent of the
    //      pivot unless it comes from k+2): its slots, S(pos, qq), cA = column
    //      k at row qq, and asum = S(pos, qq) + the old slots' part of the
    //      refresh, for every row now at a position >= k+1 ----
    const int no = ns >= 2 ? ns - 2 : 0;           // slots visible before the agreement
    const int uo = no > 0 ? no - 1 : 0;
    T apart = T(0), cA = T(0);
    auto spec = [&](int qq) {
      T lvA = T(0), lsgA = T(1);
      if (my_row && part == 0 && lp >= k + 1 && pos != qq) {
        lvA = A[(int64_t)max(pos, qq) + (int64_t)min(pos, qq) * lda];
        lsgA = pos > qq ? T(1) : T(-1);
      }
      T lrQ[NLQ];
      const T* growQ = G + (int64_t)(qq - (j + 1)) * bw;
#pragma unroll
      for (int u = 0; u < NLQ; ++u) lrQ[u] = ld_coh_t(&growQ[min(u * kWave + lane, uo)]);
      T sA = A[(int64_t)max(qq, qk) + (int64_t)min(qq, qk) * lda];
      if (qq < qk) sA = -sA;
#pragma unroll
      for (int u = 0; u < NLQ; ++u) {
        const int s = u * kWave + lane;
        if (s < no) bufQ[s] = lrQ[u];
      }
      wave_lds_sync();
      T dA = T(0);
#pragma unroll
      for (int u = 0; u < NLQ; ++u) {
        const int s = u * kWave + lane;
        if (s < no) dA = fma(bufQ[s], gcol[s], dA);
      }
      cA = sA + wave_sum(dA);
      T grA[NG];
      const int c16 = lane & 15;
#pragma unroll
      for (int kk = 0; kk < NG; ++kk) grA[kk] = g_of(bufQ, (16 * kk + c16) * S + part, no);
      T accA[4] = {T(0), T(0), T(0), T(0)};
      if (0 * 16 * S < no) refresh16<0>(accA, grA[0], L);
      if (1 * 16 * S < no) refresh16<1>(accA, grA[1], L);
      if (2 * 16 * S < no) refresh16<2>(accA, grA[2], L);
      if (3 * 16 * S < no) refresh16<3>(accA, grA[3], L);
      apart = fma(lsgA, lvA, (accA[0] + accA[1]) + (accA[2] + accA[3]));
    };
    const int qs = last ? 0 : lookup(k + 2);       // row at position k+2 before the exchange
    const int displaced = lookup(k + 1);           // row at position k+1 before the exchange
    if (!last && rowwave) spec(qs);

    exchange_collect<T>(a, stamp, k, wave, lane, s_p, s_posw, s_alpha, s_abort);
    if (s_abort) return;
    const int p = s_p;
    const int posw = s_posw;
    const T alph = s_alpha;
    // the row at position k+2 after the exchange: the displaced row when the
    // pivot came from k+2, else the same as before
    const int q = last ? 0 : (p == k + 2 ? displaced : qs);

    // ---- the pivot row's part, issued first: S(pos, posw) for every row at
    //      a position >= k+1 but the pivot (a superset of the rows that get a
    //      w), its slots, S(q, posw) and row q's slots 2t-2, 2t-1 ----
    T lvB = T(0), lsgB = T(1);
    T lrB[NLQ];
    T sB = T(0), qn0 = T(0), qn1 = T(0);
    if (rowwave) {
      if (my_row && part == 0 && lp >= k + 1 && pos != posw) {
        lvB = A[(int64_t)max(pos, posw) + (int64_t)min(pos, posw) * lda];
        lsgB = pos > posw ? T(1) : T(-1);
      }
      const T* growB = G + (int64_t)(posw - (j + 1)) * bw;
#pragma unroll
      for (int u = 0; u < NLQ; ++u) lrB[u] = ld_coh_t(&growB[min(u * kWave + lane, umax)]);
      if (!last) {
        sB = A[(int64_t)max(q, posw) + (int64_t)min(q, posw) * lda];
        if (q < posw) sB = -sB;
        if (ns >= 2) {
          const T* growQ = G + (int64_t)(q - (j + 1)) * bw;
          qn0 = ld_coh_t(&growQ[ns - 2]);
          qn1 = ld_coh_t(&growQ[ns - 1]);
        }
      }
    }

    // ---- exchange positions k+1 and p ----
    if (p != k + 1) {
      if (lane == nmoved) { mpos0 = p; midx0 = displaced; }
      if (lane + kWave == nmoved) { mpos1 = p; midx1 = displaced; }
      ++nmoved;
      if (my_row) {
        if (lp == p) lp = k + 1;
        else if (lp == k + 1) lp = p;
      }
    }
    if (!last && q != qs && rowwave) spec(q);      // the pivot came from position k+2
    const bool next2 = my_row && lp >= k + 2;      // rows that get l and w
    const bool next3 = !last && my_row && lp >= k + 3;   // rows of the next column

    T l = T(0), wv_keep = T(0), gq0 = T(0), gq1 = T(0);
    if (rowwave) {
    // ---- multiplier of column k into slot 2t ----
    if (next2) l = (alph != T(0)) ? cv / alph : T(0);
    {
      const int c = ns / S;
      const bool on = next2 && part == ns % S;
      const T v = l;
      if constexpr (S >= 2) {
        set_slot<T>(L, c, on, v);
      } else {
        LTLT_SET_GROUP(0) LTLT_SET_GROUP(16) LTLT_SET_GROUP(32) LTLT_SET_GROUP(48)
      }
    }
#pragma unroll
    for (int u = 0; u < NLQ; ++u) {
      const int s = u * kWave + lane;
      if (s < ns) bufB[s] = lrB[u];
    }
    if (!last && ns >= 2 && lane == 0) { bufQ[ns - 2] = qn0; bufQ[ns - 1] = qn1; }
    wave_lds_sync();
    // the previous step's terms: column k at row q (cA) and column k+2 (asum)
    T asum = T(0);
    if (!last) {
      cA = fma(qn1, gc1, fma(qn0, gc0, cA));
      asum = fma(w_prev, -qn0, fma(l_prev, qn1, part_sum<S>(apart)));
    }

    // ---- g of column k+1 (registers), the newest slots of row q ----
    T grB[NG];
    {
      const int c16 = lane & 15;
#pragma unroll
      for (int kk = 0; kk < NG; ++kk) grB[kk] = g_of(bufB, (16 * kk + c16) * S + part, ns);
    }
    if (!last) {
      T dB = T(0);
#pragma unroll
      for (int u = 0; u < NLQ; ++u) {
        const int s = u * kWave + lane;
        if (s < ns) dB = fma(bufQ[s], g_of(bufB, s, ns), dB);
      }
      gq0 = sB + wave_sum(dB);                     // column k+1 at row q
      gq1 = -((alph != T(0)) ? cA / alph : T(0));  // -(column k at row q) / alpha_k
    }

    // ---- column k+1 (w, slot 2t+1) and column k+2 ----
    {
      T accB[4] = {T(0), T(0), T(0), T(0)};
      if (0 * 16 * S < ns) refresh16<0>(accB, grB[0], L);
      if (1 * 16 * S < ns) refresh16<1>(accB, grB[1], L);
      if (2 * 16 * S < ns) refresh16<2>(accB, grB[2], L);
      if (3 * 16 * S < ns) refresh16<3>(accB, grB[3], L);
      const T wsum = part_sum<S>(fma(lsgB, lvB, (accB[0] + accB[1]) + (accB[2] + accB[3])));
      const T wv = next2 ? wsum : T(0);
      wv_keep = wv;
      cv = next3 ? fma(wv, gq1, fma(l, gq0, asum)) : T(0);
      {
        const int c = (ns + 1) / S;
        const bool on = next2 && part == (ns + 1) % S;
        const T v = wv;
        if constexpr (S >= 2) {
          set_slot<T>(L, c, on, v);
        } else {
          LTLT_SET_GROUP(0) LTLT_SET_GROUP(16) LTLT_SET_GROUP(32) LTLT_SET_GROUP(48)
        }
      }
      int ro = pos - (j + 1);
      asm volatile("" : "+v"(ro));
      if (next2 && part == ns % S) st_coh_t(&G[(int64_t)ro * bw + ns], l);
      if (next2 && part == (ns + 1) % S) st_coh_t(&G[(int64_t)ro * bw + ns + 1], wv);
    }
    // g of column k+2 by slot, for the next step's cA
    if (!last) {
#pragma unroll
      for (int u = 0; u < NLQ; ++u) {
        const int s = u * kWave + lane;
        gcol[s] = s < ns ? g_of(bufQ, s, ns) : (s == ns ? gq0 : (s == ns + 1 ? gq1 : T(0)));
      }
    }
    }
    if (tid == 0 && w == 0) {
      a.ipiv[k + 1] = p;
      static_cast<T*>(a.alpha)[t] = alph;
    }
    l_prev = l;
    w_prev = next2 ? wv_keep : T(0);
    gc0 = gq0;
    gc1 = gq1;
    qk = q;
    wave_lds_sync();
  }

#undef LTLT_SET_GROUP

  // ---- outputs for the trailing rows (positions >= j+bw): Lx in slot order,
  //      Bt = Lx J^T (column s+1 = -slot s for even s, column s-1 = slot s
  //      for odd s) ----
  T* PO = static_cast<T*>(a.PO);
  T* Bm = static_cast<T*>(a.Bm);
  const int tr0 = j + bw;
  if (my_row && lp >= tr0) {
    const int64_t ro = lp - tr0;
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int s = c * S + part;
      if (s < bw) {
        PO[ro + (int64_t)s * ldw] = L[c];
        if (s & 1) Bm[ro + (int64_t)(s - 1) * ldw] = L[c];
        else Bm[ro + (int64_t)(s + 1) * ldw] = -L[c];
      }
    }
  }
  if (my_row && part == 0) a.perm[lp] = pos;
}

template <typename T, int S>
hipError_t launch_pair_panel_s(const PanelArgs& a, size_t lds, hipStream_t st) {
  return launch_resident_grid(pair_panel_kernel<T, S>, (unsigned)a.P, kPanelThreads, lds, st, a);
}

template <typename T>
hipError_t launch_pair_panel(const PanelArgs& a, size_t lds, hipStream_t st) {
  if (a.P > kMaxPanelRecords || a.P > a.nrec || a.R != pair_panel_rows(a.bw) || (a.bw & 1))
    return hipErrorInvalidValue;
  switch (panel_split(a.bw)) {
    case 1: return launch_pair_panel_s<T, 1>(a, lds, st);
    case 2: return launch_pair_panel_s<T, 2>(a, lds, st);
    case 4: return launch_pair_panel_s<T, 4>(a, lds, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int S>
int pair_max_blocks_s(size_t lds) {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)pair_panel_kernel<T, S>, kPanelThreads,
                                                   lds) != hipSuccess)
    return 0;
  return per_cu * cus;
}

template <typename T>
int pair_max_blocks(int bw, size_t lds) {
  int cap;
  switch (panel_split(bw)) {
    case 1: cap = pair_max_blocks_s<T, 1>(lds); break;
    case 2: cap = pair_max_blocks_s<T, 2>(lds); break;
    case 4: cap = pair_max_blocks_s<T, 4>(lds); break;
    default: return 0;
  }
  return cap < kMaxPanelRecords ? cap : kMaxPanelRecords;
}

// alpha_k of the block's steps into A(k+1, k) (after the block's trailing
// update, which may still read the block's original entries); NaN when a
// wait of this call gave up (status[0] raised).
template <typename T>
__global__ void pair_commit_kernel(T* A, int64_t lda, int j, int nt, const T* alpha, const int* status) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < nt) A[(int64_t)(j + 2 * t + 1) + (int64_t)(j + 2 * t) * lda] = status[0] != 0 ? T(NAN) : alpha[t];
}

template <typename T>
hipError_t launch_pair_commit(T* A, int64_t lda, int j, int nt, const T* alpha, const int* status, hipStream_t s) {
  if (nt <= 0) return hipSuccess;
  hipLaunchKernelGGL(pair_commit_kernel<T>, dim3((nt + 255) / 256), dim3(256), 0, s, A, lda, j, nt, alpha, status);
  return hipGetLastError();
}

template size_t pair_lds_bytes<double>(int, int);
template size_t pair_lds_bytes<float>(int, int);
template int pair_max_blocks<double>(int, size_t);
template int pair_max_blocks<float>(int, size_t);
template hipError_t launch_pair_panel<double>(const PanelArgs&, size_t, hipStream_t);
template hipError_t launch_pair_panel<float>(const PanelArgs&, size_t, hipStream_t);
template hipError_t launch_pair_commit<double>(double*, int64_t, int, int, const double*, const int*, hipStream_t);
template hipError_t launch_pair_commit<float>(float*, int64_t, int, int, const float*, const int*, hipStream_t);

}  // namespace ltlt
