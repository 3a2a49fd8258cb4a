// Panel kernel: the column steps k = j .. j+bw-1 of one block of the pivoted
// skew-symmetric reduction P X P^T = L T L^T, run by P co-resident
// workgroups that together hold every row of the block (positions j+1..n-1).
//
// Thread layout: 512 threads (8 waves, two per SIMD) per workgroup, S lanes
// per row (S = 1, 2, 4 for blocks of up to 64, 128, 256 steps): the wave is
// split into S parts of 64/S consecutive lanes, part p holds the steps u with
// u % S == p of the same 64/S rows, so R = 512/S rows per workgroup and every
// 16-lane row of the wave belongs to one part.  A lane keeps its row's
// multipliers in registers: L[c] = multiplier of step j + c*S + p, c < 64.
//
// Rows never move between lanes.  Lane rows are the rows of the block-start
// matrix (block-start index `pos`, fixed); an exchange of positions k+1 and p
// only swaps the logical positions `lp` of the two lanes that hold them.  The
// row at position k+1 after the exchange is final from then on; the other one
// keeps its multipliers and column value where they are.
//
// A copy of the multipliers also lives in global memory, indexed by the
// block-start index, G[pos - (j+1)][u], row by row (stride bw) so that the
// pivot row's multipliers of the earlier steps, which every lane needs after
// each agreement, are one contiguous run of a few cache lines; it is the only
// data that crosses workgroups besides the exchange records.
//
// Column refresh.  The trailing matrix is stored as it was at block start
// (strict lower triangle), so the current column k is the stored column of
// the block-start index of position k, plus the not-yet-applied updates of
// steps j .. k-2.  Step s updates X(i,c) += l_i v_c - v_i l_c with v the
// column s+1 at step s, and v = alpha_{s+1} * L(:, s+2) below row s+2
// (column s+1 is the one step s+1 eliminates).  Summed over the block this is
// Lp Tx Lp^T with Tx skew tridiagonal, Tx[u,u+1] = alpha_{j+u+1}; the
// refresh of column k therefore needs only row k of Lp:
//   cv[i] = S(pos[i], pos[k]) + sum_{u<t} g_u Lp[u][i],
//   g_u = alpha_{j+u+1} Lrow[u+1] [u <= t-2] - alpha_{j+u} Lrow[u-1] [u >= 1],
//   Lrow[w] = Lp[w][k] (w <= t-2), Lrow[t-1] = 1 (unit diagonal of L),
// with S(a, b) = A(a, b) for a > b and -A(b, a) for a < b.
// The g coefficients live in registers in "row broadcast" layout: register
// gr[k], lane l holds g of slot 16k + (l % 16) of the lane's step slice, the
// same in each 16-lane row of that slice, and the refresh multiplies slot c
// by lane c % 16 of its own row through a DPP row broadcast, so no lane reads
// g from LDS.
//
// Exchange per step (one grid-wide round, no counters, no fences): every
// workgroup merges the candidates of its waves and publishes the result as
// one record of two self-validating 64-bit words (each carries the step
// stamp); records sit 256 bytes apart.  Wave 0 of every workgroup polls all
// records until each carries the current stamp and reduces them (largest
// magnitude, then smallest position: the first maximum in position order), so
// all workgroups agree on the pivot p.  A barrier hands the result to the
// other waves; from there each wave works alone: it loads the pivot row's
// multipliers from G into its own LDS area, forms the g coefficients of the
// next step and refreshes its rows.  Multipliers written to G at step k are
// read no earlier than step k+1; every wave waits for its own earlier stores
// to complete before the barrier that precedes the publication of the next
// record, so any record that validates implies that the winning row's
// multipliers are visible.
//
// After the last step the carry column (column j+bw, refreshed) is formed and
// every lane writes its row of the block's outputs at its final position:
// Lx = [Lp, carry] (rows >= j+bw+1) feeds the trailing update as one
// rank-(bw+1) product with Bt = Lx Tx^T; the rows inside the block and the
// alphas are committed into A after that update.

#include "ltlt_device.h"
#include "ltlt_exchange.h"
#include "ltlt_internal.h"

namespace ltlt {

int panel_rows(int bw) { return kPanelThreads / panel_split(bw); }

// LDS: per wave, the alpha history (TOT + 1) and the pivot row's multipliers
// padded by one entry in front (TOT + 2), TOT = steps a row can hold.
__host__ __device__ constexpr int panel_wave_lds_elems(int tot) { return (tot + 1) + (tot + 2); }
template <typename T>
size_t panel_lds_bytes(int bw, int /*R*/) {
  return (size_t)kPanelWaves * panel_wave_lds_elems(KC * panel_split(bw)) * sizeof(T);
}

template <typename T, int S>
__global__ void __launch_bounds__(kPanelThreads, 1) panel_kernel(PanelArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int R = kPanelThreads / S;
  constexpr int RW = kWave / S;                    // rows per wave
  constexpr int NG = KC / 16;                      // g registers
  constexpr int TOT = KC * S;                      // steps a row can hold
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int w = blockIdx.x;
  const int bw = a.bw, n = a.n, j = a.j;
  const int part = lane / RW;                      // step slice of this lane
  const int rloc = wave * RW + lane % RW;
  const int64_t lda = a.lda, ldw = a.ldw;
  const T* A = static_cast<const T*>(a.A);
  T* G = static_cast<T*>(a.G);

  T* my_alpha = reinterpret_cast<T*>(smem) + wave * panel_wave_lds_elems(TOT);   // alpha_{j+u}
  T* my_lrowp = my_alpha + (TOT + 1);              // my_lrowp[u + 1] = Lrow[u]
  // the agreement's results, read back together in one LDS round trip
  struct __align__(16) XRes { int p, posw, abort, pad; };
  __shared__ XRes s_x;
  __shared__ double red_v[kPanelWaves];
  __shared__ uint64_t red_k[kPanelWaves];
  __shared__ T s_alpha;

  const int row0 = j + 1 + w * R;                 // first block-start index held
  const int rows_here = max(0, min(R, n - row0));
  const bool my_row = rloc < rows_here;
  const int pos = row0 + rloc;                     // block-start index of this lane's row
  int lp = pos;                                    // its current position

  T L[KC], gr[NG];
#pragma unroll
  for (int c = 0; c < KC; ++c) L[c] = T(0);
#pragma unroll
  for (int k = 0; k < NG; ++k) gr[k] = T(0);
  if (lane == 0) my_lrowp[0] = T(0);               // Lrow[-1]: only ever multiplied, kept finite
  T cv = T(0);
  if (tid == 0) s_x.abort = 0;
  // stored column value of this row and its sign (S(a,b) = -A(b,a) above the
  // diagonal); the sign is applied in the refresh so that no code waits for
  // the load before then.  First column: index j, rows >= j+1 (lower part).
  T lv = T(0), lsg = T(1);
  if (my_row && part == 0) lv = A[(int64_t)pos + (int64_t)j * lda];
  __syncthreads();

  for (int t = 0; t <= bw; ++t) {
    const int k = j + t;
    // ---- column refresh: cv = S(pos, q) + sum_u g_u L_u over rows at >= k+1 ----
    const bool active = my_row && lp >= k + 1;
    {
      T acc[4] = {T(0), T(0), T(0), T(0)};
      static_assert(NG == 4, "four g registers");
      if (0 * 16 * S < t) refresh16<0>(acc, gr[0], L);
      if (1 * 16 * S < t) refresh16<1>(acc, gr[1], L);
      if (2 * 16 * S < t) refresh16<2>(acc, gr[2], L);
      if (3 * 16 * S < t) refresh16<3>(acc, gr[3], L);
      T sum = fma(lsg, lv, (acc[0] + acc[1]) + (acc[2] + acc[3]));   // lv is nonzero in part 0 only
      sum = part_sum<S>(sum);
      if (active) cv = sum;
    }
    if (t == bw) break;                           // carry column formed

    // ---- this wave's pivot candidate: (|cv|, position), first maximum ----
    {
      double av = -1.0;
      if (active) {
        const double m = (double)fabs(cv);
        if (m == m) av = m;                        // NaN is never a candidate
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
    exchange_pivot<T>(a, k + 1, k, wave, lane, w, red_v, red_k, s_x.p, s_x.posw, s_alpha, s_x.abort);
    const int4 xr = *reinterpret_cast<const int4*>(&s_x);
    const T alph = s_alpha;
    asm volatile("" ::"v"(xr.x), "v"(xr.y), "v"(xr.z), "v"(alph));   // both reads issued before the branch
    if (xr.z) return;
    const int p = xr.x;
    const int posw = xr.y;                         // block-start index of the pivot row

    // ---- exchange positions k+1 and p (logical only) ----
    if (my_row && p != k + 1) {
      if (lp == p) lp = k + 1;
      else if (lp == k + 1) lp = p;
    }
    const bool next = my_row && lp >= k + 2;      // rows still to be eliminated

    // ---- one round of loads: pivot row multipliers, then the next stored
    //      column.  Every lane issues the same loads (multiplier addresses
    //      clamped to steps < t, the stored column's to A(j+1, j) where it
    //      is not needed), so the in-order memory counter lets g be formed
    //      from the multipliers while the stored column, a strided row read
    //      for rows above the pivot, is still in flight. ----
    constexpr int NLQ = TOT / kWave;              // multiplier loads per lane
    T lr[NLQ];
    {
      const T* grow = G + (int64_t)(posw - (j + 1)) * bw;
      const int umax = t > 0 ? t - 1 : 0;
#pragma unroll
      for (int q = 0; q < NLQ; ++q) lr[q] = ld_coh_t(&grow[min(q * kWave + lane, umax)]);
    }
    // S(pos, posw) = +A(pos, posw) below the diagonal, -A(posw, pos) above:
    // element (max, min) of the stored triangle
    const bool ldv = next && part == 0;
    const int64_t lvi = ldv ? (int64_t)max(pos, posw) + (int64_t)min(pos, posw) * lda : (int64_t)(j + 1) + (int64_t)j * lda;
    const T lvn = A[lvi];
    __builtin_amdgcn_sched_barrier(0);             // keep the load ahead of the work below

    // ---- multiplier of step k; the pivot row's multipliers into LDS before
    //      the slot write below (a jump), so their wait counts exactly.
    //      Entries past step t hold clamped copies that g discards; lane 0
    //      then writes the unit entry over entry t+1. ----
    T l = T(0);
    if (next) l = (alph != T(0)) ? cv / alph : T(0);
#pragma unroll
    for (int q = 0; q < NLQ; ++q) my_lrowp[q * kWave + lane + 1] = lr[q];
    if (lane == 0) { my_alpha[t] = alph; my_lrowp[t + 1] = T(1); }   // Lrow[t] = 1: unit diagonal
    {
      const int c = t / S;
      const bool on = next && part == t % S;
      const T v = l;
      static_assert(KC == 64, "four groups of 16 slots");
      if constexpr (S >= 2) {
        set_slot<T>(L, c, on, v);
      } else {
        LTLT_SET_GROUP(0) LTLT_SET_GROUP(16) LTLT_SET_GROUP(32) LTLT_SET_GROUP(48)
      }
    }

    // ---- g coefficients for step k+1 (t+1 terms), row broadcast layout ----
    wave_lds_sync();
    {
      const int c = lane & 15;
      // every group's reads issued at once (in bounds for any u < TOT; the
      // entries past step t are discarded by the selects, never multiplied
      // into a kept value), rather than one group's round trip after another
#pragma unroll
      for (int kk = 0; kk < NG; ++kk) {
        const int u = (16 * kk + c) * S + part;    // < TOT
        const T a0 = my_alpha[u], a1 = my_alpha[u + 1];
        const T lm = my_lrowp[u], l1 = my_lrowp[u + 2];
        const T up = (u <= t - 1) ? a1 * l1 : T(0);
        const T g = (u >= 1) ? up - a0 * lm : up;
        gr[kk] = (u <= t) ? g : T(0);
      }
    }
    // the stored column is taken before the stores below are issued, so its
    // wait does not include their acknowledgement
    if (ldv) {
      lv = lvn;
      lsg = pos > posw ? T(1) : T(-1);
    }
    asm volatile("" : "+v"(lv), "+v"(lsg) : : "memory");
    {
      // recompute the row offset here instead of keeping a 64-bit pointer
      // live across the step loop (the kernel runs at the register limit)
      int ro = pos - (j + 1);
      asm volatile("" : "+v"(ro));
      if (next && part == t % S) st_coh_t(&G[(int64_t)ro * bw + t], l);
    }
    if (tid == 0 && w == 0) a.ipiv[k + 1] = p;
    wave_lds_sync();
  }

#undef LTLT_SET_GROUP

  // ---- outputs, by final position, straight from registers.  Rows at
  //      positions j+1 .. j+bw hold the multipliers of the steps before they
  //      became final (zeros after); trailing rows hold all of them and the
  //      carry. ----
  T* PO = static_cast<T*>(a.PO);
  T* Bm = static_cast<T*>(a.Bm);
  const int tr0 = j + bw + 1;                      // first trailing position
  const bool trailing = my_row && lp >= tr0;
  const T carry = trailing ? cv : T(0);
  const T* alpha = my_alpha;                       // alpha_{j+u}, u < bw
  if (my_row) {
    const int64_t ro = lp - (j + 1);
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const int u = c * S + part;
      if (u < bw) PO[ro + (int64_t)u * ldw] = L[c];
    }
    if (part == 0) PO[ro + (int64_t)bw * ldw] = carry;
  }
  // Bt = Lx Tx^T: column u = a_u Lx_{u+1} - a_{u-1} Lx_{u-1},
  // a_u = alpha_{j+u+1} (u <= bw-2), a_{bw-1} = 1, Lx_bw = carry.
  // Step u = c*S + part; step u+1 lives in the next part (lane + RW), slot c
  // (slot c+1 when this is the last part), step u-1 in the previous part
  // (lane - RW), slot c (slot c-1 when this is part 0).  The owner lane hands
  // out the slot its requester needs.
  const int up_src = (lane + RW) % kWave, dn_src = (lane + kWave - RW) % kWave;
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    const T give_up = (part == 0 && c + 1 < KC) ? L[c + 1 < KC ? c + 1 : c] : (part == 0 ? T(0) : L[c]);
    const T give_dn = (part == S - 1) ? (c >= 1 ? L[c >= 1 ? c - 1 : 0] : T(0)) : L[c];
    const T xp0 = S == 1 ? give_up : __shfl(give_up, up_src, kWave);
    const T xm = S == 1 ? give_dn : __shfl(give_dn, dn_src, kWave);
    const int u = c * S + part;
    if (trailing && u <= bw) {
      T v = T(0);
      if (u <= bw - 1) {
        const T au = (u <= bw - 2) ? alpha[u + 1] : T(1);
        v += au * (u + 1 == bw ? carry : xp0);
      }
      if (u >= 1) {
        const T am = (u - 1 <= bw - 2) ? alpha[u] : T(1);
        v -= am * xm;
      }
      Bm[(int64_t)(lp - tr0) + (int64_t)u * ldw] = v;
    }
  }
  // column bw when it lies past the slots (bw == TOT): -Lx_{bw-1}, step TOT-1
  // is slot KC-1 of the last part
  {
    const T last = __shfl(L[KC - 1], (lane % RW) + (S - 1) * RW, kWave);
    if (trailing && bw == TOT && part == 0) Bm[(int64_t)(lp - tr0) + (int64_t)bw * ldw] = -last;
  }
  if (my_row && part == 0) a.perm[lp] = pos;
  if (w == 0 && wave == 0) {
    T* al = static_cast<T*>(a.alpha);
    for (int u = lane; u < bw; u += kWave) al[u] = alpha[u];
  }
}

template <typename T, int S>
hipError_t launch_panel_s(const PanelArgs& a, size_t lds, hipStream_t st) {
  return launch_resident_grid(panel_kernel<T, S>, (unsigned)a.P, kPanelThreads, lds, st, a);
}

template <typename T>
hipError_t launch_panel(const PanelArgs& a, size_t lds, hipStream_t st) {
  if (a.P > kMaxPanelRecords || a.P > a.nrec || a.R != panel_rows(a.bw)) return hipErrorInvalidValue;
  switch (panel_split(a.bw)) {
    case 1: return launch_panel_s<T, 1>(a, lds, st);
    case 2: return launch_panel_s<T, 2>(a, lds, st);
    case 4: return launch_panel_s<T, 4>(a, lds, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int S>
int panel_max_blocks_s(size_t lds) {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)panel_kernel<T, S>, kPanelThreads, lds) !=
      hipSuccess)
    return 0;
  return per_cu * cus;
}

// Co-resident workgroups for a block of width bw (capped by the records one
// poll covers).
template <typename T>
int panel_max_blocks(int bw, size_t lds) {
  int cap;
  switch (panel_split(bw)) {
    case 1: cap = panel_max_blocks_s<T, 1>(lds); break;
    case 2: cap = panel_max_blocks_s<T, 2>(lds); break;
    case 4: cap = panel_max_blocks_s<T, 4>(lds); break;
    default: return 0;
  }
  return cap < kMaxPanelRecords ? cap : kMaxPanelRecords;
}

// Exchange records start with stamps that can never validate: word B stamp 0,
// and word A epoch opposite to that of the first stamp using the slot
// (slot 1 first holds s = 1, epoch 0; slot 0 first holds s = 2, epoch 1).
__global__ void rec_init_kernel(uint64_t* rec, int nrec) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 2 * kRecStride * nrec) return;
  const int slot = i / (kRecStride * nrec);
  const int word = i % kRecStride;
  rec[i] = (word == 0 && slot == 1) ? (1ull << 63) : 0ull;
}

hipError_t launch_rec_init(uint64_t* rec, int nrec_per_slot, hipStream_t s) {
  const int tot = 2 * kRecStride * nrec_per_slot;
  hipLaunchKernelGGL(rec_init_kernel, dim3((tot + 255) / 256), dim3(256), 0, s, rec, nrec_per_slot);
  return hipGetLastError();
}

template int panel_max_blocks<double>(int, size_t);
template int panel_max_blocks<float>(int, size_t);
template size_t panel_lds_bytes<double>(int, int);
template size_t panel_lds_bytes<float>(int, int);
template hipError_t launch_panel<double>(const PanelArgs&, size_t, hipStream_t);
template hipError_t launch_panel<float>(const PanelArgs&, size_t, hipStream_t);

}  // namespace ltlt
