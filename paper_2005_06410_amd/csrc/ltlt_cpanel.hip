// Complex panel kernel: the column steps k = j .. j+bw-1 of one block of the
// pivoted reduction P X P^T = L T L^T of a complex skew-symmetric X
// (X^T = -X, a transpose without conjugation), held as two real planes.
//
// The algorithm, thread layout, exchange and output order are those of the
// real panel (ltlt_panel.hip); what changes:
//  * a lane keeps KCC = 32 complex multipliers of its row (real and
//    imaginary parts in registers, 128 VGPRs in fp64, as the real panel's 64
//    real slots), so S = 1, 2, 4 lanes share a row for blocks of up to 32,
//    64, 128 steps;
//  * the refresh cv = S(pos, q) + sum_u g_u L_u takes four DPP row-broadcast
//    FMA passes per 16 slots: Re += gr Lr + (-gi) Li, Im += gr Li + gi Lr;
//  * the pivot search compares |re| + |im| (the magnitude of the BLAS complex
//    i_amax); the exchange record carries that magnitude, so the pivot value
//    itself goes through a per-row slot V[idx - j - 1] that each wave's
//    candidate lane writes before its workgroup publishes, and every wave
//    loads the winner's V in the same load round as the pivot row's
//    multipliers (a validated record implies the slot is visible, as for G);
//  * multipliers l = cv / alpha by Smith's quotient;
//  * outputs: LL = [Lr | Li | Lr] and the two right operands
//    BtA = [Btr | -Bti], BtB = [Btr | Bti] (Bt = Lx Tx^T), so that each
//    plane's trailing update is one real product of depth 2(bw+1).

#include "ltlt_device.h"
#include "ltlt_exchange.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int KCC = 32;                          // complex multiplier slots per lane

inline int cpanel_split(int bw) { return bw <= KCC ? 1 : (bw <= 2 * KCC ? 2 : 4); }
int cpanel_rows(int bw) { return kPanelThreads / cpanel_split(bw); }

// LDS per wave: alpha history (TOT + 1) and pivot-row multipliers padded by
// one entry in front (TOT + 2), each as real and imaginary arrays.
__host__ __device__ constexpr int cpanel_wave_lds_elems(int tot) { return 2 * ((tot + 1) + (tot + 2)); }
template <typename T>
size_t cpanel_lds_bytes(int bw) {
  return (size_t)kPanelWaves * cpanel_wave_lds_elems(KCC * cpanel_split(bw)) * sizeof(T);
}

// Smith's quotient x / y (y != 0).
template <typename T>
__device__ __forceinline__ void cdiv(T xr, T xi, T yr, T yi, T& zr, T& zi) {
  if (fabs(yr) >= fabs(yi)) {
    const T r = yi / yr, den = yr + yi * r;
    zr = (xr + xi * r) / den;
    zi = (xi - xr * r) / den;
  } else {
    const T r = yr / yi, den = yi + yr * r;
    zr = (xr * r + xi) / den;
    zi = (xi * r - xr) / den;
  }
}

// Lr[c] = vr, Li[c] = vi where `on`, for a wave-uniform slot c (static
// register indices: uniform branch on the group of 16, selects inside).  The
// two- and four-lane-per-row panels use cset_slot instead: a uniform jump to
// the one slot.
#define LTLT_CSET_GROUP(G0)                                                         \
  if ((c >> 4) == (G0) / 16) {                                                     \
    _Pragma("unroll") for (int i = 0; i < 16; ++i) {                               \
      Lr[(G0) + i] = (on && c == (G0) + i) ? vr : Lr[(G0) + i];                    \
      Li[(G0) + i] = (on && c == (G0) + i) ? vi : Li[(G0) + i];                    \
    }                                                                              \
  }

#define LTLT_CSLOT_CASE(i) \
  case (i): Lr[(i)] = on ? vr : Lr[(i)]; Li[(i)] = on ? vi : Li[(i)]; break;
#define LTLT_CSLOT_CASE4(i) \
  LTLT_CSLOT_CASE(i) LTLT_CSLOT_CASE((i) + 1) LTLT_CSLOT_CASE((i) + 2) LTLT_CSLOT_CASE((i) + 3)
template <typename T>
__device__ __forceinline__ void cset_slot(T (&Lr)[KCC], T (&Li)[KCC], int c, bool on, T vr, T vi) {
  static_assert(KCC == 32, "32 slots");
  switch (c) {
    LTLT_CSLOT_CASE4(0) LTLT_CSLOT_CASE4(4) LTLT_CSLOT_CASE4(8) LTLT_CSLOT_CASE4(12)
    LTLT_CSLOT_CASE4(16) LTLT_CSLOT_CASE4(20) LTLT_CSLOT_CASE4(24) LTLT_CSLOT_CASE4(28)
    default: break;
  }
}
#undef LTLT_CSLOT_CASE4
#undef LTLT_CSLOT_CASE

template <typename T, int S>
__global__ void __launch_bounds__(kPanelThreads, 1) cpanel_kernel(CPanelArgs ca) {
  extern __shared__ __align__(16) unsigned char smem[];
  const PanelArgs& a = ca.b;
  constexpr int R = kPanelThreads / S;
  constexpr int RW = kWave / S;                    // rows per wave
  constexpr int NG = KCC / 16;                     // g registers (per part)
  constexpr int TOT = KCC * S;                     // steps a row can hold
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int w = blockIdx.x;
  const int bw = a.bw, n = a.n, j = a.j;
  const int part = lane / RW;
  const int rloc = wave * RW + lane % RW;
  const int64_t lda = a.lda, ldw = a.ldw;
  const T* Ar = static_cast<const T*>(a.A);
  const T* Ai = static_cast<const T*>(ca.Ai);
  T* Gr = static_cast<T*>(a.G);
  T* Gi = static_cast<T*>(ca.Gi);
  T* Vr = static_cast<T*>(ca.Vr);
  T* Vi = static_cast<T*>(ca.Vi);

  T* my_ar = reinterpret_cast<T*>(smem) + wave * cpanel_wave_lds_elems(TOT);   // alpha_{j+u}
  T* my_ai = my_ar + (TOT + 1);
  T* my_lr = my_ai + (TOT + 1);                    // my_lr[u + 1] = Re Lrow[u]
  T* my_li = my_lr + (TOT + 2);
  __shared__ int s_p, s_posw, s_abort;
  __shared__ double red_v[kPanelWaves];
  __shared__ uint64_t red_k[kPanelWaves];
  __shared__ T s_none;                             // NaN: no finite candidate at this step

  const int row0 = j + 1 + w * R;
  const int rows_here = max(0, min(R, n - row0));
  const bool my_row = rloc < rows_here;
  const int pos = row0 + rloc;
  int lp = pos;

  T Lr[KCC], Li[KCC], gre[NG], gim[NG], gni[NG];
#pragma unroll
  for (int c = 0; c < KCC; ++c) { Lr[c] = T(0); Li[c] = T(0); }
#pragma unroll
  for (int k = 0; k < NG; ++k) { gre[k] = T(0); gim[k] = T(0); gni[k] = T(0); }
  if (lane == 0) { my_lr[0] = T(0); my_li[0] = T(0); }
  T cvr = T(0), cvi = T(0);
  if (tid == 0) s_abort = 0;
  T lvr = T(0), lvi = T(0), lsg = T(1);
  if (my_row && part == 0) {
    lvr = Ar[(int64_t)pos + (int64_t)j * lda];
    lvi = Ai[(int64_t)pos + (int64_t)j * lda];
  }
  __syncthreads();

  for (int t = 0; t <= bw; ++t) {
    const int k = j + t;
    const bool active = my_row && lp >= k + 1;
    {
      T ar[4] = {T(0), T(0), T(0), T(0)}, ai[4] = {T(0), T(0), T(0), T(0)};
      static_assert(NG == 2, "two g registers");
      if (0 * 16 * S < t) {
        refresh16<0>(ar, gre[0], Lr);
        refresh16<0>(ar, gni[0], Li);
        refresh16<0>(ai, gre[0], Li);
        refresh16<0>(ai, gim[0], Lr);
      }
      if (1 * 16 * S < t) {
        refresh16<1>(ar, gre[1], Lr);
        refresh16<1>(ar, gni[1], Li);
        refresh16<1>(ai, gre[1], Li);
        refresh16<1>(ai, gim[1], Lr);
      }
      T sr = fma(lsg, lvr, (ar[0] + ar[1]) + (ar[2] + ar[3]));
      T si = fma(lsg, lvi, (ai[0] + ai[1]) + (ai[2] + ai[3]));
      sr = part_sum<S>(sr);
      si = part_sum<S>(si);
      if (active) { cvr = sr; cvi = si; }
    }
    if (t == bw) break;

    // ---- this wave's candidate: (|re| + |im|, position), first maximum; the
    //      candidate lane leaves its value in V for the agreement ----
    {
      double av = -1.0;
      if (active) {
        const double m = (double)(fabs(cvr) + fabs(cvi));
        if (m == m) av = m;
      }
      double bv;
      int bi;
      const int src = wave_first_max(av, active ? lp : INT32_MAX, bv, bi);
      int wpos = 0;
      if (src >= 0) {
        wpos = __builtin_amdgcn_readlane(pos, src);
        if (lane == src) {
          st_coh_t(&Vr[pos - (j + 1)], cvr);
          st_coh_t(&Vi[pos - (j + 1)], cvi);
        }
      }
      if (lane == 0) {
        red_v[wave] = src >= 0 ? bv : -1.0;
        red_k[wave] = ((uint64_t)(uint32_t)bi << 32) | ((uint64_t)wpos << 1);
      }
    }
    exchange_pivot<T>(a, k + 1, k, wave, lane, w, red_v, red_k, s_p, s_posw, s_none, s_abort);
    if (s_abort) return;
    const int p = s_p;
    const int posw = s_posw;
    const bool none = s_none != s_none;

    if (my_row && p != k + 1) {
      if (lp == p) lp = k + 1;
      else if (lp == k + 1) lp = p;
    }
    const bool next = my_row && lp >= k + 2;

    // ---- one round of loads: pivot value, pivot row multipliers, then the
    //      next stored column.  Under the in-order memory counter the
    //      division waits only for the pivot value and the LDS writes below
    //      only for the multipliers, while the stored column (a strided row
    //      read for rows above the pivot; every lane loads, at A(j+1, j)
    //      where it is not needed) is still in flight. ----
    T alr = T(NAN), ali = T(NAN);
    if (!none) {
      alr = ld_coh_t(&Vr[posw - (j + 1)]);
      ali = ld_coh_t(&Vi[posw - (j + 1)]);
    }
    constexpr int NLQ = (TOT + kWave - 1) / kWave;   // multiplier loads per lane (addresses clamped)
    T lrr[NLQ], lri[NLQ];
    {
      const int64_t ro = (int64_t)(posw - (j + 1));
      const int umax = t > 0 ? t - 1 : 0;
#pragma unroll
      for (int q = 0; q < NLQ; ++q) {
        const int64_t at = ro * bw + min(q * kWave + lane, umax);
        lrr[q] = ld_coh_t(&Gr[at]);
        lri[q] = ld_coh_t(&Gi[at]);
      }
    }
    const bool ldv = next && part == 0;
    const int64_t lvat =
        ldv ? (int64_t)max(pos, posw) + (int64_t)min(pos, posw) * lda : (int64_t)(j + 1) + (int64_t)j * lda;
    const T lvrn = Ar[lvat], lvin = Ai[lvat];
    __builtin_amdgcn_sched_barrier(0);             // keep the loads ahead of the work below

    // ---- multipliers of step k; the pivot row's multipliers into LDS before
    //      the slot write below (a jump), so their wait counts exactly.
    //      Entries past step t hold clamped copies that g discards; lane 0
    //      then writes the unit entry over entry t+1. ----
    T lr = T(0), li = T(0);
    if (next) {
      if (alr != T(0) || ali != T(0)) cdiv(cvr, cvi, alr, ali, lr, li);
    }
#pragma unroll
    for (int q = 0; q < NLQ; ++q) {
      const int u = q * kWave + lane;
      if (TOT % kWave == 0 || u < TOT) { my_lr[u + 1] = lrr[q]; my_li[u + 1] = lri[q]; }
    }
    if (lane == 0) {
      my_ar[t] = alr; my_ai[t] = ali;
      my_lr[t + 1] = T(1); my_li[t + 1] = T(0);   // unit diagonal of L
    }
    {
      const int c = t / S;
      const bool on = next && part == t % S;
      const T vr = lr, vi = li;
      static_assert(KCC == 32, "two groups of 16 slots");
      if constexpr (S >= 2) {
        cset_slot<T>(Lr, Li, c, on, vr, vi);
      } else {
        LTLT_CSET_GROUP(0) LTLT_CSET_GROUP(16)
      }
    }

    // ---- g coefficients for step k+1, row broadcast layout:
    //      g_u = alpha_{u+1} Lrow[u+1] [u <= t-1] - alpha_u Lrow[u-1] [u >= 1] ----
    wave_lds_sync();
    {
      const int c = lane & 15;
#pragma unroll
      for (int kk = 0; kk < NG; ++kk) {
        if (kk * 16 * S <= t) {
          const int u = (16 * kk + c) * S + part;  // < TOT
          const T a0r = my_ar[u], a0i = my_ai[u], a1r = my_ar[u + 1], a1i = my_ai[u + 1];
          const T lmr = my_lr[u], lmi = my_li[u], l1r = my_lr[u + 2], l1i = my_li[u + 2];
          T ur = T(0), ui = T(0);
          if (u <= t - 1) { ur = a1r * l1r - a1i * l1i; ui = a1r * l1i + a1i * l1r; }
          if (u >= 1) { ur -= a0r * lmr - a0i * lmi; ui -= a0r * lmi + a0i * lmr; }
          gre[kk] = (u <= t) ? ur : T(0);
          gim[kk] = (u <= t) ? ui : T(0);
          gni[kk] = -gim[kk];
        }
      }
    }
    // the stored column is taken before the stores below are issued, so its
    // wait does not include their acknowledgement
    if (ldv) {
      lvr = lvrn;
      lvi = lvin;
      lsg = pos > posw ? T(1) : T(-1);
    }
    asm volatile("" : "+v"(lvr), "+v"(lvi), "+v"(lsg) : : "memory");
    {
      int ro = pos - (j + 1);
      asm volatile("" : "+v"(ro));
      if (next && part == t % S) {
        st_coh_t(&Gr[(int64_t)ro * bw + t], lr);
        st_coh_t(&Gi[(int64_t)ro * bw + t], li);
      }
    }
    if (tid == 0 && w == 0) a.ipiv[k + 1] = p;
    wave_lds_sync();
  }

#undef LTLT_CSET_GROUP

  // ---- outputs by final position, straight from registers ----
  const int K = bw + 1;
  T* LLr = static_cast<T*>(ca.LL);
  T* LLi = LLr + (int64_t)K * ldw;
  T* LLr2 = LLi + (int64_t)K * ldw;
  T* BAr = static_cast<T*>(ca.BtA);                // Btr
  T* BAi = BAr + (int64_t)K * ldw;                 // -Bti
  T* BBr = static_cast<T*>(ca.BtB);                // Btr
  T* BBi = BBr + (int64_t)K * ldw;                 // Bti
  const int tr0 = j + bw + 1;
  const bool trailing = my_row && lp >= tr0;
  const T carr = trailing ? cvr : T(0), cari = trailing ? cvi : T(0);
  if (my_row) {
    const int64_t ro = lp - (j + 1);
#pragma unroll
    for (int c = 0; c < KCC; ++c) {
      const int u = c * S + part;
      if (u < bw) {
        LLr[ro + (int64_t)u * ldw] = Lr[c];
        LLi[ro + (int64_t)u * ldw] = Li[c];
        LLr2[ro + (int64_t)u * ldw] = Lr[c];
      }
    }
    if (part == 0) {
      LLr[ro + (int64_t)bw * ldw] = carr;
      LLi[ro + (int64_t)bw * ldw] = cari;
      LLr2[ro + (int64_t)bw * ldw] = carr;
    }
  }
  // Bt = Lx Tx^T: column u = a_u Lx_{u+1} - a_{u-1} Lx_{u-1},
  // a_u = alpha_{j+u+1} (u <= bw-2), a_{bw-1} = 1, Lx_bw = carry; the
  // neighbouring steps come from the neighbouring parts as in the real panel.
  const int up_src = (lane + RW) % kWave, dn_src = (lane + kWave - RW) % kWave;
#pragma unroll
  for (int c = 0; c < KCC; ++c) {
    const int cu = c + 1 < KCC ? c + 1 : c, cd = c >= 1 ? c - 1 : 0;
    const T gur = (part == 0 && c + 1 < KCC) ? Lr[cu] : (part == 0 ? T(0) : Lr[c]);
    const T gui = (part == 0 && c + 1 < KCC) ? Li[cu] : (part == 0 ? T(0) : Li[c]);
    const T gdr = (part == S - 1) ? (c >= 1 ? Lr[cd] : T(0)) : Lr[c];
    const T gdi = (part == S - 1) ? (c >= 1 ? Li[cd] : T(0)) : Li[c];
    const T xpr = S == 1 ? gur : __shfl(gur, up_src, kWave);
    const T xpi = S == 1 ? gui : __shfl(gui, up_src, kWave);
    const T xmr = S == 1 ? gdr : __shfl(gdr, dn_src, kWave);
    const T xmi = S == 1 ? gdi : __shfl(gdi, dn_src, kWave);
    const int u = c * S + part;
    if (trailing && u <= bw) {
      T vr = T(0), vi = T(0);
      if (u <= bw - 1) {
        const bool last = u + 1 == bw;
        const T br = last ? carr : xpr, bi = last ? cari : xpi;
        if (u <= bw - 2) {
          const T aur = my_ar[u + 1], aui = my_ai[u + 1];
          vr += aur * br - aui * bi;
          vi += aur * bi + aui * br;
        } else {
          vr += br;
          vi += bi;
        }
      }
      if (u >= 1) {
        if (u - 1 <= bw - 2) {
          const T amr = my_ar[u], ami = my_ai[u];
          vr -= amr * xmr - ami * xmi;
          vi -= amr * xmi + ami * xmr;
        } else {
          vr -= xmr;
          vi -= xmi;
        }
      }
      const int64_t at = (int64_t)(lp - tr0) + (int64_t)u * ldw;
      BAr[at] = vr;
      BAi[at] = -vi;
      BBr[at] = vr;
      BBi[at] = vi;
    }
  }
  // column bw when it lies past the slots (bw == TOT): -Lx_{bw-1}
  {
    const int src = (lane % RW) + (S - 1) * RW;
    const T lr_last = __shfl(Lr[KCC - 1], src, kWave);
    const T li_last = __shfl(Li[KCC - 1], src, kWave);
    if (trailing && bw == TOT && part == 0) {
      const int64_t at = (int64_t)(lp - tr0) + (int64_t)bw * ldw;
      BAr[at] = -lr_last;
      BAi[at] = li_last;
      BBr[at] = -lr_last;
      BBi[at] = -li_last;
    }
  }
  if (my_row && part == 0) a.perm[lp] = pos;
  if (w == 0 && wave == 0) {
    T* alr_out = static_cast<T*>(a.alpha);
    T* ali_out = static_cast<T*>(ca.alpha_i);
    for (int u = lane; u < bw; u += kWave) { alr_out[u] = my_ar[u]; ali_out[u] = my_ai[u]; }
  }
}

template <typename T, int S>
hipError_t launch_cpanel_s(const CPanelArgs& a, size_t lds, hipStream_t st) {
  return launch_resident_grid(cpanel_kernel<T, S>, (unsigned)a.b.P, kPanelThreads, lds, st, a);
}

template <typename T>
hipError_t launch_cpanel(const CPanelArgs& a, size_t lds, hipStream_t st) {
  if (a.b.P > kMaxPanelRecords || a.b.P > a.b.nrec || a.b.R != cpanel_rows(a.b.bw) || a.b.bw > 4 * KCC)
    return hipErrorInvalidValue;
  switch (cpanel_split(a.b.bw)) {
    case 1: return launch_cpanel_s<T, 1>(a, lds, st);
    case 2: return launch_cpanel_s<T, 2>(a, lds, st);
    case 4: return launch_cpanel_s<T, 4>(a, lds, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int S>
int cpanel_max_blocks_s(size_t lds) {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)cpanel_kernel<T, S>, kPanelThreads, lds) !=
      hipSuccess)
    return 0;
  return per_cu * cus;
}

template <typename T>
int cpanel_max_blocks(int bw, size_t lds) {
  int cap;
  switch (cpanel_split(bw)) {
    case 1: cap = cpanel_max_blocks_s<T, 1>(lds); break;
    case 2: cap = cpanel_max_blocks_s<T, 2>(lds); break;
    case 4: cap = cpanel_max_blocks_s<T, 4>(lds); break;
    default: return 0;
  }
  return cap < kMaxPanelRecords ? cap : kMaxPanelRecords;
}

// ---------------------------------------------------------------------------
// Interleaved complex <-> two real planes, strict lower triangle only.  One
// workgroup per column (grid-stride over columns), rows across the threads.
template <typename T>
__global__ void __launch_bounds__(256) cplx_split_kernel(int n, const T* A, int64_t lda, T* Pr, T* Pi, int64_t ldp) {
  for (int c = blockIdx.x; c < n; c += gridDim.x) {
    const T* col = A + 2 * (int64_t)c * lda;
    for (int i = c + 1 + threadIdx.x; i < n; i += blockDim.x) {
      const T re = col[2 * (int64_t)i], im = col[2 * (int64_t)i + 1];
      Pr[(int64_t)i + (int64_t)c * ldp] = re;
      Pi[(int64_t)i + (int64_t)c * ldp] = im;
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(256) cplx_merge_kernel(int n, T* A, int64_t lda, const T* Pr, const T* Pi,
                                                         int64_t ldp) {
  for (int c = blockIdx.x; c < n; c += gridDim.x) {
    T* col = A + 2 * (int64_t)c * lda;
    for (int i = c + 1 + threadIdx.x; i < n; i += blockDim.x) {
      col[2 * (int64_t)i] = Pr[(int64_t)i + (int64_t)c * ldp];
      col[2 * (int64_t)i + 1] = Pi[(int64_t)i + (int64_t)c * ldp];
    }
  }
}

template <typename T>
hipError_t launch_cplx_split(int n, const void* A, int64_t lda, T* Pr, T* Pi, int64_t ldp, hipStream_t s) {
  if (n <= 1) return hipSuccess;
  const int g = n < 4096 ? n : 4096;
  hipLaunchKernelGGL(cplx_split_kernel<T>, dim3(g), dim3(256), 0, s, n, static_cast<const T*>(A), lda, Pr, Pi, ldp);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_cplx_merge(int n, void* A, int64_t lda, const T* Pr, const T* Pi, int64_t ldp, hipStream_t s) {
  if (n <= 1) return hipSuccess;
  const int g = n < 4096 ? n : 4096;
  hipLaunchKernelGGL(cplx_merge_kernel<T>, dim3(g), dim3(256), 0, s, n, static_cast<T*>(A), lda, Pr, Pi, ldp);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Complex Pfaffian from the (interleaved) factors: log|Pf| = sum_j log|alpha_{2j}| (fp64,
// |z| by hypot) and the phase Pf/|Pf| = det(P) prod_j (-alpha_{2j})/|alpha_{2j}|,
// both by one fixed-order tree reduction (sums of logs, products of unit
// complex numbers).
// A raised abort flag (status[0]) gives log|Pf| = NaN and phase 0.
template <typename T>
__global__ void __launch_bounds__(1024) cpfaffian_kernel(int n, const T* A, int64_t lda, const int* ipiv,
                                                         double* logabs, double* phase, const int* status) {
  __shared__ double s_log[1024], s_pr[1024], s_pi[1024];
  __shared__ int s_zero[1024];
  const int tid = threadIdx.x;
  double lg = 0.0, pr = 1.0, pi = 0.0;
  int zero = 0, neg = 0;
  const int half = n / 2;
  if ((n & 1) == 0) {
    for (int jj = tid; jj < half; jj += 1024) {
      const int64_t at = 2 * ((int64_t)(2 * jj + 1) + (int64_t)(2 * jj) * lda);   // (re, im) pairs
      const double ar = (double)A[at], ai = (double)A[at + 1];
      const double mag = hypot(ar, ai);
      if (mag == 0.0) zero = 1;
      else {
        lg += log(mag);
        const double ur = -ar / mag, ui = -ai / mag;   // factor T(2j,2j+1) = -alpha_{2j}
        const double tr = pr * ur - pi * ui;
        pi = pr * ui + pi * ur;
        pr = tr;
      }
    }
    for (int i = tid; i < n; i += 1024)
      if (ipiv[i] != i) neg ^= 1;
    if (neg) { pr = -pr; pi = -pi; }
  }
  s_log[tid] = lg; s_pr[tid] = pr; s_pi[tid] = pi; s_zero[tid] = zero;
  __syncthreads();
  for (int st = 512; st >= 1; st >>= 1) {
    if (tid < st) {
      s_log[tid] += s_log[tid + st];
      const double ar = s_pr[tid], ai = s_pi[tid], br = s_pr[tid + st], bi = s_pi[tid + st];
      s_pr[tid] = ar * br - ai * bi;
      s_pi[tid] = ar * bi + ai * br;
      s_zero[tid] |= s_zero[tid + st];
    }
    __syncthreads();
  }
  if (tid == 0) {
    if (status[0] != 0) { *logabs = NAN; phase[0] = 0.0; phase[1] = 0.0; }
    else if ((n & 1) || s_zero[0]) { *logabs = -INFINITY; phase[0] = 0.0; phase[1] = 0.0; }
    else {
      // renormalise the product of unit factors (rounding drift only)
      const double m = hypot(s_pr[0], s_pi[0]);
      *logabs = s_log[0];
      phase[0] = s_pr[0] / m;
      phase[1] = s_pi[0] / m;
    }
  }
}

template <typename T>
hipError_t launch_cpfaffian(int n, const void* A, int64_t lda, const int* ipiv, double* logabs, double* phase,
                            const int* status, hipStream_t s) {
  hipLaunchKernelGGL(cpfaffian_kernel<T>, dim3(1), dim3(1024), 0, s, n, static_cast<const T*>(A), lda, ipiv, logabs,
                     phase, status);
  return hipGetLastError();
}

#define LTLT_CINST(T)                                                                                        \
  template size_t cpanel_lds_bytes<T>(int);                                                                 \
  template int cpanel_max_blocks<T>(int, size_t);                                                           \
  template hipError_t launch_cpanel<T>(const CPanelArgs&, size_t, hipStream_t);                             \
  template hipError_t launch_cplx_split<T>(int, const void*, int64_t, T*, T*, int64_t, hipStream_t);        \
  template hipError_t launch_cplx_merge<T>(int, void*, int64_t, const T*, const T*, int64_t, hipStream_t);  \
  template hipError_t launch_cpfaffian<T>(int, const void*, int64_t, const int*, double*, double*, const int*,  \
                                          hipStream_t);
LTLT_CINST(double)
LTLT_CINST(float)
#undef LTLT_CINST

}  // namespace ltlt
