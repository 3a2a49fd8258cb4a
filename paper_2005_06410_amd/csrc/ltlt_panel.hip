// Panel kernel: the column steps k = j .. j+bw-1 of one block of the pivoted
// skew-symmetric reduction P X P^T = L T L^T, run by P co-resident
// workgroups that each own R consecutive positions (rows) of the block.
//
// Thread layout: 256 threads per workgroup, S adjacent lanes per row
// (R = 256/S rows), lane part p of a row holds the row's multipliers of the
// steps u with u % S == p in registers (L[c] = multiplier of step j + c*S + p,
// c < kCpt).  Per-row state (block-start index pos, current column value cv)
// is replicated in the S lanes of the row.
//
// A copy of the multipliers also lives in global memory, indexed by the
// block-start index (so it never needs reordering): G[pos - (j+1)][u].
//
// Column refresh.  The trailing matrix is stored as it was at block start
// (strict lower triangle), so the current column k is the stored column of
// index pos[k] gathered through pos[], plus the not-yet-applied updates of
// steps j .. k-2.  Step s updates X(i,c) += l_i v_c - v_i l_c with v the
// column s+1 at step s, and v = alpha_{s+1} * L(:, s+2) below row s+2
// (column s+1 is the one step s+1 eliminates).  Summed over the block this is
// Lp Tx Lp^T with Tx skew tridiagonal, Tx[u,u+1] = alpha_{j+u+1}; the
// refresh of column k therefore needs only row k of Lp:
//   cv[i] = S(pos[i], pos[k]) + sum_{u<t} g_u Lp[u][i],
//   g_u = alpha_{j+u+1} Lrow[u+1] [u <= t-2] - alpha_{j+u} Lrow[u-1] [u >= 1],
//   Lrow[w] = Lp[w][k] (w <= t-2), Lrow[t-1] = 1 (unit diagonal of L),
// with S(a, b) = A(a, b) for a > b and -A(b, a) for a < b.
//
// Exchange per step (one grid-wide round, no counters, no fences): every
// workgroup publishes its local pivot candidate as one 16-byte record of two
// self-validating 64-bit words (each carries the step stamp), and the owner
// of position k+1 publishes that position the same way.  Wave 0 of every
// workgroup polls all records until each carries the current stamp, then
// reduces them in the same order (largest magnitude, then smallest position:
// the first maximum in position order), so all agree on the pivot p.  The
// pivot row's multipliers (and, for the owner of p, those of the row leaving
// k+1) are read from G together with the next stored column, in one round of
// loads.  Multipliers written to G at step k are read no earlier than step
// k+1; each workgroup waits for its own earlier stores to complete before
// publishing the record of the following step, so any record that validates
// implies those stores are visible.
//
// After the last step the carry column (column j+bw, refreshed) is formed and
// the block's outputs are written: Lx = [Lp, carry] (rows >= j+bw+1) feeds
// the trailing update as one rank-(bw+1) product with Bt = Lx Tx^T; the rows
// inside the block and the alphas are committed into A after that update.

#include "ltlt_device.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int kCpt = 64;   // multipliers per lane (register resident)

// Lanes per row for a block of width bw.
int panel_split(int bw) { return bw <= kCpt ? 1 : (bw <= 2 * kCpt ? 2 : 4); }

template <typename T>
size_t panel_lds_bytes(int bw, int R) {
  const int S = kThreads / R;
  size_t t = 0;
  t += (size_t)S * kCpt * sizeof(T);              // g, split by lane part
  t += (size_t)(bw + 1) * sizeof(T) * 3;          // alpha, lrow, oldrow
  t += (size_t)R * (bw + 1) * sizeof(T);          // multipliers gathered for the outputs
  return t + 64;
}

// Record words.  s = k + 1 is the step stamp (1 <= s < 2^21).
//   word A = bits(|cv|) | epoch(s) << 63,   epoch(s) = (s >> 1) & 1
//   word B = (s << 43) | (sign(cv) << 42) | (pos << 21) | idx
// A record slot alternates with s & 1 and every record location is written at
// every step of its slot, so a slot holds stamp s or s-2 and the epoch bit
// alone tells them apart in word A; word B carries the full stamp.
constexpr uint64_t kIdxNone = 0x1FFFFFull;
constexpr int kRecWords = 2;    // records packed: 8 per 128-byte line, one wave poll touches few lines
__device__ __forceinline__ uint64_t rec_a(double absv, int s) {
  return (uint64_t)__double_as_longlong(absv) | ((uint64_t)((s >> 1) & 1) << 63);
}
__device__ __forceinline__ uint64_t rec_b(int s, int sgn, int pos, uint64_t idx) {
  return ((uint64_t)s << 43) | ((uint64_t)sgn << 42) | ((uint64_t)pos << 21) | idx;
}
__device__ __forceinline__ bool rec_valid(uint64_t a, uint64_t b, int s) {
  return (int)(a >> 63) == ((s >> 1) & 1) && (int)(b >> 43) == s;
}
__device__ __forceinline__ uint64_t ld_coh64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st_coh_t(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T ld_coh_t(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// S(a, b) of the stored (strict lower) skew matrix, a != b.
template <typename T>
__device__ __forceinline__ T skew_at(const T* A, int64_t lda, int a, int b) {
  return a > b ? A[(int64_t)a + (int64_t)b * lda] : -A[(int64_t)b + (int64_t)a * lda];
}

template <typename T, int S>
__global__ void __launch_bounds__(kThreads, 1) panel_kernel(PanelArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int R = kThreads / S;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int w = blockIdx.x;
  const int bw = a.bw, n = a.n, j = a.j, P = a.P;
  const int rloc = tid / S;            // row of this lane
  const int part = tid % S;            // multiplier slice of this lane
  const int64_t lda = a.lda, ldw = a.ldw;
  const T* A = static_cast<const T*>(a.A);
  T* G = static_cast<T*>(a.G);

  T *gp, *alpha, *lrow, *oldrow, *dump;
  {
    unsigned char* p = smem;
    gp = reinterpret_cast<T*>(p); p += (size_t)S * kCpt * sizeof(T);
    alpha = reinterpret_cast<T*>(p); p += (size_t)(bw + 1) * sizeof(T);
    lrow = reinterpret_cast<T*>(p); p += (size_t)(bw + 1) * sizeof(T);
    oldrow = reinterpret_cast<T*>(p); p += (size_t)(bw + 1) * sizeof(T);
    dump = reinterpret_cast<T*>(p);
  }
  __shared__ double red_v[kThreads / kWave];
  __shared__ int red_i[kThreads / kWave], red_p[kThreads / kWave];
  __shared__ T red_c[kThreads / kWave];
  __shared__ int s_p, s_posw, s_posk, s_abort;
  __shared__ T s_alpha, s_cvk;

  const int row0 = j + 1 + w * R;                 // first position owned
  const int rows_here = max(0, min(R, n - row0));
  const int my_i = row0 + rloc;
  const bool my_row = rloc < rows_here;

  T L[kCpt];
#pragma unroll
  for (int c = 0; c < kCpt; ++c) L[c] = T(0);
  for (int e = tid; e < S * kCpt; e += kThreads) gp[e] = T(0);
  int pos = my_i;                                  // block-start index of this row
  T cv = T(0);
  if (tid == 0) s_abort = 0;
  // first stored column: index j, rows >= j+1 (lower part only)
  T lv = T(0);
  if (my_row && part == 0) lv = A[(int64_t)my_i + (int64_t)j * lda];
  __syncthreads();

  for (int t = 0; t <= bw; ++t) {
    const int k = j + t;
    // ---- column refresh: cv = S(pos, q) + sum_u g_u L_u over rows >= k+1 ----
    const bool active = my_row && (my_i >= k + 1);
    {
      const T* gq = gp + part * kCpt;
      T a0 = T(0), a1 = T(0), a2 = T(0), a3 = T(0);
#pragma unroll
      for (int c = 0; c < kCpt; c += 4) {
        a0 += gq[c] * L[c];
        a1 += gq[c + 1] * L[c + 1];
        a2 += gq[c + 2] * L[c + 2];
        a3 += gq[c + 3] * L[c + 3];
      }
      T acc = ((a0 + a1) + (a2 + a3)) + lv;      // lv is nonzero in part 0 only
      if (S >= 2) acc += __shfl_xor(acc, 1, kWave);
      if (S >= 4) acc += __shfl_xor(acc, 2, kWave);
      if (active) cv = acc;
    }
    if (t == bw) break;                           // carry column formed

    // ---- local pivot candidate ----
    double bv = -1.0;
    int bi = INT32_MAX;
    if (active) {
      const double av = (double)fabs(cv);
      if (av == av) { bv = av; bi = my_i; }       // NaN is never a candidate
    }
    wave_argmax_dpp(bv, bi);
    if (bi == INT32_MAX) {
      if (lane == 0) { red_v[wave] = -1.0; red_i[wave] = INT32_MAX; }
    } else if (my_i == bi && part == 0) {         // the candidate's own lane
      red_v[wave] = bv; red_i[wave] = bi; red_c[wave] = cv; red_p[wave] = pos;
    }
    const int s = k + 1;
    uint64_t* recs = a.rec + (size_t)(s & 1) * (size_t)(a.kslot + 1) * kRecWords;
    wait_stores();                                // this wave's earlier G stores are complete
    if (my_i == k + 1 && my_row && part == 0) {   // owner of position k+1 publishes it
      st_coh64(&recs[kRecWords * a.kslot + 0], rec_a((double)fabs(cv), s));
      st_coh64(&recs[kRecWords * a.kslot + 1], rec_b(s, cv < T(0) ? 1 : 0, pos, (uint64_t)(k + 1)));
    }
    __syncthreads();
    // ---- publish this workgroup's candidate (lane 0 of wave 0) ----
    if (tid == 0) {
      double cb = red_v[0];
      int ci = red_i[0], cw = 0;
      for (int wv = 1; wv < kThreads / kWave; ++wv) {
        const double ov = red_v[wv];
        const int oi = red_i[wv];
        if (ov > cb || (ov == cb && oi < ci)) { cb = ov; ci = oi; cw = wv; }
      }
      if (ci == INT32_MAX) {
        st_coh64(&recs[kRecWords * w + 0], rec_a(0.0, s));
        st_coh64(&recs[kRecWords * w + 1], rec_b(s, 0, 0, kIdxNone));
      } else {
        st_coh64(&recs[kRecWords * w + 0], rec_a(cb, s));
        st_coh64(&recs[kRecWords * w + 1], rec_b(s, red_c[cw] < T(0) ? 1 : 0, red_p[cw], (uint64_t)ci));
      }
    }
    // ---- poll all records and reduce (wave 0); entry u == P is position k+1 ----
    if (wave == 0) {
      double gv = -1.0;
      int gi = INT32_MAX, gpos = 0, gsg = 0;
      int kpos = 0, ksg = 0;
      double kabs = 0.0;
      const uint64_t t0 = wall_ticks();
      for (int u0 = 0; u0 <= P; u0 += kWave) {
        const int u = u0 + lane;
        if (u <= P) {
          const int ri = (u < P) ? u : a.kslot;
          uint64_t ra, rb;
          for (;;) {
            ra = ld_coh64(&recs[kRecWords * ri + 0]);
            rb = ld_coh64(&recs[kRecWords * ri + 1]);
            if (rec_valid(ra, rb, s)) break;
            if (wall_ticks() - t0 > kWaitLimitTicks || ld_coh(a.status) != 0) {
              atomicOr(a.status, 1);
              s_abort = 1;
              break;
            }
            __builtin_amdgcn_s_sleep(0);
          }
          const double av = __longlong_as_double((long long)(ra & 0x7FFFFFFFFFFFFFFFull));
          const int ix = (int)(rb & kIdxNone);
          const int px = (int)((rb >> 21) & kIdxNone);
          const int sg = (int)((rb >> 42) & 1);
          if (u < P) {
            if ((uint64_t)ix != kIdxNone && (av > gv || (av == gv && ix < gi))) {
              gv = av; gi = ix; gpos = px; gsg = sg;
            }
          } else {
            kabs = av; kpos = px; ksg = sg;
          }
        }
      }
      const int klane = P % kWave;                // lane that read the position-(k+1) record
      kabs = __shfl(kabs, klane, kWave);
      kpos = __shfl(kpos, klane, kWave);
      ksg = __shfl(ksg, klane, kWave);
      {
        // wave argmax on (|value|, position); the winning lane then supplies
        // the block-start index and sign of the winner
        const int my_gi = gi;
        wave_argmax_dpp(gv, gi);
        const unsigned long long hit = __ballot(gi != INT32_MAX && my_gi == gi);
        const int src = hit ? __ffsll(hit) - 1 : 0;
        gpos = __shfl(gpos, src, kWave);
        gsg = __shfl(gsg, src, kWave);
      }
      if (lane == 0) {
        const T ck = ksg ? -(T)kabs : (T)kabs;
        s_cvk = ck;
        s_posk = kpos;
        if (gi == INT32_MAX) {                    // no finite candidate: keep k+1
          s_p = k + 1; s_alpha = ck; s_posw = kpos;
        } else {
          s_p = gi; s_alpha = gsg ? -(T)gv : (T)gv; s_posw = gpos;
        }
      }
    }
    __syncthreads();
    if (s_abort) return;
    const int p = s_p;
    const int posw = s_posw, posk = s_posk;
    const T alph = s_alpha, cvk = s_cvk;
    // ---- one round of loads: next stored column, pivot row, leaving row ----
    const bool is_k1 = my_row && my_i == k + 1;
    const bool is_p = my_row && p != k + 1 && my_i == p;
    if (is_p) pos = posk;                         // the row leaving k+1 lands at p
    if (is_k1) pos = posw;
    if (my_row && part == 0 && my_i >= k + 2) lv = skew_at(A, lda, pos, posw);
    // the pivot row's multipliers (all workgroups) and, in the workgroup that
    // owns p, those of the row leaving k+1: one value per thread, one round
    const bool wg_owns_p = (p != k + 1) && p >= row0 && p < row0 + rows_here;
    if (tid < t) {
      lrow[tid] = ld_coh_t(&G[(int64_t)(posw - (j + 1)) + (int64_t)tid * ldw]);
      if (wg_owns_p) oldrow[tid] = ld_coh_t(&G[(int64_t)(posk - (j + 1)) + (int64_t)tid * ldw]);
    }
    __syncthreads();
    if (is_p) {
#pragma unroll
      for (int c = 0; c < kCpt; ++c) {
        const int u = c * S + part;
        L[c] = u < t ? oldrow[u < t ? u : 0] : T(0);
      }
      cv = cvk;
    }
    // ---- multipliers of step k (the row now at k+1 is final: its
    //      multipliers are taken from G for the output) ----
    if (my_row && my_i >= k + 2) {
      const T l = (alph != T(0)) ? cv / alph : T(0);
      const int cslot = t / S;
      if (part == t % S) {
#pragma unroll
        for (int c = 0; c < kCpt; ++c)
          if (c == cslot) L[c] = l;
        st_coh_t(&G[(int64_t)(pos - (j + 1)) + (int64_t)t * ldw], l);
      }
    }
    // g coefficients for step k+1 (t+1 terms); alpha_{j+t} and Lrow[t] = 1 are new
    if (tid <= t) {
      const int u = tid;
      T gu = T(0);
      if (u <= t - 1) {
        const T an = (u + 1 == t) ? alph : alpha[u + 1];
        const T ln = (u + 1 == t) ? T(1) : lrow[u + 1];
        gu += an * ln;
      }
      if (u >= 1) {
        const T am = (u == t) ? alph : alpha[u];
        gu -= am * lrow[u - 1];
      }
      gp[(u % S) * kCpt + u / S] = gu;
    }
    if (tid == 0) { alpha[t] = alph; if (w == 0) a.ipiv[k + 1] = p; }
    __syncthreads();
  }

  // ---- outputs: multipliers through LDS (Bt needs neighbouring columns).
  //      Rows still active hold every multiplier in registers; the final
  //      pivot rows (positions j+1 .. j+bw) read theirs from G, whose entries
  //      all predate the last exchange. ----
  wait_stores();
  __syncthreads();
  const int tr0 = j + bw + 1;                      // first trailing position
  if (my_row) {
    if (my_i >= tr0) {
#pragma unroll
      for (int c = 0; c < kCpt; ++c) {
        const int u = c * S + part;
        if (u < bw) dump[u * R + rloc] = L[c];
      }
      if (part == 0) dump[bw * R + rloc] = cv;    // carry
    } else {
      const T* src = G + (int64_t)(pos - (j + 1));
      for (int u = part; u < bw; u += S) dump[u * R + rloc] = ld_coh_t(&src[(int64_t)u * ldw]);
      if (part == 0) dump[bw * R + rloc] = T(0);
    }
  }
  __syncthreads();
  T* PO = static_cast<T*>(a.PO);
  T* Bm = static_cast<T*>(a.Bm);
  for (int r = tid; r < rows_here; r += kThreads) {
    const int ii = row0 + r;
    const int64_t ro = ii - (j + 1);
    for (int u = 0; u < bw; ++u) PO[ro + u * ldw] = dump[u * R + r];
    if (ii >= tr0) {
      const T carry = dump[bw * R + r];
      PO[ro + (int64_t)bw * ldw] = carry;
      const int64_t rb = ii - tr0;
      // Bt = Lx Tx^T: column u = a_u Lx_{u+1} - a_{u-1} Lx_{u-1},
      // a_u = alpha_{j+u+1} (u <= bw-2), a_{bw-1} = 1, Lx_bw = carry.
      for (int u = 0; u <= bw; ++u) {
        T v = T(0);
        if (u <= bw - 1) {
          const T au = (u <= bw - 2) ? alpha[u + 1] : T(1);
          v += au * dump[(u + 1) * R + r];
        }
        if (u >= 1) {
          const T am = (u - 1 <= bw - 2) ? alpha[u] : T(1);
          v -= am * dump[(u - 1) * R + r];
        }
        Bm[rb + u * ldw] = v;
      }
    }
  }
  if (my_row && part == 0) a.perm[my_i] = pos;
  if (w == 0) {
    T* al = static_cast<T*>(a.alpha);
    for (int u = tid; u < bw; u += kThreads) al[u] = alpha[u];
  }
}

template <typename T, int S>
hipError_t allow_panel_lds() {
  static bool done = false;
  if (done) return hipSuccess;
  hipFuncAttributes fa;
  hipError_t e = hipFuncGetAttributes(&fa, (const void*)panel_kernel<T, S>);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)panel_kernel<T, S>, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)(160 * 1024 - fa.sharedSizeBytes));
  if (e != hipSuccess) return e;
  done = true;
  return hipSuccess;
}

template <typename T, int S>
hipError_t launch_panel_s(const PanelArgs& a, size_t lds, hipStream_t st) {
  hipError_t e = allow_panel_lds<T, S>();
  if (e != hipSuccess) return e;
  PanelArgs copy = a;
  void* args[] = {&copy};
  return hipLaunchCooperativeKernel((const void*)panel_kernel<T, S>, dim3(a.P), dim3(kThreads), args,
                                    (unsigned)lds, st);
}

template <typename T>
hipError_t launch_panel(const PanelArgs& a, size_t lds, hipStream_t st) {
  switch (kThreads / a.R) {
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
  if (allow_panel_lds<T, S>() != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)panel_kernel<T, S>, kThreads, lds) !=
      hipSuccess)
    return 0;
  return per_cu * cus;
}

template <typename T>
int panel_max_blocks(int R, size_t lds) {
  switch (kThreads / R) {
    case 1: return panel_max_blocks_s<T, 1>(lds);
    case 2: return panel_max_blocks_s<T, 2>(lds);
    case 4: return panel_max_blocks_s<T, 4>(lds);
    default: return 0;
  }
}

int panel_rows(int bw) { return kThreads / panel_split(bw); }

// Exchange records start with stamps that can never validate: word B stamp 0,
// and word A epoch opposite to that of the first stamp using the slot
// (slot 1 first holds s = 1, epoch 0; slot 0 first holds s = 2, epoch 1).
__global__ void rec_init_kernel(uint64_t* rec, int nrec) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 2 * kRecWords * nrec) return;
  const int slot = i / (kRecWords * nrec);
  const int word = i % kRecWords;
  rec[i] = (word == 0 && slot == 1) ? (1ull << 63) : 0ull;
}

hipError_t launch_rec_init(uint64_t* rec, int nrec_per_slot, hipStream_t s) {
  const int tot = 2 * kRecWords * nrec_per_slot;
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
