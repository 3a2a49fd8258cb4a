// Exchange machinery shared by the panel kernels: the per-step pivot
// agreement between the co-resident workgroups of a panel (records, poll,
// reduction), the register-slot helpers and the part sums of a row.
#pragma once

#include "ltlt_device.h"
#include "ltlt_internal.h"

namespace ltlt {

constexpr int kPollPerLane = kMaxPanelRecords / kWave;   // records per polling lane
constexpr int KC = 64;                                   // multiplier slots per lane

// Lanes per row and register slots per lane for a block of width bw.
inline int panel_split(int bw) { return bw <= KC ? 1 : (bw <= 2 * KC ? 2 : 4); }

// Record words.  s is the step stamp (1 <= s < 2^21; it grows by one per
// exchange, so consecutive exchanges use alternate record slots).
//   word A = bits(|cv|) | epoch(s) << 63,   epoch(s) = (s >> 1) & 1
//   word B = (s << 43) | (sign(cv) << 42) | (pos << 21) | lp
// A record slot alternates with s & 1 and every record location is written at
// every step of its slot, so a slot holds stamp s or s-2 and the epoch bit
// alone tells them apart in word A; word B carries the full stamp.
constexpr uint64_t kIdxNone = 0x1FFFFFull;
__device__ __forceinline__ uint64_t rec_a(double absv, int s) {
  return ((uint64_t)__double_as_longlong(absv) & 0x7FFFFFFFFFFFFFFFull) | ((uint64_t)((s >> 1) & 1) << 63);
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

// LDS written by some lanes of a wave is read by other lanes of the same wave:
// wait for the wave's LDS operations and keep the compiler from moving memory
// accesses across this point.
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// L[c] = v where `on`, for a wave-uniform slot c: a uniform branch on the
// group of 16 slots, then selects inside the group, so that register indices
// stay static and the other 48 slots are untouched.
#define LTLT_SET_GROUP(G0)                                                       \
  if ((c >> 4) == (G0) / 16) {                                                  \
    _Pragma("unroll") for (int i = 0; i < 16; ++i) L[(G0) + i] = (on && c == (G0) + i) ? v : L[(G0) + i]; \
  }

// L[c] = v where `on`, for a wave-uniform slot c < KC: a uniform jump to the
// one slot (register indices stay static and only that slot is written),
// instead of LTLT_SET_GROUP's selects over a whole group of 16.  Measured
// faster in the two- and four-lane-per-row panels; with one lane per row the
// jump table's control flow pushed the kernel past its register budget, so
// that panel keeps the group form.
#define LTLT_SLOT_CASE(i) \
  case (i): L[(i)] = on ? v : L[(i)]; break;
#define LTLT_SLOT_CASE4(i) LTLT_SLOT_CASE(i) LTLT_SLOT_CASE((i) + 1) LTLT_SLOT_CASE((i) + 2) LTLT_SLOT_CASE((i) + 3)
#define LTLT_SLOT_CASE16(i) \
  LTLT_SLOT_CASE4(i) LTLT_SLOT_CASE4((i) + 4) LTLT_SLOT_CASE4((i) + 8) LTLT_SLOT_CASE4((i) + 12)
template <typename T>
__device__ __forceinline__ void set_slot(T (&L)[KC], int c, bool on, T v) {
  static_assert(KC == 64, "64 slots");
  switch (c) {
    LTLT_SLOT_CASE16(0) LTLT_SLOT_CASE16(16) LTLT_SLOT_CASE16(32) LTLT_SLOT_CASE16(48)
    default: break;
  }
}
#undef LTLT_SLOT_CASE16
#undef LTLT_SLOT_CASE4
#undef LTLT_SLOT_CASE

// v + (v of lane ^ 16) or v + (v of lane ^ 32) through the gfx950 lane
// swaps (no LDS crossbar round trip): with both operands v, permlane16_swap
// returns in every 16-lane row the values of the even row of its pair and
// of the odd row (permlane32_swap: of the lower and the upper half), whose
// sum has the same two terms as v + shfl_xor(v, 16 | 32), bit for bit.
template <int OFF>
__device__ __forceinline__ unsigned xor_pair(unsigned x, unsigned& other) {
  if constexpr (OFF == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    other = r[1];
    return r[0];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    other = r[1];
    return r[0];
  }
}
template <int OFF>
__device__ __forceinline__ double xor_add(double v) {
  unsigned lo1, hi1;
  const unsigned lo0 = xor_pair<OFF>((unsigned)__double2loint(v), lo1);
  const unsigned hi0 = xor_pair<OFF>((unsigned)__double2hiint(v), hi1);
  return __hiloint2double((int)hi0, (int)lo0) + __hiloint2double((int)hi1, (int)lo1);
}
template <int OFF>
__device__ __forceinline__ float xor_add(float v) {
  unsigned o;
  const unsigned a = xor_pair<OFF>(__float_as_uint(v), o);
  return __uint_as_float(a) + __uint_as_float(o);
}
// Sum of v over the S parts of a row (lanes lane ^ 16, lane ^ 32).
template <int S, typename T>
__device__ __forceinline__ T part_sum(T v) {
  if constexpr (S == 4) v = xor_add<16>(v);
  if constexpr (S >= 2) v = xor_add<32>(v);
  return v;
}

// One grid-wide pivot agreement, in two halves called by every thread of the
// workgroup (work that does not depend on the pivot may run in between).
// Each wave has put its first-maximum candidate in red_v / red_k (lane 0:
// |cv|, key = position << 32 | block-start index << 1 | sign).
// exchange_publish: every wave waits for its own earlier stores (so a
// validated record implies they are visible), a barrier, then wave 0 merges
// the waves and publishes the workgroup's record for stamp s.
// exchange_collect: wave 0 polls every record until all carry stamp s and
// reduces them (largest magnitude, then smallest position); the result lands
// in s_p (pivot position), s_posw (its block-start index) and s_alpha
// (signed pivot value; NaN and p = k+1 when no finite candidate exists),
// handed to the other waves by a barrier.  A wait that exceeds its bound, or
// finds the call's abort flag raised, raises the status words and s_abort.
__device__ __forceinline__ void exchange_publish(const PanelArgs& a, int s, int wave, int lane, int w,
                                                 const double* red_v, const uint64_t* red_k) {
  uint64_t* recs = a.rec + (size_t)(s & 1) * (size_t)a.nrec * kRecStride;
  wait_stores();
  __syncthreads();
  if (wave == 0) {
    double cb = red_v[0];
    uint64_t ck = red_k[0];
#pragma unroll
    for (int wv = 1; wv < kPanelWaves; ++wv) {
      const double ov = red_v[wv];
      const uint64_t ok = red_k[wv];
      const bool take = (ov > cb) | ((ov == cb) & (ok < ck));
      cb = take ? ov : cb;
      ck = take ? ok : ck;
    }
    if (lane == 0) {
      const int ci = (int)(ck >> 32);
      const bool none = ci == INT32_MAX;
      st_coh64(&recs[(size_t)kRecStride * w + 0], rec_a(none ? 0.0 : cb, s));
      st_coh64(&recs[(size_t)kRecStride * w + 1],
               rec_b(s, (int)(ck & 1), (int)((ck >> 1) & kIdxNone), none ? kIdxNone : (uint64_t)ci));
    }
  }
}

template <typename T>
__device__ __forceinline__ void exchange_collect(const PanelArgs& a, int s, int k, int wave, int lane, int& s_p,
                                                 int& s_posw, T& s_alpha, int& s_abort) {
  const int P = a.P;
  const uint64_t* recs = a.rec + (size_t)(s & 1) * (size_t)a.nrec * kRecStride;
  if (wave == 0) {
    const int q_n = (P + kWave - 1) / kWave;
    const uint64_t t0 = wall_ticks();
    uint64_t ra[kPollPerLane], rb[kPollPerLane];
    for (;;) {
#pragma unroll
      for (int q = 0; q < kPollPerLane; ++q) {
        const int u = q * kWave + lane;
        if (q < q_n && u < P) {
          ra[q] = ld_coh64(&recs[(size_t)kRecStride * u + 0]);
          rb[q] = ld_coh64(&recs[(size_t)kRecStride * u + 1]);
        }
      }
      const int stv = ld_coh(a.status);           // same round trip as the records
      bool ok = true;
#pragma unroll
      for (int q = 0; q < kPollPerLane; ++q) {
        const int u = q * kWave + lane;
        if (q < q_n && u < P) ok = ok && rec_valid(ra[q], rb[q], s);
      }
      // a wait of this call that gave up elsewhere ends this one too, even
      // when every record has arrived
      if (stv != 0 || (__ballot(!ok) != 0 && wall_ticks() - t0 > kWaitLimitTicks)) {
        if (lane == 0) { raise_wait_status(a.status); s_abort = 1; }
        break;
      }
      if (__ballot(!ok) == 0) break;
      __builtin_amdgcn_s_sleep(0);
    }
    double gv = -1.0;
    int gi = INT32_MAX, gpos = 0, gsg = 0;
#pragma unroll
    for (int q = 0; q < kPollPerLane; ++q) {
      const int u = q * kWave + lane;
      if (q < q_n && u < P) {
        const double av = __longlong_as_double((long long)(ra[q] & 0x7FFFFFFFFFFFFFFFull));
        const int ix = (int)(rb[q] & kIdxNone);
        const bool take = ((uint64_t)ix != kIdxNone) & ((av > gv) | ((av == gv) & (ix < gi)));
        gv = take ? av : gv;
        gi = take ? ix : gi;
        gpos = take ? (int)((rb[q] >> 21) & kIdxNone) : gpos;
        gsg = take ? (int)((rb[q] >> 42) & 1) : gsg;
      }
    }
    double vmax;
    int kmin;
    const int src = wave_first_max(gv, gi, vmax, kmin);
    if (lane == 0) {
      if (src < 0) {                              // no finite candidate: no exchange
        s_p = k + 1; s_posw = k + 1; s_alpha = T(NAN);
      } else {
        s_p = kmin;
        s_posw = __builtin_amdgcn_readlane(gpos, src);
        s_alpha = __builtin_amdgcn_readlane(gsg, src) ? -(T)vmax : (T)vmax;
      }
    }
  }
  __syncthreads();
}

// Both halves back to back.
template <typename T>
__device__ __forceinline__ void exchange_pivot(const PanelArgs& a, int s, int k, int wave, int lane, int w,
                                               const double* red_v, const uint64_t* red_k, int& s_p,
                                               int& s_posw, T& s_alpha, int& s_abort) {
  exchange_publish(a, s, wave, lane, w, red_v, red_k);
  exchange_collect<T>(a, s, k, wave, lane, s_p, s_posw, s_alpha, s_abort);
}

}  // namespace ltlt
