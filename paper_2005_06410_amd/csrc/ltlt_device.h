// Device-side helpers shared by the gfx950 kernels of the LTL^T library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ltlt {

constexpr int kWave = 64;            // CDNA wavefront width

// ---------------------------------------------------------------------------
// Coherent (agent-scope) relaxed accesses.  On gfx950 these compile to
// global loads/stores with the sc1 bit: they bypass the non-coherent part of
// the per-XCD L2, so data written this way by one workgroup is seen by any
// other workgroup that reads it this way, without the full-L2 writeback /
// invalidate that an agent-scope release/acquire fence costs.  Ordering
// between a workgroup's data stores and its later flag update comes from
// waiting for the stores to complete (s_waitcnt vmcnt(0)) before the flag.
// ---------------------------------------------------------------------------
__device__ __forceinline__ double ld_coh(const double* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_coh(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_coh(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wait_stores() {
  // vmcnt(0) expcnt(0) lgkmcnt(0): every earlier memory operation of this
  // wave has completed.
  __builtin_amdgcn_s_waitcnt(0);
}

// Wall clock for bounded device-side waits (constant 100 MHz counter).
__device__ __forceinline__ uint64_t wall_ticks() { return __builtin_amdgcn_s_memrealtime(); }
constexpr uint64_t kWaitLimitTicks = 200000000ull;   // 2 s at 100 MHz

// Bounded-wait status, two words per device:
//   status[0]  this call's abort flag: cleared when a call starts, raised when
//              one of its waits gives up; every later wait of the call gives up
//              at once, and the kernels that write results (commit, Pfaffian)
//              write NaN / sign 0 instead;
//   status[1]  sticky: raised together with status[0], cleared only when the
//              host reads it (ltlt_device_status), so a failed call is seen
//              even if later calls succeed.
__device__ __forceinline__ void raise_wait_status(int* status) {
  atomicOr(status, 1);
  atomicOr(status + 1, 1);
}

// (|value|, index) pair reduction: larger magnitude wins, ties go to the
// smaller index.  Magnitudes are compared as doubles (exact for fp32 input).
__device__ __forceinline__ void argmax_merge(double& bv, int& bi, double ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
}

__device__ __forceinline__ void wave_argmax(double& bv, int& bi) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    double ov = __shfl_xor(bv, off, kWave);
    int oi = __shfl_xor(bi, off, kWave);
    argmax_merge(bv, bi, ov, oi);
  }
}

// One DPP step of a wave-wide (|value|, index) max: every lane merges the
// pair of the lane selected by CTRL; lanes without a source (row edges,
// masked rows) merge the identity (-1, INT32_MAX).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void dpp_argmax_step(double& v, int& i) {
  const int lo = __double2loint(v), hi = __double2hiint(v);
  const int ilo = __double2loint(-1.0), ihi = __double2hiint(-1.0);
  const int olo = __builtin_amdgcn_update_dpp(ilo, lo, CTRL, ROW_MASK, 0xF, false);
  const int ohi = __builtin_amdgcn_update_dpp(ihi, hi, CTRL, ROW_MASK, 0xF, false);
  const int oi = __builtin_amdgcn_update_dpp(INT32_MAX, i, CTRL, ROW_MASK, 0xF, false);
  const double ov = __hiloint2double(ohi, olo);
  if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
}

// Wave-wide argmax through DPP row shifts and row broadcasts (no LDS
// permutes): the result is complete in lane 63 and returned to all lanes.
// Values must be >= -1 and not NaN (callers map NaN to -1: not a candidate).
__device__ __forceinline__ void wave_argmax_dpp(double& v, int& i) {
  dpp_argmax_step<0x111, 0xF>(v, i);   // row_shr:1
  dpp_argmax_step<0x112, 0xF>(v, i);   // row_shr:2
  dpp_argmax_step<0x114, 0xF>(v, i);   // row_shr:4
  dpp_argmax_step<0x118, 0xF>(v, i);   // row_shr:8   -> lane 15 of each row holds the row's result
  dpp_argmax_step<0x142, 0xA>(v, i);   // row_bcast:15 into rows 1 and 3
  dpp_argmax_step<0x143, 0xC>(v, i);   // row_bcast:31 into rows 2 and 3 -> lane 63 complete
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), 63);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), 63);
  v = __hiloint2double(hi, lo);
  i = __builtin_amdgcn_readlane(i, 63);
}

// ---------------------------------------------------------------------------
// Register-resident column refresh and first-maximum search, shared by the
// panel and the batched kernels.
// ---------------------------------------------------------------------------

// The 16 slots of one g register: acc[c % 4] += g(lane (lane & ~15) + c) * L[c0 + c]
// through v_fmac with a DPP row broadcast (row_newbcast, gfx950).  One asm
// block, led by the two wait states a DPP read needs after a VALU write of its
// source, so that no compiler-inserted copy of g can sit in between.
#define LTLT_FMAC16(OP)                                                                                  \
  asm volatile("s_nop 1\n"                                                                               \
               OP " %0, %4, %5 row_newbcast:0 row_mask:0xf bank_mask:0xf\n"                              \
               OP " %1, %4, %6 row_newbcast:1 row_mask:0xf bank_mask:0xf\n"                              \
               OP " %2, %4, %7 row_newbcast:2 row_mask:0xf bank_mask:0xf\n"                              \
               OP " %3, %4, %8 row_newbcast:3 row_mask:0xf bank_mask:0xf\n"                              \
               OP " %0, %4, %9 row_newbcast:4 row_mask:0xf bank_mask:0xf\n"                              \
               OP " %1, %4, %10 row_newbcast:5 row_mask:0xf bank_mask:0xf\n"                             \
               OP " %2, %4, %11 row_newbcast:6 row_mask:0xf bank_mask:0xf\n"                             \
               OP " %3, %4, %12 row_newbcast:7 row_mask:0xf bank_mask:0xf\n"                             \
               OP " %0, %4, %13 row_newbcast:8 row_mask:0xf bank_mask:0xf\n"                             \
               OP " %1, %4, %14 row_newbcast:9 row_mask:0xf bank_mask:0xf\n"                             \
               OP " %2, %4, %15 row_newbcast:10 row_mask:0xf bank_mask:0xf\n"                            \
               OP " %3, %4, %16 row_newbcast:11 row_mask:0xf bank_mask:0xf\n"                            \
               OP " %0, %4, %17 row_newbcast:12 row_mask:0xf bank_mask:0xf\n"                            \
               OP " %1, %4, %18 row_newbcast:13 row_mask:0xf bank_mask:0xf\n"                            \
               OP " %2, %4, %19 row_newbcast:14 row_mask:0xf bank_mask:0xf\n"                            \
               OP " %3, %4, %20 row_newbcast:15 row_mask:0xf bank_mask:0xf\n"                            \
               : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])                                  \
               : "v"(g), "v"(L[c0 + 0]), "v"(L[c0 + 1]), "v"(L[c0 + 2]), "v"(L[c0 + 3]), "v"(L[c0 + 4]), \
                 "v"(L[c0 + 5]), "v"(L[c0 + 6]), "v"(L[c0 + 7]), "v"(L[c0 + 8]), "v"(L[c0 + 9]),         \
                 "v"(L[c0 + 10]), "v"(L[c0 + 11]), "v"(L[c0 + 12]), "v"(L[c0 + 13]), "v"(L[c0 + 14]),    \
                 "v"(L[c0 + 15]))
template <int K, int NS>
__device__ __forceinline__ void refresh16(double (&acc)[4], double g, const double (&L)[NS]) {
  constexpr int c0 = 16 * K;
  LTLT_FMAC16("v_fmac_f64_dpp");
}
template <int K, int NS>
__device__ __forceinline__ void refresh16(float (&acc)[4], float g, const float (&L)[NS]) {
  constexpr int c0 = 16 * K;
  LTLT_FMAC16("v_fmac_f32_dpp");
}
#undef LTLT_FMAC16

// Wave-wide maximum of an unsigned key (every lane gets it): DPP row shifts
// and row broadcasts folded into v_max_u32 (a lane without a source is not
// written and keeps its key), two wait states before each DPP read; lane 63
// ends with the maximum.
__device__ __forceinline__ unsigned wave_umax(unsigned x) {
  asm volatile(
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 row_shr:1 row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 row_shr:2 row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 row_shr:4 row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 row_shr:8 row_mask:0xf bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
      "s_nop 1\n"
      "v_max_u32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
      "s_nop 1\n"
      : "+v"(x));
  return (unsigned)__builtin_amdgcn_readlane((int)x, 63);
}
// First maximum of (value, key) over the wave: the largest value, and among
// equal values the smallest key (then the lowest lane).  Values are >= 0 for
// candidates and -1 for lanes without one (NaN is never passed); keys are >= 0
// (INT32_MAX for no candidate).  The wave maximum is found on the high 32 bits
// of the value (order-preserving for non-negative doubles, +1 so that 0 means
// "no candidate").  Lanes that tie there are resolved exactly: when every
// tied value is +0 -- a stretch of zeros, which zero-structured input gives
// every wave at every step -- by one more wave reduction of the keys;
// otherwise (equal high words of nonzero values, rare) one lane at a time.
// A two-reduction form for every tie was measured slower on dense input: its
// code changes the schedule of the step loop around it.  Returns the winning
// lane (-1 when no lane has a candidate) and sets vmax / kmin to its value
// and key.
__device__ __forceinline__ int wave_first_max(double v, int key, double& vmax, int& kmin) {
  const unsigned hk = v >= 0.0 ? (unsigned)__double2hiint(v) + 1u : 0u;
  const unsigned mh = wave_umax(hk);
  if (mh == 0) { vmax = -1.0; kmin = INT32_MAX; return -1; }
  const bool tie_hi = hk == mh;
  unsigned long long hit = __ballot(tie_hi);
  int src = __ffsll(hit) - 1;
  unsigned blo = (unsigned)__builtin_amdgcn_readlane(__double2loint(v), src);
  kmin = __builtin_amdgcn_readlane(key, src);
  hit &= hit - 1;
  if (__builtin_expect(hit != 0, 0)) {
    if (mh == 1u && __ballot(tie_hi && __double2loint(v) != 0) == 0) {   // every tied value is +0
      kmin = (int)~wave_umax(tie_hi ? ~(unsigned)key : 0u);
      src = __ffsll(__ballot(tie_hi && key == kmin)) - 1;
    } else {
      while (hit) {
        const int l2 = __ffsll(hit) - 1;
        const unsigned lo2 = (unsigned)__builtin_amdgcn_readlane(__double2loint(v), l2);
        const int k2 = __builtin_amdgcn_readlane(key, l2);
        if (lo2 > blo || (lo2 == blo && k2 < kmin)) { blo = lo2; kmin = k2; src = l2; }
        hit &= hit - 1;
      }
    }
  }
  vmax = __hiloint2double((int)(mh - 1u), (int)blo);
  return src;
}

}  // namespace ltlt
