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

}  // namespace ltlt
