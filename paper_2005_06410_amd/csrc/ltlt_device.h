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

}  // namespace ltlt
