// Measured matrix-core rate of this device: every wave runs a register-only
// loop of 16 independent 16x16x4 MFMAs (fp64 v_mfma_f64_16x16x4_f64, or fp32
// v_mfma_f32_16x16x4_f32), accumulating in VGPRs, with two workgroups of four
// waves per CU.  Nothing else is executed, so the rate is the ceiling that
// the trailing update's MFMA loop can approach here; it is reported next to
// the published peak.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ltlt.h"
#include "ltlt_internal.h"

namespace ltlt {
namespace {

typedef double v4d __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;

template <typename T> struct ProbeMfma;
template <> struct ProbeMfma<double> {
  typedef v4d acc_t;
  static __device__ __forceinline__ acc_t run(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
};
template <> struct ProbeMfma<float> {
  typedef v4f acc_t;
  static __device__ __forceinline__ acc_t run(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

template <typename T>
__global__ void __launch_bounds__(kProbeThreads, 2) mfma_loop_kernel(T* out, int iters) {
  typedef typename ProbeMfma<T>::acc_t acc_t;
  const int tid = threadIdx.x;
  T a[4], b[4];
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    a[x] = T(1e-3) * T(tid + x);
    b[x] = T(1e-3) * T(tid - x);
  }
  acc_t acc[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) acc[x][y] = acc_t{0, 0, 0, 0};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) acc[x][y] = ProbeMfma<T>::run(a[x], b[y], acc[x][y]);
  }
  T s = T(0);
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) s += acc[x][y][0] + acc[x][y][3];
  out[(size_t)blockIdx.x * kProbeThreads + tid] = s;   // keeps the loop live
}

template <typename T>
int run_probe(int64_t iters, double* tflops, hipStream_t s) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return LTLT_ERR_HIP_BASE - (int)e;
  const int grid = 2 * cus;
  T* out = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float ms = 0.0f;
  e = hipMalloc(&out, (size_t)grid * kProbeThreads * sizeof(T));
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) {   // untimed warm-up launch
    hipLaunchKernelGGL(mfma_loop_kernel<T>, dim3(grid), dim3(kProbeThreads), 0, s, out, (int)(iters / 8 + 1));
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(mfma_loop_kernel<T>, dim3(grid), dim3(kProbeThreads), 0, s, out, (int)iters);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);                // cleanup: the first error is the one reported
  if (e1) (void)hipEventDestroy(e1);
  if (out) (void)hipFree(out);
  if (e != hipSuccess) return LTLT_ERR_HIP_BASE - (int)e;
  // 4 waves per workgroup, 16 MFMAs per iteration, 2*16*16*4 flops each
  const double flops = (double)grid * 4.0 * (double)iters * 16.0 * 2048.0;
  *tflops = ms > 0.0f ? flops / ((double)ms * 1e-3) / 1e12 : 0.0;
  return LTLT_OK;
}

}  // namespace
}  // namespace ltlt

extern "C" int ltlt_mfma_probe(int dtype, int64_t iters, double* tflops, hipStream_t stream) {
  if (dtype != LTLT_F64 && dtype != LTLT_F32) return -1;
  if (iters < 1 || iters > 100000000) return -2;
  if (tflops == nullptr) return -3;
  return dtype == LTLT_F64 ? ltlt::run_probe<double>(iters, tflops, stream)
                           : ltlt::run_probe<float>(iters, tflops, stream);
}
