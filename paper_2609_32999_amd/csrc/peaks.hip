// Measurement aids: kernels that show the achievable matrix-core and memory
// rates of the running GPU.  They are not part of the composed-prefill path;
// the benchmark reports their rates next to the published peaks, so that a
// kernel's fraction of peak can also be read against what this GPU sustains
// at the clock it holds under load.
#include <hip/hip_runtime.h>

#include "kernels_common.h"
#include "tsr_internal.h"
#include "../../include/tsr_measure.h"

namespace tsr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kPeakThreads = 256;
constexpr int kChains = 8;   // independent accumulators: no MFMA waits on another

// Back-to-back v_mfma_f32_32x32x16_bf16 on register operands, no memory
// traffic in the loop.  Each wave issues iters * kChains MFMAs.
__global__ __launch_bounds__(kPeakThreads) void peak_mfma_kernel(float* out, int iters) {
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1.0f + 0.001f * (threadIdx.x & 7));
    b[e] = (__bf16)(0.5f - 0.01f * e);
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[(size_t)blockIdx.x * kPeakThreads + threadIdx.x] = s;
}

// Grid-stride copy, 16 bytes per lane per access.
__global__ __launch_bounds__(kPeakThreads) void peak_copy_kernel(const uint4* __restrict__ src,
                                                                 uint4* __restrict__ dst,
                                                                 size_t n) {
  const size_t stride = (size_t)gridDim.x * kPeakThreads;
  for (size_t i = (size_t)blockIdx.x * kPeakThreads + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

}  // namespace

}  // namespace tsr

extern "C" {

int64_t tsr_peak_mfma_flops(int32_t n_workgroups, int32_t iters) {
  if (n_workgroups <= 0 || iters <= 0) return 0;
  return (int64_t)n_workgroups * (tsr::kPeakThreads / 64) * iters * tsr::kChains *
         (2LL * 32 * 32 * 16);
}

tsr_status tsr_peak_mfma(int32_t n_workgroups, int32_t iters, float* dev_out, void* stream) {
  if (n_workgroups <= 0 || iters <= 0 || dev_out == nullptr) {
    tsr::set_error("peak_mfma: n_workgroups and iters must be positive and dev_out non-NULL");
    return TSR_ERR_INVALID_ARG;
  }
  hipLaunchKernelGGL(tsr::peak_mfma_kernel, dim3(n_workgroups), dim3(tsr::kPeakThreads), 0,
                     static_cast<hipStream_t>(stream), dev_out, iters);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tsr::device_fail("peak_mfma launch", e);
  return TSR_OK;
}

tsr_status tsr_peak_copy(void* dst, const void* src, size_t bytes, void* stream) {
  if (dst == nullptr || src == nullptr || bytes == 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) % 16 != 0) {
    tsr::set_error("peak_copy: pointers must be non-NULL and 16-byte aligned, bytes a "
                   "positive multiple of 16");
    return TSR_ERR_INVALID_ARG;
  }
  const size_t n = bytes / 16;
  const size_t want = (n + tsr::kPeakThreads - 1) / tsr::kPeakThreads;
  const int grid = (int)(want < 8192 ? want : 8192);
  hipLaunchKernelGGL(tsr::peak_copy_kernel, dim3(grid), dim3(tsr::kPeakThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint4*>(src),
                     static_cast<uint4*>(dst), n);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tsr::device_fail("peak_copy launch", e);
  return TSR_OK;
}

}  // extern "C"
