// Plain device copy used as the reference kernel for hardware byte counters:
// it reads and writes exactly `bytes` bytes, so FETCH_SIZE / WRITE_SIZE of any
// other kernel can be scaled to bytes by comparing with this one.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gspn.h"

namespace {

__global__ void __launch_bounds__(256) gspn_copy_calibration_kernel(const uint4* __restrict__ src,
                                                                   uint4* __restrict__ dst, size_t n16,
                                                                   const uint8_t* __restrict__ s8,
                                                                   uint8_t* __restrict__ d8, size_t tail) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) dst[i] = src[i];
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < tail; i += stride) d8[i] = s8[i];
}

}  // namespace

extern "C" int gspn_copy_calibration(const void* src, void* dst, size_t bytes, void* stream) {
  if (bytes == 0) return GSPN_OK;
  if (!src || !dst) return GSPN_ERR_NULL;
  const uintptr_t s = (uintptr_t)src, d = (uintptr_t)dst;
  if (s < d + bytes && d < s + bytes) return GSPN_ERR_ALIAS;
  if (s % 16 || d % 16) return GSPN_ERR_ALIGN;
  const size_t n16 = bytes / 16, tail = bytes - n16 * 16;
  // four workgroups per compute unit, each striding over the buffer: the
  // fastest copy shape measured on MI355X (more workgroups lose write bandwidth)
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks == 0) blocks = 1;
  hipLaunchKernelGGL(gspn_copy_calibration_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     (hipStream_t)stream, (const uint4*)src, (uint4*)dst, n16,
                     (const uint8_t*)src + n16 * 16, (uint8_t*)dst + n16 * 16, tail);
  return hipGetLastError() == hipSuccess ? GSPN_OK : GSPN_ERR_HIP;
}
