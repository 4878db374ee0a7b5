// Cartesian product LUT of the activation and weight codebooks (Sec. III-B).
// The accelerator keeps the products and both codebooks in its on-chip LUT
// (Sec. IV-A); the LUT block mirrors that: 256 fp32 products + C_A + C_W.
#include "common.h"

namespace oasis {

__global__ void __launch_bounds__(256) k_build_lut(Codebooks cb, int b_a, int b_w,
                                                   oasis_lut_block* __restrict__ out) {
  write_lut_entry(cb, b_a, b_w, threadIdx.x, out);  // one entry per thread, 256 threads
}

hipError_t launch_build_lut(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                            oasis_lut_block* out, hipStream_t s) {
  Codebooks cb = {};
  for (int i = 0; i < (1 << b_a); ++i) cb.act[i] = cb_act[i];
  for (int i = 0; i < (1 << b_w); ++i) cb.wgt[i] = cb_wgt[i];
  hipLaunchKernelGGL(k_build_lut, dim3(1), dim3(256), 0, s, cb, b_a, b_w, out);
  return hipGetLastError();
}

__global__ void __launch_bounds__(256) k_fill_zero(float* __restrict__ y, size_t count) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < count; i += stride) y[i] = 0.0f;
}

hipError_t launch_fill_zero(float* y, size_t count, hipStream_t s) {
  if (count == 0) return hipSuccess;
  size_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, s, y, count);
  return hipGetLastError();
}

}  // namespace oasis
