// Error compensation of the outlier branch (Sec. III-C2):
//   Y'[i][j] = s_j * sum_e r_ie * C_W[w(p_ie, j)].
// Each listed outlier channel p fetches input channel p of the weight codes
// (one contiguous row of words in the input-channel-major layout), the codes
// are dequantized with the weight codebook (the Dequant Unit) and multiplied
// by the residual (the MAC units), then merged into the main-branch output.
//
// One workgroup per (token, 256 output columns); the token's channel ids and
// residuals are wave-uniform, so they travel through scalar loads, and
// zero residuals (channels compensated through the max list already) are
// skipped.
#include "common.h"

namespace oasis {

constexpr int CT = 256;

__global__ void __launch_bounds__(CT) k_compensate(CompArgs A) {
  __shared__ float cw[16];
  const int tid = threadIdx.x;
  if (tid < 16) cw[tid] = h2f(A.lut->cb_wgt[tid]);
  __syncthreads();
  const int j = blockIdx.y * CT + tid;
  const int i = blockIdx.x;
  const int k = A.k;
  const int d_out = A.d_out;
  const size_t kr = (size_t)i * k;
  const float* res = A.residual + (size_t)i * 2 * k;
  float acc = 0.0f;
  if (j < d_out) {
    for (int e = 0; e < 2 * k; ++e) {
      const float r = res[e];
      const int p = e < k ? A.max_idx[kr + e] : A.min_idx[kr + (e - k)];
      if (r == 0.0f || p < 0 || p >= A.d_in) continue;  // uniform branch
      const uint32_t w = A.idx_w[(size_t)(p >> 3) * d_out + j];
      const uint32_t code = (w >> (4 * (p & 7))) & 15u;
      acc += r * cw[code];
    }
    float* dst = A.y + (size_t)i * d_out + j;
    const float v = A.w_scale[j] * acc;
    if (A.accumulate)
      *dst += v;
    else
      *dst = v;
  }
}

hipError_t launch_compensate(const CompArgs& a, hipStream_t s) {
  if (a.n == 0 || a.d_out == 0) return hipSuccess;
  if (a.k == 0) {
    if (a.accumulate) return hipSuccess;
    return launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
  }
  dim3 grid(a.n, (a.d_out + CT - 1) / CT);
  hipLaunchKernelGGL(k_compensate, grid, dim3(CT), 0, s, a);
  return hipGetLastError();
}

}  // namespace oasis
