// Error compensation of the outlier branch (Sec. III-C2):
//   Y'[i][j] = s_j * sum_e r_ie * C_W[w(p_ie, j)].
// Each listed outlier channel p fetches input channel p of the weight codes
// (one contiguous row of words in the input-channel-major layout), the codes
// are dequantized with the weight codebook (the Dequant Unit) and multiplied
// by the residual (the MAC units), then merged into the main-branch output.
//
// One workgroup per (token, 64 output columns); its 4 waves split the token's
// 2k listed channels and are summed through LDS.  A lane owns one column and
// issues the word loads of 16 listed channels before using any of them, so
// the outlier stream costs a few memory latencies rather than one per
// outlier.  Channel ids and residuals are wave-uniform (scalar loads); zero
// residuals (channels already compensated through the max list) are skipped.
#include "common.h"

namespace oasis {

constexpr int CMP_COLS = 64;
constexpr int CMP_BATCH = 16;

__global__ void __launch_bounds__(256) k_compensate(CompArgs A) {
  __shared__ float cw[16];
  __shared__ float red[4][CMP_COLS];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid < 16) cw[tid] = h2f(A.lut->cb_wgt[tid]);
  const int i = blockIdx.x;
  const int j = blockIdx.y * CMP_COLS + lane;
  const int k = A.k, E = 2 * k;
  const int d_out = A.d_out, d_in = A.d_in;
  const size_t kr = (size_t)i * k;
  const float* res = A.residual + (size_t)i * E;
  // this wave's share of the listed channels
  const int per = (E + 3) / 4;
  const int e_beg = min(E, wave * per), e_end = min(E, e_beg + per);
  const bool col_ok = j < d_out;
  __syncthreads();

  float acc = 0.0f;
  for (int e0 = e_beg; e0 < e_end; e0 += CMP_BATCH) {
    int sh[CMP_BATCH];
    float r[CMP_BATCH];
    uint32_t w[CMP_BATCH];
#pragma unroll
    for (int u = 0; u < CMP_BATCH; ++u) {
      const int e = e0 + u;
      int p = -1;
      r[u] = 0.0f;
      if (e < e_end) {
        p = e < k ? A.max_idx[kr + e] : A.min_idx[kr + (e - k)];
        r[u] = res[e];
      }
      const bool live = p >= 0 && p < d_in && r[u] != 0.0f;  // wave-uniform
      if (!live) r[u] = 0.0f;
      sh[u] = live ? 4 * (p & 7) : 0;
      w[u] = 0u;
      if (live && col_ok) w[u] = A.idx_w[(size_t)(p >> 3) * d_out + j];
    }
#pragma unroll
    for (int u = 0; u < CMP_BATCH; ++u) acc += r[u] * cw[(w[u] >> sh[u]) & 15u];
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && col_ok) {
    const float v = A.w_scale[j] * (red[0][lane] + red[1][lane] + red[2][lane] + red[3][lane]);
    float* dst = A.y + (size_t)i * d_out + j;
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
  dim3 grid(a.n, (a.d_out + CMP_COLS - 1) / CMP_COLS);
  hipLaunchKernelGGL(k_compensate, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace oasis
