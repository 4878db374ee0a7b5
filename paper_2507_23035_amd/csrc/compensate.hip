// Error compensation of the outlier branch (Sec. III-C2):
//   Y'[i][j] = s_j * sum_e r_ie * C_W[w(p_ie, j)].
// Each listed outlier channel p fetches input channel p of the weight codes
// (one contiguous row of words in the input-channel-major layout), the codes
// are dequantized with the weight codebook (the Dequant Unit) and multiplied
// by the residual (the MAC units), then merged into the main-branch output.
//
// One workgroup per (token, 64 or 256 output columns); its 4 waves split the
// token's 2k listed channels and are summed through LDS.  A lane owns one or
// four columns and issues the word loads of 16 listed channels before using
// any of them, so the outlier stream costs a few memory latencies rather than
// one per outlier.  Channel ids and residuals are wave-uniform (scalar loads); zero
// residuals (channels already compensated through the max list) are skipped.
#include "common.h"

namespace oasis {

constexpr int CMP_BATCH = 16;

// CW output columns per lane (16-byte loads when CW == 4): WG = 64 * CW columns.
template <int CW>
__global__ void __launch_bounds__(256) k_compensate(CompArgs A) {
  __shared__ float cw[16];
  __shared__ float red[4][64 * CW];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  if (tid < 16) cw[tid] = h2f(A.lut->cb_wgt[tid]);
  const int i = blockIdx.x;
  const int j = blockIdx.y * 64 * CW + CW * lane;
  const int k = A.k, E = 2 * k;
  const int d_out = A.d_out, d_in = A.d_in;
  const size_t kr = (size_t)i * k;
  const float* res = A.residual + (size_t)i * E;
  // this wave's share of the listed channels
  const int per = (E + 3) / 4;
  const int e_beg = min(E, wave * per), e_end = min(E, e_beg + per);
  const bool vec_ok = CW == 4 && (d_out & 3) == 0 && j + 3 < d_out;
  __syncthreads();

  float acc[CW];
#pragma unroll
  for (int c = 0; c < CW; ++c) acc[c] = 0.0f;
  for (int e0 = e_beg; e0 < e_end; e0 += CMP_BATCH) {
    int sh[CMP_BATCH];
    float r[CMP_BATCH];
    uint32_t w[CMP_BATCH][CW];
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
#pragma unroll
      for (int c = 0; c < CW; ++c) w[u][c] = 0u;
      if (live) {
        const uint32_t* row = A.idx_w + (size_t)(p >> 3) * d_out;
        if (vec_ok) {
          const uint4_t v = *reinterpret_cast<const uint4_t*>(row + j);
#pragma unroll
          for (int c = 0; c < CW; ++c) w[u][c] = v[c];
        } else {
#pragma unroll
          for (int c = 0; c < CW; ++c)
            if (j + c < d_out) w[u][c] = row[j + c];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < CMP_BATCH; ++u)
#pragma unroll
      for (int c = 0; c < CW; ++c) acc[c] += r[u] * cw[(w[u][c] >> sh[u]) & 15u];
  }
#pragma unroll
  for (int c = 0; c < CW; ++c) red[wave][CW * lane + c] = acc[c];
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      const int jj = j + c;
      if (jj >= d_out) continue;
      const int q = CW * lane + c;
      const float v = A.w_scale[jj] * (red[0][q] + red[1][q] + red[2][q] + red[3][q]);
      float* dst = A.y + (size_t)i * d_out + jj;
      *dst = A.accumulate ? *dst + v : v;
    }
  }
}

hipError_t launch_compensate(const CompArgs& a, hipStream_t s) {
  if (a.n == 0 || a.d_out == 0) return hipSuccess;
  if (a.k == 0) {
    if (a.accumulate) return hipSuccess;
    return launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
  }
  // few tokens: one column per lane for more workgroups; many: 16-byte loads
  if (a.n <= 64) {
    dim3 grid(a.n, (a.d_out + 63) / 64);
    hipLaunchKernelGGL(k_compensate<1>, grid, dim3(256), 0, s, a);
  } else {
    dim3 grid(a.n, (a.d_out + 255) / 256);
    hipLaunchKernelGGL(k_compensate<4>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace oasis
