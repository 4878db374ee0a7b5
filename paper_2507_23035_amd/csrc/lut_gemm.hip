// Look-ahead WAQ LUT-GEMM, the main branch of Sec. III-C1:
//   Y*[i][j] = t_i * s_j * sum_p LUT[(a_ip << b_w) | w_pj].
//
// Two kernels compute it.
//
// k_gemm_lut: the scheme of Sec. III-B taken literally - every (token,
// channel, column) triple concatenates its two codes and adds the LUT entry
// they select.  The 1 KB LUT is replicated in LDS (one copy per bank of a
// half-wave) so 32 lanes gathering different entries never collide.
//
// k_gemm_mfma_*: the LUT is the outer product of the two codebooks
// (entry (a, w) = C_A[a] * C_W[w]), so the sum over p is the dense
// contraction sum_p C_A[a_ip] * C_W[w_pj] of exact fp16 centroid values.
// Codes are expanded to those fp16 values in registers (a byte of two codes
// selects a packed pair from a 256-entry LDS table) and fed to
// v_mfma_f32_16x16x32_f16.  Every product equals its LUT entry bit for bit;
// only the fp32 summation order differs from the literal scheme.
//
// MFMA operand mapping (16x16x32): A = weight codes (row m = output column),
// B = activation codes (column = token).  Lane (g, m), g = lane / 16, holds the
// 8 codes of one 32-bit word.  Within a block of 16 words (128 channels) lane
// group g and step s use word 4g + s on both sides, so the weight rows are read
// as full 256-byte segments and each token's 4 words as one 16-byte load; the
// order in which channels enter the MFMA is irrelevant to the sum.
#include "common.h"

namespace oasis {

// ----------------------------------------------------------------------------
// shared helpers
// ----------------------------------------------------------------------------
constexpr int DEC_R = 8;  // replication of the byte -> fp16 pair tables

// byte b -> (C[b & 15] | C[b >> 4] << 16): the two fp16 centroids of its codes
__device__ __forceinline__ void build_pair_table(uint32_t* tab, const uint16_t* cb, int tid,
                                                 int nthreads) {
  for (int e = tid; e < 256 * DEC_R; e += nthreads) {
    const int b = e / DEC_R;
    tab[e] = (uint32_t)cb[b & 15] | ((uint32_t)cb[b >> 4] << 16);
  }
}

__device__ __forceinline__ half8_t expand_word(uint32_t w, const uint32_t* tab, int lane_off) {
  uint4_t r;
  r[0] = tab[((w >> 0) & 0xFFu) * DEC_R + lane_off];
  r[1] = tab[((w >> 8) & 0xFFu) * DEC_R + lane_off];
  r[2] = tab[((w >> 16) & 0xFFu) * DEC_R + lane_off];
  r[3] = tab[((w >> 24) & 0xFFu) * DEC_R + lane_off];
  return __builtin_bit_cast(half8_t, r);
}

__device__ __forceinline__ uint4_t load_w4(const uint32_t* __restrict__ idx_w, size_t row_off,
                                           int j, int d_out, bool vec_ok) {
  uint4_t v = {0u, 0u, 0u, 0u};
  const uint32_t* p = idx_w + row_off + j;
  if (vec_ok && j + 3 < d_out) {
    v = *reinterpret_cast<const uint4_t*>(p);
  } else {
    if (j + 0 < d_out) v[0] = p[0];
    if (j + 1 < d_out) v[1] = p[1];
    if (j + 2 < d_out) v[2] = p[2];
    if (j + 3 < d_out) v[3] = p[3];
  }
  return v;
}

// The 16-column x 16-token MFMA tiles of one wave: CG groups of 64 columns
// (4 tiles each) by TF groups of 16 tokens.  Runs the blocks of 16 words in
// [blk_begin, blk_end) with a stride, accumulating into acc.
template <int CG, int TF>
__device__ __forceinline__ void mfma_blocks(const GemmArgs& A, int j0, int tok0, int blk_begin,
                                            int blk_end, int blk_stride, const uint32_t* tabW,
                                            const uint32_t* tabA,
                                            float4_t (&acc)[CG * 4][TF]) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, m = lane & 15;
  const int lane_off = lane & (DEC_R - 1);
  const int KB = A.d_in >> 3;
  const int d_out = A.d_out;
  const bool vec_ok = (d_out & 3) == 0;
  const size_t arow_words = (size_t)(A.d_in >> 3);
  const uint32_t* aw = reinterpret_cast<const uint32_t*>(A.idx_act);

  for (int blk = blk_begin; blk < blk_end; blk += blk_stride) {
    const int kw0 = blk * 16 + 4 * g;  // this lane group's first word in the block
    // activation words of this lane's tokens: 4 consecutive words, one per step
    uint4_t av[TF];
#pragma unroll
    for (int f = 0; f < TF; ++f) {
      const int tok = tok0 + 16 * f + m;
      av[f] = uint4_t{0u, 0u, 0u, 0u};
      if (tok < A.n) {
        const uint32_t* src = aw + (size_t)tok * arow_words + kw0;
        if (kw0 + 3 < KB && (arow_words & 3) == 0) {
          av[f] = *reinterpret_cast<const uint4_t*>(src);
        } else {
#pragma unroll
          for (int s = 0; s < 4; ++s)
            if (kw0 + s < KB) av[f][s] = src[s];
        }
      }
    }
    // weight words: 4 rows (steps) x CG*4 columns for this lane
    uint4_t wv[4][CG];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int kw = kw0 + s;
#pragma unroll
      for (int h = 0; h < CG; ++h) {
        if (kw < KB)
          wv[s][h] = load_w4(A.idx_w, (size_t)kw * d_out, j0 + 64 * h + 4 * m, d_out, vec_ok);
        else
          wv[s][h] = uint4_t{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bool live = (kw0 + s) < KB;  // words past the end contribute nothing
      half8_t bf[TF];
#pragma unroll
      for (int f = 0; f < TF; ++f) {
        bf[f] = expand_word(av[f][s], tabA, lane_off);
        const bool tok_ok = (tok0 + 16 * f + m) < A.n;
        if (!(live && tok_ok)) bf[f] = half8_t{0, 0, 0, 0, 0, 0, 0, 0};
      }
#pragma unroll
      for (int h = 0; h < CG; ++h) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const half8_t af = expand_word(wv[s][h][c], tabW, lane_off);
#pragma unroll
          for (int f = 0; f < TF; ++f)
            acc[4 * h + c][f] =
                __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf[f], acc[4 * h + c][f], 0, 0, 0);
        }
      }
    }
  }
}

// Output of tile (4h + c, f): lane (g, tc) holds rows m = 4g + r, i.e. output
// columns j0 + 64h + 16g + 4r + c of token tok0 + 16f + tc.
__device__ __forceinline__ void store_out(const GemmArgs& A, int tok, int j, float v, bool atomic) {
  if (tok >= A.n || j >= A.d_out) return;
  float* dst = A.y + (size_t)tok * A.d_out + j;
  const float val = A.act_scale[tok] * A.w_scale[j] * v;
  if (atomic)
    atomicAdd(dst, val);
  else if (A.accumulate)
    *dst += val;
  else
    *dst = val;
}

// ----------------------------------------------------------------------------
// MFMA kernel, decode tiling: 4 waves share 64 columns and split the words of
// the WG's input-channel slice; gridDim.z slices are merged with atomics.
// ----------------------------------------------------------------------------
template <int TF>
__global__ void __launch_bounds__(256) k_gemm_mfma_decode(GemmArgs A, int blk_per_split) {
  __shared__ uint32_t tabW[256 * DEC_R];
  __shared__ uint32_t tabA[256 * DEC_R];
  __shared__ float4_t red[4][4 * TF][64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  build_pair_table(tabW, A.lut->cb_wgt, tid, 256);
  build_pair_table(tabA, A.lut->cb_act, tid, 256);
  __syncthreads();

  const int j0 = blockIdx.x * 64;
  const int nblk = (A.d_in / 8 + 15) / 16;
  const int b0 = blockIdx.z * blk_per_split;
  const int b1 = min(nblk, b0 + blk_per_split);

  float4_t acc[4][TF];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int f = 0; f < TF; ++f) acc[c][f] = float4_t{0.f, 0.f, 0.f, 0.f};

  mfma_blocks<1, TF>(A, j0, 0, b0 + wave, b1, 4, tabW, tabA, acc);

#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int f = 0; f < TF; ++f) red[wave][c * TF + f][lane] = acc[c][f];
  __syncthreads();

  const bool atomic = gridDim.z > 1;
  const int g = lane >> 4, tc = lane & 15;
  for (int t = wave; t < 4 * TF; t += 4) {
    float4_t v = red[0][t][lane] + red[1][t][lane] + red[2][t][lane] + red[3][t][lane];
    const int c = t / TF, f = t % TF;
    const int tok = 16 * f + tc;
#pragma unroll
    for (int r = 0; r < 4; ++r) store_out(A, tok, j0 + 16 * g + 4 * r + c, v[r], atomic);
  }
}

// ----------------------------------------------------------------------------
// MFMA kernel, prefill tiling: 2 x 2 waves, each 64 columns x 64 tokens, over
// the whole reduction; WG tile 128 columns x 128 tokens.
// ----------------------------------------------------------------------------
constexpr int PF_TF = 4;

__global__ void __launch_bounds__(256) k_gemm_mfma_prefill(GemmArgs A) {
  __shared__ uint32_t tabW[256 * DEC_R];
  __shared__ uint32_t tabA[256 * DEC_R];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  build_pair_table(tabW, A.lut->cb_wgt, tid, 256);
  build_pair_table(tabA, A.lut->cb_act, tid, 256);
  __syncthreads();

  const int j0 = blockIdx.x * 128 + (wave & 1) * 64;
  const int tok0 = blockIdx.y * 128 + (wave >> 1) * 64;
  const int nblk = (A.d_in / 8 + 15) / 16;

  float4_t acc[4][PF_TF];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int f = 0; f < PF_TF; ++f) acc[c][f] = float4_t{0.f, 0.f, 0.f, 0.f};

  if (j0 < A.d_out && tok0 < A.n)
    mfma_blocks<1, PF_TF>(A, j0, tok0, 0, nblk, 1, tabW, tabA, acc);

  const int g = lane >> 4, tc = lane & 15;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int f = 0; f < PF_TF; ++f)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        store_out(A, tok0 + 16 * f + tc, j0 + 16 * g + 4 * r + c, acc[c][f][r], false);
}

hipError_t launch_gemm_mfma(const GemmArgs& a, hipStream_t s) {
  const int KB = a.d_in / 8;
  const int nblk = (KB + 15) / 16;
  if (a.n <= 32) {
    const int ct = (a.d_out + 63) / 64;
    int split = (2048 + ct - 1) / ct;
    split = min(split, max(1, nblk / 4));
    split = max(1, split);
    int bps = (nblk + split - 1) / split;
    split = (nblk + bps - 1) / bps;
    if (split > 1 && !a.accumulate) {
      hipError_t e = launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
      if (e != hipSuccess) return e;
    }
    dim3 grid(ct, 1, max(1, split));
    if (a.n <= 16)
      hipLaunchKernelGGL(k_gemm_mfma_decode<1>, grid, dim3(256), 0, s, a, max(1, bps));
    else
      hipLaunchKernelGGL(k_gemm_mfma_decode<2>, grid, dim3(256), 0, s, a, max(1, bps));
  } else {
    dim3 grid((a.d_out + 127) / 128, (a.n + 127) / 128, 1);
    hipLaunchKernelGGL(k_gemm_mfma_prefill, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Literal LUT kernel: one LDS lookup per (token, channel, column).
// WG = 4 waves over 64 columns and LUT_TN tokens; the waves interleave the
// words of the WG's input-channel slice and are reduced through LDS.
// ----------------------------------------------------------------------------
constexpr int LUT_R = 32;   // LUT copies: lane l of a half-wave reads copy l
constexpr int LUT_TN = 8;   // tokens per WG

__global__ void __launch_bounds__(256) k_gemm_lut(GemmArgs A, int words_per_split) {
  __shared__ float lut_s[256 * LUT_R];
  __shared__ float red[4][LUT_TN][64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int e = tid; e < 256 * LUT_R; e += 256) lut_s[e] = A.lut->lut[e / LUT_R];
  __syncthreads();

  const int j = blockIdx.x * 64 + lane;
  const int tok0 = blockIdx.y * LUT_TN;
  const int ntok = min(LUT_TN, A.n - tok0);
  const int KB = A.d_in >> 3;
  const int w0 = blockIdx.z * words_per_split;
  const int w1 = min(KB, w0 + words_per_split);
  const int b_w = A.b_w;
  const int copy = lane & (LUT_R - 1);
  const uint32_t* aw = reinterpret_cast<const uint32_t*>(A.idx_act);
  const size_t arow = (size_t)KB;

  float acc[LUT_TN];
#pragma unroll
  for (int t = 0; t < LUT_TN; ++t) acc[t] = 0.f;

  if (j < A.d_out) {
    for (int kw = w0 + wave; kw < w1; kw += 4) {
      const uint32_t w = A.idx_w[(size_t)kw * A.d_out + j];
      int woff[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) woff[e] = (int)((w >> (4 * e)) & 15u) * LUT_R + copy;
#pragma unroll
      for (int t = 0; t < LUT_TN; ++t) {
        if (t < ntok) {
          const uint32_t a = aw[(size_t)(tok0 + t) * arow + kw];  // same for the whole wave
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int concat_hi = (int)((a >> (4 * e)) & 15u) << b_w;  // (a << b_w) | w
            acc[t] += lut_s[concat_hi * LUT_R + woff[e]];
          }
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < LUT_TN; ++t) red[wave][t][lane] = acc[t];
  __syncthreads();
  const bool atomic = gridDim.z > 1;
  for (int t = wave; t < LUT_TN; t += 4) {
    const float v = red[0][t][lane] + red[1][t][lane] + red[2][t][lane] + red[3][t][lane];
    if (t < ntok) store_out(A, tok0 + t, j, v, atomic);
  }
}

hipError_t launch_gemm_lut(const GemmArgs& a, hipStream_t s) {
  const int KB = a.d_in / 8;
  const int ct = (a.d_out + 63) / 64;
  const int tt = (a.n + LUT_TN - 1) / LUT_TN;
  int split = (1024 + ct * tt - 1) / (ct * tt);
  split = max(1, min(split, KB / 16));
  int wps = (KB + split - 1) / split;
  wps = max(1, wps);
  split = max(1, (KB + wps - 1) / wps);
  if (split > 1 && !a.accumulate) {
    hipError_t e = launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
    if (e != hipSuccess) return e;
  }
  dim3 grid(ct, tt, split);
  hipLaunchKernelGGL(k_gemm_lut, grid, dim3(256), 0, s, a, wps);
  return hipGetLastError();
}

}  // namespace oasis
