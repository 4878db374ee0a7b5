// Internal helpers shared by the OASIS HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oasis.h"

namespace oasis {

constexpr int kWave = 64;

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef uint32_t uint4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float h2f(uint16_t bits) {
  return (float)__builtin_bit_cast(_Float16, bits);
}

// Workgroups are dealt to the 8 XCDs round-robin (id mod 8).  Map ids so that
// each XCD gets a contiguous range of tiles and neighbouring tiles share its
// L2.  A bijection on [0, T).
__device__ __forceinline__ int xcd_tile(int b, int T) {
  const int per = T >> 3;
  return b < 8 * per ? (b & 7) * per + (b >> 3) : b;
}

// Inclusive prefix sum over the 64 lanes of a wave, with DPP lane moves:
// Hillis-Steele inside each row of 16 lanes, then the row totals broadcast
// to the rows above (lanes outside a row or outside the row mask add 0).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0u, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0u, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Maximum over the wave (same lane moves), returned in every lane.
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x111, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x112, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x114, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x118, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x142, 0xA, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0u, v, 0x143, 0xC, 0xF, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Sum over aligned groups of P consecutive lanes (P = 1, 2, 4 or 8, the same
// in every lane); every lane of a group receives the group's sum.
__device__ __forceinline__ uint32_t group_sum(uint32_t v, uint32_t P) {
  if (P >= 2u) v += __builtin_amdgcn_update_dpp(0u, v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  if (P >= 4u) v += __builtin_amdgcn_update_dpp(0u, v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  if (P >= 8u) v += __builtin_amdgcn_update_dpp(0u, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  return v;
}

// Inclusive scan of one 64-bit value per thread over the block (NT threads).
// Each call needs its own `tmp` (NT / 64 words): there is no trailing barrier.
template <int NT>
__device__ __forceinline__ uint64_t block_scan64(uint64_t v, uint64_t* tmp) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    uint64_t u = __shfl_up(v, off, 64);
    if (lane >= off) v += u;
  }
  if (lane == 63) tmp[wid] = v;
  __syncthreads();
  uint64_t base = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w)
    if (w < wid) base += tmp[w];
  return v + base;
}
// Everything the host launchers need; argument checking happens in api.cpp.
// Codebooks by value (fp16 bits; entries past 2^b are 0).
struct Codebooks {
  uint16_t act[16];
  uint16_t wgt[16];
};

// Entry e (< 256) of the LUT block: lut[e] = fp32(C_A[e >> b_w]) *
// fp32(C_W[e mod 2^b_w]), 0 past 2^(b_a + b_w); for e < 16 also both
// codebook entries.  A product of two fp16 values has at most 22 significant
// bits, so it is exact in fp32.
__device__ __forceinline__ void write_lut_entry(const Codebooks& cb, int b_a, int b_w, int e,
                                                oasis_lut_block* out) {
  float v = 0.0f;
  if (e < (1 << (b_a + b_w))) v = h2f(cb.act[e >> b_w]) * h2f(cb.wgt[e & ((1 << b_w) - 1)]);
  out->lut[e] = v;
  if (e < 16) {
    out->cb_act[e] = e < (1 << b_a) ? cb.act[e] : (uint16_t)0;
    out->cb_wgt[e] = e < (1 << b_w) ? cb.wgt[e] : (uint16_t)0;
  }
}

struct QuantArgs {
  const uint16_t* x;
  int n, d_in, b_a, k, scale_mode;
  const oasis_lut_block* lut;
  uint8_t* idx_act;
  float* act_scale;
  int32_t* max_idx;
  int32_t* min_idx;
  float* residual;
  // LUT build in the same launch: when lut_out is set, C_A comes from cb and
  // workgroup 0 also writes the LUT block (lut is not read)
  oasis_lut_block* lut_out;
  Codebooks cb;
  int b_w;
  // OASIS-S: outliers are x >= thr_hi and x <= thr_lo (k = places per side)
  int static_thr;
  float thr_hi, thr_lo;
};

struct GemmArgs {
  const uint8_t* idx_act;
  const float* act_scale;
  int n, d_in;
  const uint32_t* idx_w;
  const float* w_scale;
  int d_out;
  const oasis_lut_block* lut;
  int b_a, b_w;
  float* y;
  int accumulate;
  // optional outlier lists: when k > 0 the GEMM also adds the compensation
  const int32_t* max_idx;
  const int32_t* min_idx;
  const float* residual;
  int k;
  // optional: the codes in the row layout ([d_in][ceil(d_out/8)] words); when
  // set, the compensation reads its rows from here (0.5 B per outlier and column)
  const uint32_t* idx_wr;
  // optional: per-output-channel weight codebooks, fp16 [d_out][16]; when set
  // they replace the LUT block's C_W (GEMV kernel only)
  const uint16_t* cb_cols;
  // value operand (many-token kernel only): the B operand is an fp16 matrix
  // [n][a_row / 2] (idx_act holds its bytes) instead of activation codes, and
  // the reduction runs over ceil(2 * *kdyn / 64) blocks of 64 positions (a
  // length known on the device only)
  const int* kdyn;
  int a_row;  // bytes per row of that matrix
  // optional (many-token kernel): after the main reduction, ceil(2 * *nheavy /
  // 64) more blocks with the fp16 value operand hv ([n] rows of 2 * kSplitPos
  // bytes) and the weight codes hw (GEMM layout, kSplitPos / 8 rows)
  const int* nheavy;
  const uint8_t* hv;
  const uint32_t* hw;
};

struct CompArgs {
  const int32_t* max_idx;
  const int32_t* min_idx;
  const float* residual;
  int n, k;
  const uint32_t* idx_w;
  const oasis_lut_block* lut;
  int b_w;
  const float* w_scale;
  int d_in, d_out;
  float* y;
  int accumulate;
  // optional: compacted lists (row-layout kernel only): token i's live entries
  // are max_idx[i][0..cnt[i]) (channels) and residual[i][0..cnt[i]), in list
  // order, each row 2k long; min_idx is not read
  const int32_t* cnt;
};

// Heavy / sparse split of the compensation for many tokens: channels listed
// by at least one token in eight (at most kSplitHeavy of them, lowest
// channels first) are compensated as a dense contraction on the matrix cores,
// the other entries by the row-layout kernel.  The workspace holds the
// per-channel counts, the heavy channel list, the dense residual operand, the
// heavy channels' weight codes and the compacted lists of the other entries.
constexpr int kSplitHeavy = 256;
constexpr int kSplitPos = 2 * kSplitHeavy;  // dense positions: hi and lo half of each channel
struct SplitLayout {
  size_t count, slot, hlist, pow2, rh, idxh, spp, spr, spc, total;
};
SplitLayout split_layout(int n, int d_in, int d_out, int k);
hipError_t launch_compensate_split(const CompArgs& a, const uint32_t* idx_w_gemm, void* ws,
                                   hipStream_t s);
// the dense part: the many-token MFMA kernel with an fp16 value operand
hipError_t launch_gemm_values(const GemmArgs& a, hipStream_t s);
// the many-token MFMA kernel over the codes, then the dense positions a.hv/a.hw
hipError_t launch_gemm_heavy(const GemmArgs& a, hipStream_t s);
// y (+)= Y* + Y' with the heavy channels inside the GEMM (g: n > 32, d_in % 64
// == 0; a: the compensation's arguments, its idx_w in the row layout)
hipError_t launch_gemm_compensated_split(const GemmArgs& g, const CompArgs& a,
                                         const uint32_t* idx_w_gemm, void* ws, hipStream_t s);

// Bytes of dynamic LDS the quantize kernel needs for a token of d_in values
// and k outliers per side.
size_t quantize_lds_bytes(int d_in, int k, bool inlier = false);

hipError_t launch_build_lut(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                            oasis_lut_block* out, hipStream_t s);
hipError_t launch_quantize(const QuantArgs& a, hipStream_t s);
hipError_t launch_cluster(const QuantArgs& a, hipStream_t s);   // scale + codes only
hipError_t launch_outliers(const QuantArgs& a, hipStream_t s);  // lists + residuals only
// inlier scale: t from the channels in neither list, then codes and residuals
// (after a launch that wrote the lists; reads C_A from a.lut)
hipError_t launch_inlier_codes(const QuantArgs& a, hipStream_t s);
hipError_t launch_gemm_lut(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_mfma(const GemmArgs& a, hipStream_t s);
// per-output-channel weight codebooks (a.cb_cols), n <= 32
hipError_t launch_gemm_percol(const GemmArgs& a, hipStream_t s);
// Y (+)= Y* + Y' in one launch when a.n <= kFusedMaxTokens.
constexpr int kFusedMaxTokens = 32;
hipError_t launch_compensate(const CompArgs& a, hipStream_t s);
// Same, with idx_w in the row layout (uint32 [d_in][ceil(d_out / 8)]).
hipError_t launch_compensate_wr(const CompArgs& a, hipStream_t s);
hipError_t launch_fill_zero(float* y, size_t count, hipStream_t s);

}  // namespace oasis
