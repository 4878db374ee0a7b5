// C ABI of liboasis: host-side argument checking and kernel launches.
// Every check happens before anything is enqueued, so an error status means
// nothing ran.  No exception crosses the ABI.
#include <cmath>
#include <cstdint>
#include <cstring>

#include "common.h"

namespace {

// IEEE binary16 bits -> float (host side, exact).
float half_bits_to_float(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
  const uint32_t exp = (h >> 10) & 0x1Fu;
  const uint32_t man = h & 0x3FFu;
  float out;
  if (exp == 0) {
    out = std::ldexp((float)man, -24);
    if (sign) out = -out;
    return out;
  }
  if (exp == 31) {
    uint32_t bits = sign | 0x7F800000u | (man << 13);
    std::memcpy(&out, &bits, 4);
    return out;
  }
  uint32_t bits = sign | ((exp + 112u) << 23) | (man << 13);
  std::memcpy(&out, &bits, 4);
  return out;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }
bool bits_ok(int b) { return b >= 1 && b <= 4; }
// The GEMM kernels address codes with 32-bit buffer offsets, up to one block
// of 16 weight rows past the last (partial) block.
bool offsets_fit(int n, int d_in, int d_out) {
  const uint64_t kb = (uint64_t)(d_in / 8) + 31;
  return kb * (uint64_t)d_out * 4u < (1ull << 31) && (uint64_t)(n + 1) * kb * 4u < (1ull << 31);
}

constexpr size_t kMaxLds = 160 * 1024;

int launched(hipError_t e) { return e == hipSuccess ? OASIS_OK : OASIS_ERR_LAUNCH; }

}  // namespace

extern "C" {

const char* oasis_status_str(int status) {
  switch (status) {
    case OASIS_OK: return "ok";
    case OASIS_ERR_NULL: return "null pointer";
    case OASIS_ERR_SHAPE: return "bad shape";
    case OASIS_ERR_BITS: return "bit-width outside 1..4";
    case OASIS_ERR_K: return "k outside 0..d_in";
    case OASIS_ERR_CODEBOOK: return "codebook not finite or activation codebook not ascending";
    case OASIS_ERR_ALIGN: return "misaligned pointer";
    case OASIS_ERR_MODE: return "unknown scale mode or algorithm";
    case OASIS_ERR_LAUNCH: return "HIP launch failed";
    case OASIS_ERR_TOO_LARGE: return "size exceeds kernel limits";
    case OASIS_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    default: return "unknown status";
  }
}

const char* oasis_version(void) { return "oasis 0.1 gfx950"; }

// Inlier scale: with top-k lists the quantize launch computes t, the codes
// and the residuals itself once its lists exist; with fixed thresholds the
// quantize launch (absmax scale) writes the lists, then a second launch
// recomputes t, the codes and the residuals from them.
// The fused form also needs the listed-channel bitmap and the entries in
// LDS; where they do not fit, the two launches are used as well.
static int quantize_launch(oasis::QuantArgs a, hipStream_t stream) {
  const bool inlier = a.scale_mode == OASIS_SCALE_INLIER;
  const bool fused = inlier && !a.static_thr && a.k > 0 &&
                     oasis::quantize_lds_bytes(a.d_in, a.k, true) <= kMaxLds;
  if (inlier && !fused) a.scale_mode = OASIS_SCALE_ABSMAX;
  hipError_t e = oasis::launch_quantize(a, stream);
  if (e != hipSuccess || !inlier || fused) return launched(e);
  if (a.lut_out) a.lut = a.lut_out;
  return launched(oasis::launch_inlier_codes(a, stream));
}

int oasis_build_lut(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                    oasis_lut_block* out, hipStream_t stream) {
  if (!cb_act || !cb_wgt || !out) return OASIS_ERR_NULL;
  if (!bits_ok(b_a) || !bits_ok(b_w)) return OASIS_ERR_BITS;
  for (int i = 0; i < (1 << b_a); ++i) {
    const float v = half_bits_to_float(cb_act[i]);
    if (!std::isfinite(v)) return OASIS_ERR_CODEBOOK;
    if (i > 0 && !(v > half_bits_to_float(cb_act[i - 1]))) return OASIS_ERR_CODEBOOK;
  }
  for (int i = 0; i < (1 << b_w); ++i)
    if (!std::isfinite(half_bits_to_float(cb_wgt[i]))) return OASIS_ERR_CODEBOOK;
  if (!aligned(out, 16)) return OASIS_ERR_ALIGN;
  return launched(oasis::launch_build_lut(cb_act, b_a, cb_wgt, b_w, out, stream));
}

int oasis_quantize_act(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut, int b_a,
                       int k, int scale_mode, uint8_t* idx_act, float* act_scale,
                       int32_t* max_idx, int32_t* min_idx, float* residual, hipStream_t stream) {
  if (n < 0 || d_in < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (scale_mode != OASIS_SCALE_ABSMAX && scale_mode != OASIS_SCALE_NONE &&
      scale_mode != OASIS_SCALE_INLIER)
    return OASIS_ERR_MODE;
  if (d_in > 65536) return OASIS_ERR_TOO_LARGE;
  if (oasis::quantize_lds_bytes(d_in, k) > kMaxLds) return OASIS_ERR_TOO_LARGE;
  if (n == 0) return OASIS_OK;
  if (!x || !lut || !act_scale || (d_in > 0 && !idx_act)) return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual)) return OASIS_ERR_NULL;
  if (!aligned(x, 16) || !aligned(lut, 16) || !aligned(idx_act, 16) || !aligned(act_scale, 4) ||
      !aligned(max_idx, 4) || !aligned(min_idx, 4) || !aligned(residual, 4))
    return OASIS_ERR_ALIGN;
  oasis::QuantArgs a{x, n, d_in, b_a, k, scale_mode, lut, idx_act, act_scale,
                     max_idx, min_idx, residual, nullptr, {}, 0};
  return quantize_launch(a, stream);
}

int oasis_quantize_act_static(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut,
                              int b_a, int k, int scale_mode, float thr_hi, float thr_lo,
                              uint8_t* idx_act, float* act_scale, int32_t* max_idx,
                              int32_t* min_idx, float* residual, hipStream_t stream) {
  if (n < 0 || d_in < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (scale_mode != OASIS_SCALE_ABSMAX && scale_mode != OASIS_SCALE_NONE &&
      scale_mode != OASIS_SCALE_INLIER)
    return OASIS_ERR_MODE;
  if (std::isnan(thr_hi) || std::isnan(thr_lo) || !(thr_lo < thr_hi)) return OASIS_ERR_MODE;
  if (d_in > 65536) return OASIS_ERR_TOO_LARGE;
  if (oasis::quantize_lds_bytes(d_in, k) > kMaxLds) return OASIS_ERR_TOO_LARGE;
  if (n == 0) return OASIS_OK;
  if (!x || !lut || !act_scale || (d_in > 0 && !idx_act)) return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual)) return OASIS_ERR_NULL;
  if (!aligned(x, 16) || !aligned(lut, 16) || !aligned(idx_act, 16) || !aligned(act_scale, 4) ||
      !aligned(max_idx, 4) || !aligned(min_idx, 4) || !aligned(residual, 4))
    return OASIS_ERR_ALIGN;
  oasis::QuantArgs a{x, n, d_in, b_a, k, scale_mode, lut, idx_act, act_scale,
                     max_idx, min_idx, residual, nullptr, {}, 0, 1, thr_hi, thr_lo};
  return quantize_launch(a, stream);
}

// oasis_build_lut_quantize_act and its OASIS-S form: every check, then one
// launch whose first workgroup also writes the LUT block.
static int build_lut_quantize(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                              oasis_lut_block* lut, const uint16_t* x, int n, int d_in, int k,
                              int scale_mode, int static_thr, float thr_hi, float thr_lo,
                              uint8_t* idx_act, float* act_scale, int32_t* max_idx,
                              int32_t* min_idx, float* residual, hipStream_t stream) {
  if (!cb_act || !cb_wgt || !lut) return OASIS_ERR_NULL;
  if (n < 0 || d_in < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a) || !bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (scale_mode != OASIS_SCALE_ABSMAX && scale_mode != OASIS_SCALE_NONE &&
      scale_mode != OASIS_SCALE_INLIER)
    return OASIS_ERR_MODE;
  if (static_thr && (std::isnan(thr_hi) || std::isnan(thr_lo) || !(thr_lo < thr_hi)))
    return OASIS_ERR_MODE;
  for (int i = 0; i < (1 << b_a); ++i) {
    const float v = half_bits_to_float(cb_act[i]);
    if (!std::isfinite(v)) return OASIS_ERR_CODEBOOK;
    if (i > 0 && !(v > half_bits_to_float(cb_act[i - 1]))) return OASIS_ERR_CODEBOOK;
  }
  for (int i = 0; i < (1 << b_w); ++i)
    if (!std::isfinite(half_bits_to_float(cb_wgt[i]))) return OASIS_ERR_CODEBOOK;
  if (d_in > 65536) return OASIS_ERR_TOO_LARGE;
  if (oasis::quantize_lds_bytes(d_in, k) > kMaxLds) return OASIS_ERR_TOO_LARGE;
  if (n > 0 && (!x || !act_scale || (d_in > 0 && !idx_act))) return OASIS_ERR_NULL;
  if (n > 0 && k > 0 && (!max_idx || !min_idx || !residual)) return OASIS_ERR_NULL;
  if (!aligned(x, 16) || !aligned(lut, 16) || !aligned(idx_act, 16) || !aligned(act_scale, 4) ||
      !aligned(max_idx, 4) || !aligned(min_idx, 4) || !aligned(residual, 4))
    return OASIS_ERR_ALIGN;
  if (n == 0) return launched(oasis::launch_build_lut(cb_act, b_a, cb_wgt, b_w, lut, stream));
  oasis::QuantArgs a{x, n, d_in, b_a, k, scale_mode, lut, idx_act, act_scale,
                     max_idx, min_idx, residual, lut, {}, b_w, static_thr, thr_hi, thr_lo};
  for (int i = 0; i < (1 << b_a); ++i) a.cb.act[i] = cb_act[i];
  for (int i = 0; i < (1 << b_w); ++i) a.cb.wgt[i] = cb_wgt[i];
  return quantize_launch(a, stream);
}

int oasis_build_lut_quantize_act(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                                 oasis_lut_block* lut, const uint16_t* x, int n, int d_in, int k,
                                 int scale_mode, uint8_t* idx_act, float* act_scale,
                                 int32_t* max_idx, int32_t* min_idx, float* residual,
                                 hipStream_t stream) {
  return build_lut_quantize(cb_act, b_a, cb_wgt, b_w, lut, x, n, d_in, k, scale_mode, 0, 0.0f,
                            0.0f, idx_act, act_scale, max_idx, min_idx, residual, stream);
}

int oasis_build_lut_quantize_act_static(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt,
                                        int b_w, oasis_lut_block* lut, const uint16_t* x, int n,
                                        int d_in, int k, int scale_mode, float thr_hi,
                                        float thr_lo, uint8_t* idx_act, float* act_scale,
                                        int32_t* max_idx, int32_t* min_idx, float* residual,
                                        hipStream_t stream) {
  return build_lut_quantize(cb_act, b_a, cb_wgt, b_w, lut, x, n, d_in, k, scale_mode, 1, thr_hi,
                            thr_lo, idx_act, act_scale, max_idx, min_idx, residual, stream);
}

int oasis_cluster_act(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut, int b_a,
                      int scale_mode, uint8_t* idx_act, float* act_scale, hipStream_t stream) {
  if (n < 0 || d_in < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a)) return OASIS_ERR_BITS;
  if (scale_mode != OASIS_SCALE_ABSMAX && scale_mode != OASIS_SCALE_NONE) return OASIS_ERR_MODE;
  if (d_in > 65536) return OASIS_ERR_TOO_LARGE;
  if (n == 0) return OASIS_OK;
  if (!x || !lut || !act_scale || (d_in > 0 && !idx_act)) return OASIS_ERR_NULL;
  if (!aligned(x, 16) || !aligned(lut, 16) || !aligned(idx_act, 16) || !aligned(act_scale, 4))
    return OASIS_ERR_ALIGN;
  oasis::QuantArgs a{x, n, d_in, b_a, 0, scale_mode, lut, idx_act, act_scale,
                     nullptr, nullptr, nullptr, nullptr, {}, 0};
  return launched(oasis::launch_cluster(a, stream));
}

int oasis_detect_outliers(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut, int b_a,
                          int k, int scale_mode, int32_t* max_idx, int32_t* min_idx,
                          float* residual, hipStream_t stream) {
  if (n < 0 || d_in < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (scale_mode != OASIS_SCALE_ABSMAX && scale_mode != OASIS_SCALE_NONE) return OASIS_ERR_MODE;
  if (d_in > 65536) return OASIS_ERR_TOO_LARGE;
  if (oasis::quantize_lds_bytes(d_in, k) > kMaxLds) return OASIS_ERR_TOO_LARGE;
  if (n == 0 || k == 0) return OASIS_OK;
  if (!x || !lut || !max_idx || !min_idx || !residual) return OASIS_ERR_NULL;
  if (!aligned(x, 16) || !aligned(lut, 16) || !aligned(max_idx, 4) || !aligned(min_idx, 4) ||
      !aligned(residual, 4))
    return OASIS_ERR_ALIGN;
  oasis::QuantArgs a{x, n, d_in, b_a, k, scale_mode, lut, nullptr, nullptr,
                     max_idx, min_idx, residual, nullptr, {}, 0};
  return launched(oasis::launch_outliers(a, stream));
}

int oasis_lut_gemm(const uint8_t* idx_act, const float* act_scale, int n, int d_in,
                   const uint32_t* idx_w, const float* w_scale, int d_out,
                   const oasis_lut_block* lut, int b_a, int b_w, int algo, float* y,
                   int accumulate, hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a) || !bits_ok(b_w)) return OASIS_ERR_BITS;
  if (algo != OASIS_ALGO_LUT && algo != OASIS_ALGO_MFMA) return OASIS_ERR_MODE;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!act_scale || !w_scale || !lut || !y || (d_in > 0 && (!idx_act || !idx_w)))
    return OASIS_ERR_NULL;
  if (!aligned(idx_act, 16) || !aligned(idx_w, 16) || !aligned(lut, 16) || !aligned(y, 4) ||
      !aligned(act_scale, 4) || !aligned(w_scale, 4))
    return OASIS_ERR_ALIGN;
  if (!offsets_fit(n, d_in, d_out)) return OASIS_ERR_TOO_LARGE;
  if (d_in == 0) {  // empty reduction: Y* = 0
    if (accumulate) return OASIS_OK;
    return launched(oasis::launch_fill_zero(y, (size_t)n * d_out, stream));
  }
  oasis::GemmArgs a{idx_act, act_scale, n, d_in, idx_w, w_scale, d_out, lut, b_a, b_w, y,
                    accumulate ? 1 : 0, nullptr, nullptr, nullptr, 0};
  return launched(algo == OASIS_ALGO_LUT ? oasis::launch_gemm_lut(a, stream)
                                         : oasis::launch_gemm_mfma(a, stream));
}

int oasis_outlier_compensate(const int32_t* max_idx, const int32_t* min_idx, const float* residual,
                             int n, int k, const uint32_t* idx_w, const oasis_lut_block* lut,
                             int b_w, const float* w_scale, int d_in, int d_out, float* y,
                             int accumulate, hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!lut || !w_scale || !y) return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual || !idx_w)) return OASIS_ERR_NULL;
  if (!aligned(max_idx, 4) || !aligned(min_idx, 4) || !aligned(residual, 4) ||
      !aligned(idx_w, 4) || !aligned(lut, 16) || !aligned(w_scale, 4) || !aligned(y, 4))
    return OASIS_ERR_ALIGN;
  // the row-grouped kernel (many tokens) addresses the codes with 32-bit
  // buffer offsets
  if ((uint64_t)(d_in / 8) * (uint64_t)d_out * 4u >= (1ull << 31)) return OASIS_ERR_TOO_LARGE;
  oasis::CompArgs a{max_idx, min_idx, residual, n, k, idx_w, lut, b_w, w_scale, d_in, d_out, y,
                    accumulate ? 1 : 0};
  return launched(oasis::launch_compensate(a, stream));
}

int oasis_outlier_compensate_rows(const int32_t* max_idx, const int32_t* min_idx,
                                  const float* residual, int n, int k, const uint32_t* idx_wr,
                                  const oasis_lut_block* lut, int b_w, const float* w_scale,
                                  int d_in, int d_out, float* y, int accumulate,
                                  hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!lut || !w_scale || !y) return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual || !idx_wr)) return OASIS_ERR_NULL;
  if (!aligned(max_idx, 4) || !aligned(min_idx, 4) || !aligned(residual, 4) ||
      !aligned(idx_wr, 4) || !aligned(lut, 16) || !aligned(w_scale, 4) || !aligned(y, 4))
    return OASIS_ERR_ALIGN;
  // byte offsets into the codes are 32-bit
  if ((uint64_t)d_in * (uint64_t)((d_out + 7) / 8) * 4u >= (1ull << 31)) return OASIS_ERR_TOO_LARGE;
  oasis::CompArgs a{max_idx, min_idx, residual, n, k, idx_wr, lut, b_w, w_scale, d_in, d_out, y,
                    accumulate ? 1 : 0};
  return launched(oasis::launch_compensate_wr(a, stream));
}

size_t oasis_outlier_compensate_split_workspace(int n, int d_in, int d_out, int k) {
  if (n < 0 || d_in < 0 || d_out < 0 || k < 0) return 0;
  return oasis::split_layout(n, d_in, d_out, k).total;
}

int oasis_outlier_compensate_split(const int32_t* max_idx, const int32_t* min_idx,
                                   const float* residual, int n, int k, const uint32_t* idx_w,
                                   const uint32_t* idx_wr, const oasis_lut_block* lut, int b_w,
                                   const float* w_scale, int d_in, int d_out, float* y,
                                   int accumulate, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!lut || !w_scale || !y) return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual || !idx_w || !idx_wr)) return OASIS_ERR_NULL;
  if (!aligned(max_idx, 4) || !aligned(min_idx, 4) || !aligned(residual, 4) ||
      !aligned(idx_w, 16) || !aligned(idx_wr, 4) || !aligned(lut, 16) || !aligned(w_scale, 4) ||
      !aligned(y, 4))
    return OASIS_ERR_ALIGN;
  // 32-bit byte offsets into the row-layout codes, the heavy rows and the
  // dense operand
  if ((uint64_t)d_in * (uint64_t)((d_out + 7) / 8) * 4u >= (1ull << 31)) return OASIS_ERR_TOO_LARGE;
  if (!offsets_fit(n, oasis::kSplitPos, d_out) ||
      (uint64_t)(n + 1) * 2u * oasis::kSplitPos >= (1ull << 31))
    return OASIS_ERR_TOO_LARGE;
  if (k > 0) {
    if (!workspace || !aligned(workspace, 256)) return OASIS_ERR_WORKSPACE;
    if (workspace_bytes < oasis::split_layout(n, d_in, d_out, k).total) return OASIS_ERR_WORKSPACE;
  }
  oasis::CompArgs a{max_idx, min_idx, residual, n, k, idx_wr, lut, b_w, w_scale, d_in, d_out, y,
                    accumulate ? 1 : 0, nullptr};
  return launched(oasis::launch_compensate_split(a, idx_w, workspace, stream));
}

static int gemm_compensated(const uint8_t* idx_act, const float* act_scale, int n, int d_in,
                            const uint32_t* idx_w, const uint32_t* idx_wr, const float* w_scale,
                            int d_out, const oasis_lut_block* lut, int b_a, int b_w,
                            const int32_t* max_idx, const int32_t* min_idx,
                            const float* residual, int k, float* y, int accumulate,
                            hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a) || !bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!act_scale || !w_scale || !lut || !y || (d_in > 0 && (!idx_act || !idx_w)))
    return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual)) return OASIS_ERR_NULL;
  if (!aligned(idx_act, 16) || !aligned(idx_w, 16) || !aligned(lut, 16) || !aligned(y, 4) ||
      !aligned(act_scale, 4) || !aligned(w_scale, 4) || !aligned(max_idx, 4) ||
      !aligned(min_idx, 4) || !aligned(residual, 4) || !aligned(idx_wr, 4))
    return OASIS_ERR_ALIGN;
  if (!offsets_fit(n, d_in, d_out)) return OASIS_ERR_TOO_LARGE;
  if (idx_wr && (uint64_t)d_in * (uint64_t)((d_out + 7) / 8) * 4u >= (1ull << 31))
    return OASIS_ERR_TOO_LARGE;
  if (d_in == 0) {  // no channels: Y* = Y' = 0
    if (accumulate) return OASIS_OK;
    return launched(oasis::launch_fill_zero(y, (size_t)n * d_out, stream));
  }
  if (n <= oasis::kFusedMaxTokens) {
    oasis::GemmArgs a{idx_act, act_scale, n, d_in, idx_w, w_scale, d_out, lut, b_a, b_w, y,
                      accumulate ? 1 : 0, max_idx, min_idx, residual, k, idx_wr};
    return launched(oasis::launch_gemm_mfma(a, stream));
  }
  // many tokens: main branch into y, then the compensation merged into it
  oasis::GemmArgs a{idx_act, act_scale, n, d_in, idx_w, w_scale, d_out, lut, b_a, b_w, y,
                    accumulate ? 1 : 0, nullptr, nullptr, nullptr, 0, nullptr};
  hipError_t e = oasis::launch_gemm_mfma(a, stream);
  if (e != hipSuccess || k == 0) return launched(e);
  oasis::CompArgs c{max_idx, min_idx, residual, n, k, idx_wr ? idx_wr : idx_w, lut, b_w,
                    w_scale, d_in, d_out, y, 1};
  return launched(idx_wr ? oasis::launch_compensate_wr(c, stream)
                         : oasis::launch_compensate(c, stream));
}

int oasis_lut_gemm_compensated_split(const uint8_t* idx_act, const float* act_scale, int n,
                                     int d_in, const uint32_t* idx_w, const uint32_t* idx_wr,
                                     const float* w_scale, int d_out, const oasis_lut_block* lut,
                                     int b_a, int b_w, const int32_t* max_idx,
                                     const int32_t* min_idx, const float* residual, int k,
                                     float* y, int accumulate, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a) || !bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!act_scale || !w_scale || !lut || !y || (d_in > 0 && (!idx_act || !idx_w)))
    return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual || !idx_wr)) return OASIS_ERR_NULL;
  if (!aligned(idx_act, 16) || !aligned(idx_w, 16) || !aligned(lut, 16) || !aligned(y, 4) ||
      !aligned(act_scale, 4) || !aligned(w_scale, 4) || !aligned(max_idx, 4) ||
      !aligned(min_idx, 4) || !aligned(residual, 4) || !aligned(idx_wr, 4))
    return OASIS_ERR_ALIGN;
  if (!offsets_fit(n, d_in, d_out)) return OASIS_ERR_TOO_LARGE;
  if (idx_wr && (uint64_t)d_in * (uint64_t)((d_out + 7) / 8) * 4u >= (1ull << 31))
    return OASIS_ERR_TOO_LARGE;
  if (!offsets_fit(n, oasis::kSplitPos, d_out) ||
      (uint64_t)(n + 1) * 2u * oasis::kSplitPos >= (1ull << 31))
    return OASIS_ERR_TOO_LARGE;
  // few tokens or no lists: the fused GEMV (or the GEMM alone), no workspace
  if (n <= oasis::kFusedMaxTokens || k == 0 || d_in == 0)
    return gemm_compensated(idx_act, act_scale, n, d_in, idx_w, idx_wr, w_scale, d_out, lut, b_a,
                            b_w, max_idx, min_idx, residual, k, y, accumulate, stream);
  if (!workspace || !aligned(workspace, 256) ||
      workspace_bytes < oasis::split_layout(n, d_in, d_out, k).total)
    return OASIS_ERR_WORKSPACE;
  oasis::GemmArgs g{idx_act, act_scale, n, d_in, idx_w, w_scale, d_out, lut, b_a, b_w, y, 1,
                    nullptr, nullptr, nullptr, 0, nullptr};
  oasis::CompArgs c{max_idx, min_idx, residual, n, k, idx_wr, lut, b_w, w_scale, d_in, d_out, y,
                    accumulate ? 1 : 0, nullptr};
  if (d_in % 64 == 0)
    return launched(oasis::launch_gemm_compensated_split(g, c, idx_w, workspace, stream));
  // other reductions (the 16x16x32 kernel): split compensation, then the GEMM
  hipError_t e = oasis::launch_compensate_split(c, idx_w, workspace, stream);
  if (e != hipSuccess) return launched(e);
  return launched(oasis::launch_gemm_mfma(g, stream));
}

int oasis_lut_gemm_compensated(const uint8_t* idx_act, const float* act_scale, int n, int d_in,
                               const uint32_t* idx_w, const float* w_scale, int d_out,
                               const oasis_lut_block* lut, int b_a, int b_w,
                               const int32_t* max_idx, const int32_t* min_idx,
                               const float* residual, int k, float* y, int accumulate,
                               hipStream_t stream) {
  return gemm_compensated(idx_act, act_scale, n, d_in, idx_w, nullptr, w_scale, d_out, lut, b_a,
                          b_w, max_idx, min_idx, residual, k, y, accumulate, stream);
}

int oasis_lut_gemm_compensated_rows(const uint8_t* idx_act, const float* act_scale, int n,
                                    int d_in, const uint32_t* idx_w, const uint32_t* idx_wr,
                                    const float* w_scale, int d_out, const oasis_lut_block* lut,
                                    int b_a, int b_w, const int32_t* max_idx,
                                    const int32_t* min_idx, const float* residual, int k,
                                    float* y, int accumulate, hipStream_t stream) {
  if (k > 0 && n > 0 && d_out > 0 && d_in > 0 && !idx_wr) return OASIS_ERR_NULL;
  return gemm_compensated(idx_act, act_scale, n, d_in, idx_w, idx_wr, w_scale, d_out, lut, b_a,
                          b_w, max_idx, min_idx, residual, k, y, accumulate, stream);
}

int oasis_lut_gemm_compensated_percol(const uint8_t* idx_act, const float* act_scale, int n,
                                      int d_in, const uint32_t* idx_w, const float* w_scale,
                                      int d_out, const oasis_lut_block* lut,
                                      const uint16_t* cb_wgt_cols, int b_a, int b_w,
                                      const int32_t* max_idx, const int32_t* min_idx,
                                      const float* residual, int k, float* y, int accumulate,
                                      hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  if (!bits_ok(b_a) || !bits_ok(b_w)) return OASIS_ERR_BITS;
  if (k < 0 || k > d_in) return OASIS_ERR_K;
  if (n == 0 || d_out == 0) return OASIS_OK;
  if (!act_scale || !w_scale || !lut || !y || !cb_wgt_cols || (d_in > 0 && (!idx_act || !idx_w)))
    return OASIS_ERR_NULL;
  if (k > 0 && (!max_idx || !min_idx || !residual)) return OASIS_ERR_NULL;
  if (!aligned(idx_act, 16) || !aligned(idx_w, 16) || !aligned(lut, 16) || !aligned(y, 4) ||
      !aligned(act_scale, 4) || !aligned(w_scale, 4) || !aligned(max_idx, 4) ||
      !aligned(min_idx, 4) || !aligned(residual, 4) || !aligned(cb_wgt_cols, 16))
    return OASIS_ERR_ALIGN;
  if (!offsets_fit(n, d_in, d_out)) return OASIS_ERR_TOO_LARGE;
  if (d_in == 0) {  // no channels: Y* = Y' = 0
    if (accumulate) return OASIS_OK;
    return launched(oasis::launch_fill_zero(y, (size_t)n * d_out, stream));
  }
  oasis::GemmArgs a{idx_act, act_scale, n, d_in, idx_w, w_scale, d_out, lut, b_a, b_w, y,
                    accumulate ? 1 : 0, max_idx, min_idx, residual, k, nullptr, cb_wgt_cols};
  return launched(oasis::launch_gemm_percol(a, stream));
}

int oasis_pack_weight_indices(const uint8_t* w_idx, int d_in, int d_out, uint32_t* out) {
  if (!w_idx || !out) return OASIS_ERR_NULL;
  if (d_in < 0 || d_out < 0 || (d_in % 8) != 0) return OASIS_ERR_SHAPE;
  for (int b = 0; b < d_in / 8; ++b) {
    uint32_t* row = out + (size_t)b * d_out;
    for (int j = 0; j < d_out; ++j) row[j] = 0;
    for (int e = 0; e < 8; ++e) {
      const uint8_t* src = w_idx + (size_t)(8 * b + e) * d_out;
      for (int j = 0; j < d_out; ++j) row[j] |= (uint32_t)(src[j] & 15u) << (4 * e);
    }
  }
  return OASIS_OK;
}

int oasis_pack_weight_rows(const uint8_t* w_idx, int d_in, int d_out, uint32_t* out) {
  if (!w_idx || !out) return OASIS_ERR_NULL;
  if (d_in < 0 || d_out < 0) return OASIS_ERR_SHAPE;
  const int wn = (d_out + 7) / 8;
  for (int p = 0; p < d_in; ++p) {
    const uint8_t* src = w_idx + (size_t)p * d_out;
    uint32_t* row = out + (size_t)p * wn;
    for (int m = 0; m < wn; ++m) {
      uint32_t w = 0;
      for (int c = 0; c < 8 && 8 * m + c < d_out; ++c) w |= (uint32_t)(src[8 * m + c] & 15u) << (4 * c);
      row[m] = w;
    }
  }
  return OASIS_OK;
}

}  // extern "C"
