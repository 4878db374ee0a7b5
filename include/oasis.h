/*
 * oasis.h - C ABI of the OASIS hot path on AMD MI355X (gfx950).
 *
 * OASIS (arXiv 2507.23035) multiplies non-uniformly (K-Means codebook)
 * quantized activations and weights without dequantizing them: the products
 * of every activation centroid with every weight centroid are precomputed in
 * a Cartesian product LUT (Sec. III-B), activations are clustered per token
 * at run time and the dynamic top-k outliers of each token are compensated
 * in a separate branch (look-ahead computation + error compensation,
 * Sec. III-C; outlier detection, Sec. IV-D).
 *
 * Conventions shared by every call
 *  - Tensor pointers are DEVICE pointers owned by the caller; the library
 *    allocates no device memory and keeps no state between calls.  Pointers
 *    documented as HOST pointers are read during the call only.
 *  - fp16 values are passed as their IEEE binary16 bit patterns (uint16_t).
 *  - Every call is asynchronous on `stream` (NULL = the null stream) and
 *    returns an oasis_status code; argument errors are detected on the host
 *    before anything is launched.  Nothing throws across the ABI.
 *  - Index tensors hold one 4-bit code per nibble for every bit-width 1..4.
 *  - Activations must be finite (NaN is outside the contract: memory stays
 *    safe but results are unspecified).
 *  - Calls are thread-compatible: concurrent calls must not share outputs.
 *
 * Index layouts
 *  - idx_act : uint8 [n][d_in/2]; channel 2q in the low nibble of byte q.
 *  - idx_w   : uint32 [d_in/8][d_out]; word (b, j) holds the codes of input
 *              channels 8b..8b+7 of output column j, channel 8b+e in bits
 *              4e..4e+3.  (Input-channel-major, so one input channel of all
 *              output columns, which the compensation fetches, is one
 *              contiguous row of words.)
 *  - idx_wr  : uint32 [d_in][ceil(d_out/8)]; word m of row p holds the codes
 *              of input channel p for output columns 8m..8m+7, column 8m+c
 *              in bits 4c..4c+3 (the row layout: one input channel is d_out/2
 *              contiguous bytes; read by oasis_outlier_compensate_rows).
 *  - y       : fp32 [n][d_out], row-major.
 */
#ifndef OASIS_H
#define OASIS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum oasis_status {
  OASIS_OK = 0,
  OASIS_ERR_NULL = -1,        /* a required pointer is NULL                        */
  OASIS_ERR_SHAPE = -2,       /* n/d_in/d_out negative, d_out < 1, d_in % 8 != 0   */
  OASIS_ERR_BITS = -3,        /* bit-width outside 1..4                            */
  OASIS_ERR_K = -4,           /* k < 0 or k > d_in                                 */
  OASIS_ERR_CODEBOOK = -5,    /* activation codebook not strictly ascending, or a
                                 codebook entry is not finite                      */
  OASIS_ERR_ALIGN = -6,       /* a pointer is not aligned as documented            */
  OASIS_ERR_MODE = -7,        /* unknown scale mode or algorithm                   */
  OASIS_ERR_LAUNCH = -8,      /* the HIP runtime refused a launch                  */
  OASIS_ERR_TOO_LARGE = -9,   /* a size exceeds what a kernel supports             */
  OASIS_ERR_WORKSPACE = -10   /* workspace missing, too small or misaligned        */
};

enum oasis_scale_mode {
  OASIS_SCALE_ABSMAX = 0,     /* t_i = max_p |x_ip| (outliers included)            */
  OASIS_SCALE_NONE = 1,       /* t_i = 1                                           */
  OASIS_SCALE_INLIER = 2      /* t_i = max |x_ip| over the channels in neither
                                 outlier list (0 if every channel is listed); the
                                 lists come first, so there is no look-ahead split:
                                 a second launch computes t, codes and residuals */
};

enum oasis_gemm_algo {
  OASIS_ALGO_LUT = 0,         /* one LDS LUT lookup per (token, channel, column)   */
  OASIS_ALGO_MFMA = 1         /* rank-1 LUT: exact fp16 factors on matrix cores    */
};

/* The LUT block: the Cartesian product LUT plus both codebooks, the content
 * of the accelerator's on-chip LUT (Sec. IV-A: it stores the products and
 * the activation and weight codebooks).  1088 bytes, 16-byte aligned. */
typedef struct oasis_lut_block {
  float lut[256];          /* lut[(a << b_w) | w] = C_A[a] * C_W[w], exact fp32; */
                           /* entries at and beyond 2^(b_a+b_w) are 0            */
  uint16_t cb_act[16];     /* C_A (fp16 bits), first 2^b_a used, rest 0          */
  uint16_t cb_wgt[16];     /* C_W (fp16 bits), first 2^b_w used, rest 0          */
} oasis_lut_block;

/* Human-readable name of a status code (static string). */
const char* oasis_status_str(int status);

/* Library version string, e.g. "oasis 0.1 gfx950". */
const char* oasis_version(void);

/*
 * oasis_build_lut - Cartesian product LUT (Sec. III-B; on-chip LUT, Sec. IV-A).
 *   cb_act : HOST fp16 [2^b_a], strictly ascending, finite (the Clustering
 *            Unit's binary search needs the order, Sec. IV-C).
 *   cb_wgt : HOST fp16 [2^b_w], finite.
 *   out    : DEVICE oasis_lut_block, 16-byte aligned; fully overwritten.
 * Errors: NULL, BITS, CODEBOOK, ALIGN, LAUNCH.
 */
int oasis_build_lut(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                    oasis_lut_block* out, hipStream_t stream);

/*
 * oasis_quantize_act - per-token activation quantization and dynamic top-k
 * outlier detection (Sec. III-A, III-C1; Clustering Unit, Sec. IV-C;
 * Orizuru, Sec. IV-D; Error Calculation Unit, Sec. IV-A).
 *   x         : DEVICE fp16 [n][d_in], 16-byte aligned.
 *   lut       : DEVICE LUT block built with the same b_a (its C_A is used).
 *   k         : outliers per side per token, 0 <= k <= d_in.
 *   scale_mode: OASIS_SCALE_ABSMAX, OASIS_SCALE_NONE or OASIS_SCALE_INLIER.
 * Outputs (DEVICE, fully overwritten):
 *   idx_act   : uint8 [n][d_in/2] cluster index of EVERY channel, outliers
 *               included: #{c : x >= fp32(t * b_c)} with
 *               b_c = fp32(C_A[c] + C_A[c+1]) * 0.5 (half-open intervals).
 *   act_scale : fp32 [n], t_i.
 *   max_idx   : int32 [n][k], the k largest channels, largest first, ties to
 *               the lower channel (-0 == +0).
 *   min_idx   : int32 [n][k], the k smallest channels, smallest first, same
 *               tie rule.
 *   residual  : fp32 [n][2k]; [i][e] = fp32(x - fp32(t*C_A[a])) of max_idx
 *               entry e, [i][k+e] the same for min_idx entry e, or 0 when
 *               that channel is also in the token's max list (the union is
 *               compensated once).
 *   When k == 0, max_idx/min_idx/residual may be NULL.
 * Errors: NULL, SHAPE, BITS, K, ALIGN, MODE, TOO_LARGE (d_in > 65536), LAUNCH.
 */
int oasis_quantize_act(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut, int b_a,
                       int k, int scale_mode, uint8_t* idx_act, float* act_scale,
                       int32_t* max_idx, int32_t* min_idx, float* residual, hipStream_t stream);

/*
 * oasis_quantize_act_static - OASIS-S (Sec. V-A): the outliers are found with
 * fixed thresholds learned offline instead of the per-token top-k.
 *   Scale and codes as in oasis_quantize_act.  The max list holds the
 *   channels with x >= thr_hi, the min list those with x <= thr_lo, each in
 *   channel order and at most k of them (k = places per side); the places
 *   left hold channel -1 and residual 0 (the compensation calls skip them).
 *   Residuals as in oasis_quantize_act.  thr_lo < thr_hi, neither NaN
 *   (+-inf allowed).  With OASIS_SCALE_INLIER, t excludes the listed
 *   channels (unused places excluded nothing).
 * Errors: NULL, SHAPE, BITS, K, ALIGN, MODE (scale mode or thresholds),
 * TOO_LARGE, LAUNCH.
 */
int oasis_quantize_act_static(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut,
                              int b_a, int k, int scale_mode, float thr_hi, float thr_lo,
                              uint8_t* idx_act, float* act_scale, int32_t* max_idx,
                              int32_t* min_idx, float* residual, hipStream_t stream);

/*
 * oasis_build_lut_quantize_act - oasis_build_lut followed by
 * oasis_quantize_act, in one launch: the first workgroup of the quantize
 * kernel also writes the LUT block, and every workgroup takes C_A from the
 * codebook arguments, so a caller that rebuilds the LUT with every batch pays
 * no extra launch (the paper builds it once per layer, Sec. IV-A).
 *   cb_act, b_a, cb_wgt, b_w, lut : as in oasis_build_lut (lut is written;
 *            the other calls of the step read it after this one).
 *   x, n, d_in, k, scale_mode and the outputs : as in oasis_quantize_act.
 *   n == 0 builds the LUT alone.
 * Errors: those of both calls.
 */
int oasis_build_lut_quantize_act(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt, int b_w,
                                 oasis_lut_block* lut, const uint16_t* x, int n, int d_in, int k,
                                 int scale_mode, uint8_t* idx_act, float* act_scale,
                                 int32_t* max_idx, int32_t* min_idx, float* residual,
                                 hipStream_t stream);

/*
 * oasis_build_lut_quantize_act_static - oasis_build_lut followed by
 * oasis_quantize_act_static (OASIS-S, Sec. V-A), in one launch as in
 * oasis_build_lut_quantize_act.  Arguments, outputs and errors: those of the
 * two calls.
 */
int oasis_build_lut_quantize_act_static(const uint16_t* cb_act, int b_a, const uint16_t* cb_wgt,
                                        int b_w, oasis_lut_block* lut, const uint16_t* x, int n,
                                        int d_in, int k, int scale_mode, float thr_hi,
                                        float thr_lo, uint8_t* idx_act, float* act_scale,
                                        int32_t* max_idx, int32_t* min_idx, float* residual,
                                        hipStream_t stream);

/*
 * oasis_cluster_act - the main branch's share of oasis_quantize_act: scale
 * and cluster index of every channel (Sec. III-C1: the whole token is
 * clustered, outliers included), without outlier detection.  Same arguments
 * and outputs as oasis_quantize_act restricted to idx_act and act_scale.
 * With oasis_detect_outliers on a second stream this is the GPU form of the
 * look-ahead schedule: the main-branch GEMM needs only these outputs, so it
 * does not wait for outlier detection (Sec. II-C, III-C).  OASIS_SCALE_INLIER
 * needs the lists first and is refused (MODE).
 * Errors: NULL, SHAPE, BITS, ALIGN, MODE, TOO_LARGE, LAUNCH.
 */
int oasis_cluster_act(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut, int b_a,
                      int scale_mode, uint8_t* idx_act, float* act_scale, hipStream_t stream);

/*
 * oasis_detect_outliers - the outlier branch's share of oasis_quantize_act
 * (Orizuru and the Error Calculation Unit, Sec. IV-A, IV-D): max_idx,
 * min_idx and residual exactly as oasis_quantize_act writes them (the scale
 * and the cluster index of each outlier are recomputed from x).  k == 0 is a
 * no-op.  OASIS_SCALE_INLIER is refused (MODE), as in oasis_cluster_act.
 * Errors: NULL, SHAPE, BITS, K, ALIGN, MODE, TOO_LARGE, LAUNCH.
 */
int oasis_detect_outliers(const uint16_t* x, int n, int d_in, const oasis_lut_block* lut, int b_a,
                          int k, int scale_mode, int32_t* max_idx, int32_t* min_idx,
                          float* residual, hipStream_t stream);

/*
 * oasis_lut_gemm - look-ahead WAQ LUT-GEMM, the main branch (Sec. III-B,
 * III-C1): Y*[i][j] = t_i * s_j * sum_p LUT[(a_ip << b_w) | w_pj].
 *   idx_act, act_scale : from oasis_quantize_act (n tokens, d_in channels);
 *               idx_act 16-byte aligned.
 *   idx_w     : DEVICE uint32 [d_in/8][d_out] weight codes (layout above),
 *               16-byte aligned.
 *   w_scale   : DEVICE fp32 [d_out], s_j.
 *   lut       : DEVICE LUT block (b_a, b_w as built).
 *   algo      : OASIS_ALGO_LUT accumulates LUT entries fetched from LDS;
 *               OASIS_ALGO_MFMA uses that the LUT is the outer product of
 *               the codebooks, so the sum is a dense contraction of exact
 *               fp16 centroid values, run on matrix cores (fp32 accumulate).
 *               Both equal the definition up to fp32 summation order.
 *   y         : DEVICE fp32 [n][d_out], 4-byte aligned.
 *   accumulate != 0 : y += Y*  (merge into a compensation term written first);
 *   accumulate == 0 : y  = Y*.
 *   The literal-LUT kernel may merge partial sums over input-channel slices
 *   with fp32 atomics, so its summation order can vary run to run.
 *   The weight codes and the activation codes must each be < 2 GiB.
 * Errors: NULL, SHAPE, BITS, ALIGN, MODE, TOO_LARGE, LAUNCH.
 */
int oasis_lut_gemm(const uint8_t* idx_act, const float* act_scale, int n, int d_in,
                   const uint32_t* idx_w, const float* w_scale, int d_out,
                   const oasis_lut_block* lut, int b_a, int b_w, int algo, float* y,
                   int accumulate, hipStream_t stream);

/*
 * oasis_outlier_compensate - error compensation of the outlier branch
 * (Sec. III-C2; Dequant Unit and MAC units, Sec. IV-A):
 *   Y'[i][j] = s_j * sum_e residual[i][e] * C_W[w(p_e, j)], p_e running over
 *   max_idx[i][0..k) then min_idx[i][0..k).
 *   accumulate != 0 : y += Y'   (merge into the main-branch result);
 *   accumulate == 0 : y  = Y'.
 *   Channel ids must lie in [0, d_in) (ids from oasis_quantize_act do).
 *   k == 0 with accumulate != 0 is a no-op; with accumulate == 0 it zeroes y.
 * Errors: NULL, SHAPE, BITS, K, ALIGN, TOO_LARGE (d_in/8 * d_out * 4 >= 2^31:
 * the codes must be < 2 GiB), LAUNCH.
 */
int oasis_outlier_compensate(const int32_t* max_idx, const int32_t* min_idx, const float* residual,
                             int n, int k, const uint32_t* idx_w, const oasis_lut_block* lut,
                             int b_w, const float* w_scale, int d_in, int d_out, float* y,
                             int accumulate, hipStream_t stream);

/*
 * oasis_outlier_compensate_rows - the same error compensation (Sec. III-C2)
 * from the weight codes in the row layout idx_wr (see oasis_pack_weight_rows):
 * each listed outlier channel p reads exactly row p, d_out/2 bytes, where the
 * idx_w layout costs 4 bytes per (outlier, column).  For many tokens.
 *   idx_wr : DEVICE uint32 [d_in][ceil(d_out/8)]; word m of row p holds the
 *            codes of input channel p for output columns 8m..8m+7, column
 *            8m+c in bits 4c..4c+3 (zero past d_out).
 *   Every other argument, the result and accumulate as in
 *   oasis_outlier_compensate (sums in list order per output).
 * Errors: NULL, SHAPE, BITS, K, ALIGN, TOO_LARGE (d_in * ceil(d_out/8) * 4
 * >= 2^31), LAUNCH.
 */
int oasis_outlier_compensate_rows(const int32_t* max_idx, const int32_t* min_idx,
                                  const float* residual, int n, int k, const uint32_t* idx_wr,
                                  const oasis_lut_block* lut, int b_w, const float* w_scale,
                                  int d_in, int d_out, float* y, int accumulate,
                                  hipStream_t stream);

/*
 * oasis_outlier_compensate_split - the error compensation of Sec. III-C2 for
 * many tokens, split by channel.  Outliers of LLM activations gather in a few
 * channels that most tokens list: channels listed by at least max(2, n / 8)
 * tokens (at most 256 of them, lowest channels first) are compensated
 * together as a dense contraction on the matrix cores (the residuals of a
 * token, scaled by a power of two, as an fp16 hi/lo pair per channel), every
 * other entry by the row-layout kernel of oasis_outlier_compensate_rows over
 * compacted per-token lists.  The result is Y' of oasis_outlier_compensate;
 * which channels count as heavy changes only the fp32 summation order.  (A
 * list naming a channel twice with nonzero residuals has both entries summed,
 * in an order that may vary between runs.)
 *   idx_w     : DEVICE weight codes in the GEMM layout (the dense part reads
 *               the heavy channels' rows from here).
 *   idx_wr    : DEVICE weight codes in the row layout (the other entries).
 *   workspace : DEVICE scratch of at least
 *               oasis_outlier_compensate_split_workspace(n, d_in, d_out, k)
 *               bytes, 256-byte aligned, owned by the caller; overwritten.
 *               Calls that share a workspace must not overlap.
 *   Every other argument, the result and accumulate as in
 *   oasis_outlier_compensate.
 * Errors: NULL, SHAPE, BITS, K, ALIGN, TOO_LARGE (either code layout of
 * 2^31 bytes or more), WORKSPACE, LAUNCH.
 */
size_t oasis_outlier_compensate_split_workspace(int n, int d_in, int d_out, int k);
int oasis_outlier_compensate_split(const int32_t* max_idx, const int32_t* min_idx,
                                   const float* residual, int n, int k, const uint32_t* idx_w,
                                   const uint32_t* idx_wr, const oasis_lut_block* lut, int b_w,
                                   const float* w_scale, int d_in, int d_out, float* y,
                                   int accumulate, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * oasis_lut_gemm_compensated_split - main branch and compensation for many
 * tokens with the heavy channels of oasis_outlier_compensate_split inside the
 * GEMM: the compacted lists of the other entries are compensated first
 * (y = or += their Y'), then the GEMM reduces over the activation codes and
 * over the heavy channels' residuals divided by t_i (fp16 hi/lo pairs) in one
 * pass, y += Y* + Y'.  A heavy channel whose residual over t_i is not below
 * 2^15 (or whose token has t_i = 0) is compensated with the lists instead, so
 * every scale mode gives Y = Y* + Y' of oasis_lut_gemm_compensated up to fp32
 * summation order.
 *   Arguments and results as oasis_lut_gemm_compensated_rows, plus the
 *   workspace of oasis_outlier_compensate_split (the same size query,
 *   oasis_outlier_compensate_split_workspace(n, d_in, d_out, k)).
 *   n <= 32 tokens or k == 0: the call of oasis_lut_gemm_compensated_rows
 *   (no workspace needed).  d_in not a multiple of 64: the split compensation
 *   then the GEMM, two passes over y.
 * Errors: NULL, SHAPE, BITS, K, ALIGN, TOO_LARGE, WORKSPACE, LAUNCH.
 */
int oasis_lut_gemm_compensated_split(const uint8_t* idx_act, const float* act_scale, int n,
                                     int d_in, const uint32_t* idx_w, const uint32_t* idx_wr,
                                     const float* w_scale, int d_out, const oasis_lut_block* lut,
                                     int b_a, int b_w, const int32_t* max_idx,
                                     const int32_t* min_idx, const float* residual, int k,
                                     float* y, int accumulate, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/*
 * oasis_lut_gemm_compensated_split_noalloc - oasis_lut_gemm_compensated_split
 * for callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the workspace is a static
 * device array of 32 MiB inside the library (one per GPU, held until the
 * process ends); the call allocates nothing.  Every call on one GPU shares
 * that array, so calls that overlap on a GPU (other streams, other threads)
 * race; stream-ordered calls do not.
 *   Arguments, results and errors as oasis_lut_gemm_compensated_split without
 *   the workspace; TOO_LARGE when the workspace the call needs
 *   (oasis_outlier_compensate_split_workspace) exceeds 32 MiB.
 */
int oasis_lut_gemm_compensated_split_noalloc(const uint8_t* idx_act, const float* act_scale,
                                             int n, int d_in, const uint32_t* idx_w,
                                             const uint32_t* idx_wr, const float* w_scale,
                                             int d_out, const oasis_lut_block* lut, int b_a,
                                             int b_w, const int32_t* max_idx,
                                             const int32_t* min_idx, const float* residual,
                                             int k, float* y, int accumulate,
                                             hipStream_t stream);

/*
 * oasis_lut_gemm_compensated - main branch and outlier branch in one call
 * (look-ahead computation with error compensation, Sec. III-C):
 *   y (+)= Y* + Y', with Y* as in oasis_lut_gemm and Y' as in
 *   oasis_outlier_compensate (same arguments, same layouts).
 *   For n <= 32 tokens both terms come from one kernel: every workgroup
 *   adds the compensation of its output columns while it streams the
 *   weights, so the outlier branch costs no extra pass.  For larger n the
 *   call runs the MFMA GEMM and then the compensation kernel.
 *   k == 0 (lists may be NULL) gives Y* alone.
 * Errors: NULL, SHAPE, BITS, K, ALIGN, TOO_LARGE, LAUNCH.
 */
int oasis_lut_gemm_compensated(const uint8_t* idx_act, const float* act_scale, int n, int d_in,
                               const uint32_t* idx_w, const float* w_scale, int d_out,
                               const oasis_lut_block* lut, int b_a, int b_w,
                               const int32_t* max_idx, const int32_t* min_idx,
                               const float* residual, int k, float* y, int accumulate,
                               hipStream_t stream);

/*
 * oasis_lut_gemm_compensated_rows - oasis_lut_gemm_compensated with the
 * outlier branch reading the codes in the row layout idx_wr (see
 * oasis_pack_weight_rows) while the main branch streams idx_w: a listed
 * outlier costs 0.5 B per output column instead of 4 B.  For few tokens the
 * call reads idx_wr only when 8 * n * k >= d_in (below that the GEMM layout's
 * rows, which the same launch streams, are cheaper).  Same arguments,
 * results and errors as oasis_lut_gemm_compensated, plus idx_wr (DEVICE,
 * 4-byte aligned; NULL only when k == 0) and TOO_LARGE when
 * d_in * ceil(d_out/8) * 4 >= 2^31.
 */
int oasis_lut_gemm_compensated_rows(const uint8_t* idx_act, const float* act_scale, int n,
                                    int d_in, const uint32_t* idx_w, const uint32_t* idx_wr,
                                    const float* w_scale, int d_out, const oasis_lut_block* lut,
                                    int b_a, int b_w, const int32_t* max_idx,
                                    const int32_t* min_idx, const float* residual, int k,
                                    float* y, int accumulate, hipStream_t stream);

/*
 * oasis_lut_gemm_compensated_percol - oasis_lut_gemm_compensated with an
 * independent weight codebook per output channel: column j's LUT slice is
 * C_A x C_W[j] (the Cartesian product of Sec. III-B, built per 16-column
 * tile in LDS) and the compensation dequantizes with C_W[j] (Sec. III-C2);
 * s_j still scales column j.  A shared codebook is the case of equal rows
 * (bit for bit the same y as oasis_lut_gemm_compensated).
 *   cb_wgt_cols : DEVICE fp16 [d_out][16], 16-byte aligned; entries past
 *                 2^b_w are read but never selected (any finite value).
 *   lut         : a LUT block built with the same b_a (its C_A is used).
 *   Any n: one launch of the GEMV kernel per 32 tokens (each launch
 *   re-reads idx_w, so large n is slower per token than the shared-codebook
 *   prefill kernel).
 * Other arguments, results and errors as oasis_lut_gemm_compensated.
 */
int oasis_lut_gemm_compensated_percol(const uint8_t* idx_act, const float* act_scale, int n,
                                      int d_in, const uint32_t* idx_w, const float* w_scale,
                                      int d_out, const oasis_lut_block* lut,
                                      const uint16_t* cb_wgt_cols, int b_a, int b_w,
                                      const int32_t* max_idx, const int32_t* min_idx,
                                      const float* residual, int k, float* y, int accumulate,
                                      hipStream_t stream);

/*
 * oasis_pack_weight_indices - HOST helper: pack w_idx uint8 [d_in][d_out]
 * (codes 0..15, row-major, host memory) into the idx_w layout above
 * (host memory, d_in/8 * d_out words).  Errors: NULL, SHAPE.
 */
int oasis_pack_weight_indices(const uint8_t* w_idx, int d_in, int d_out, uint32_t* out);

/*
 * oasis_pack_weight_rows - HOST helper: pack w_idx uint8 [d_in][d_out]
 * (codes 0..15, row-major, host memory) into the row layout idx_wr of
 * oasis_outlier_compensate_rows (host memory, d_in * ceil(d_out/8) words;
 * the paper's own layout of the weight index matrix, one input channel per
 * contiguous row).  Errors: NULL, SHAPE.
 */
int oasis_pack_weight_rows(const uint8_t* w_idx, int d_in, int d_out, uint32_t* out);

#ifdef __cplusplus
}
#endif

#endif /* OASIS_H */
