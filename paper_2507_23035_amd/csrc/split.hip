// Error compensation of many tokens (Sec. III-C2) split by channel:
//   Y'[i][j] = s_j * sum_e r_ie * C_W[w(p_ie, j)]
//            = s_j * sum_{h in H} R[i][h] * C_W[w(h, j)]        (heavy channels)
//            + s_j * sum_{e : p_ie not in H} r_ie * C_W[w(p_ie, j)] (the rest)
// with R[i][h] the residual of token i at heavy channel h (0 when the token
// does not list it).  Activation outliers of LLMs gather in a few channels
// that most tokens list, so the first sum is a dense contraction over a short
// reduction: it runs on the matrix cores (the many-token MFMA kernel with an
// fp16 value operand), the second on the row-layout kernel over compacted
// lists.
//
// Dense operand: R is scaled per token by a power of two 2^-E_i (exact) so
// that |R 2^-E_i| < 2, then split into fp16 hi = fp16(v) and lo = fp16(v - hi);
// hi + lo equals v to about 2^-22 relative, and C_W values are exact fp16, so
// the products carry no more error than the fp32 sums.  Positions 2h and 2h+1
// of the reduction are the hi and lo halves of heavy channel h, both paired
// with channel h's weight code; the kernel's per-token scale is 2^E_i.
//
// Heavy channels: listed by at least max(2, n / 8) tokens (a live entry:
// nonzero residual, channel in range), the first kSplitHeavy of them in
// channel order.  Which channels are heavy changes only the summation order.
#include <algorithm>
#include <mutex>

#include "common.h"

namespace oasis {

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

SplitLayout split_layout(int n, int d_in, int d_out, int k) {
  SplitLayout L;
  size_t o = 0;
  const size_t E = 2 * (size_t)k;
  L.count = o; o += align256(4 * (size_t)d_in);
  L.slot = o; o += align256(4 * (size_t)d_in);
  L.hlist = o; o += align256(4 * (size_t)(kSplitHeavy + 1));  // + the count nh
  L.pow2 = o; o += align256(4 * (size_t)n);
  L.rh = o; o += align256(2 * (size_t)kSplitPos * n);
  L.idxh = o; o += align256(4 * (size_t)(kSplitPos / 8) * d_out);
  L.spp = o; o += align256(4 * E * n);
  L.spr = o; o += align256(4 * E * n);
  L.spc = o; o += align256(4 * (size_t)n);
  L.total = o;
  return L;
}

// entry f of the lists: token f / 2k, place f mod 2k; live when its
// residual is nonzero and its channel in range
__device__ __forceinline__ bool split_entry(const CompArgs& A, size_t f, int& p, float& r) {
  const int E = 2 * A.k;
  const size_t i = f / (size_t)E;
  const int e = (int)(f - i * (size_t)E);
  p = e < A.k ? A.max_idx[i * A.k + e] : A.min_idx[i * A.k + (e - A.k)];
  r = A.residual[i * (size_t)E + e];
  return r != 0.0f && p >= 0 && p < A.d_in;
}

// how many tokens list each channel.  LDS: a histogram of the workgroup's
// share of the entries (d_in <= kSplitLdsBins), flushed with one global add
// per touched channel - the heavy channels are listed by most tokens, and
// global atomics on them from every entry would serialize.
constexpr int kSplitLdsBins = 16384;
template <bool LDS, int NT>
__global__ void __launch_bounds__(NT) k_split_count(CompArgs A, int* __restrict__ count) {
  __shared__ int hist[LDS ? kSplitLdsBins : 1];
  const size_t tot = (size_t)A.n * 2 * A.k;
  if constexpr (LDS) {
    for (int p = threadIdx.x; p < A.d_in; p += NT) hist[p] = 0;
    __syncthreads();
  }
  // eight entries' loads in flight before their counts
  constexpr int U = 8;
  const size_t stride = (size_t)gridDim.x * NT;
  for (size_t f0 = (size_t)blockIdx.x * NT + threadIdx.x; f0 < tot; f0 += U * stride) {
    int p[U];
    float r[U];
    bool live[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t f = f0 + (size_t)u * stride;
      live[u] = f < tot && split_entry(A, f, p[u], r[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (live[u]) {
        if constexpr (LDS) atomicAdd(&hist[p[u]], 1);
        else atomicAdd(&count[p[u]], 1);
      }
    }
  }
  if constexpr (LDS) {
    __syncthreads();
    for (int p = threadIdx.x; p < A.d_in; p += NT)
      if (hist[p]) atomicAdd(&count[p], hist[p]);
  }
}

// heavy channels in channel order: slot[p] = index in the list or -1;
// hlist[0..nh) = the channels, hlist[kSplitHeavy] = nh; one workgroup
__global__ void __launch_bounds__(1024) k_split_select(int d_in, int thr,
                                                        const int* __restrict__ count,
                                                        int* __restrict__ slot,
                                                        int* __restrict__ hlist) {
  __shared__ uint64_t tmp[16];
  __shared__ int total;
  const int t = threadIdx.x;
  const int per = (d_in + 1023) / 1024;
  const int p0 = min(d_in, t * per), p1 = min(d_in, p0 + per);
  // the counts of up to 16 channels per thread are read at once (d_in <=
  // 16384, the LDS count's limit; beyond it, a second pass reads them again)
  constexpr int PR = 16;
  int cnt[PR];
#pragma unroll
  for (int q = 0; q < PR; ++q) cnt[q] = p0 + q < p1 ? count[p0 + q] : 0;
  uint64_t mine = 0;
#pragma unroll
  for (int q = 0; q < PR; ++q) mine += cnt[q] >= thr;
  for (int p = p0 + PR; p < p1; ++p) mine += count[p] >= thr;
  const uint64_t incl = block_scan64<1024>(mine, tmp);
  int idx = (int)(incl - mine);
  auto place = [&](int p, int c) {
    int sl = -1;
    if (c >= thr) {
      if (idx < kSplitHeavy) {
        sl = idx;
        hlist[idx] = p;
      }
      ++idx;
    }
    slot[p] = sl;
  };
#pragma unroll
  for (int q = 0; q < PR; ++q)
    if (p0 + q < p1) place(p0 + q, cnt[q]);
  for (int p = p0 + PR; p < p1; ++p) place(p, count[p]);
  if (t == 1023) total = (int)min((uint64_t)kSplitHeavy, incl);  // the last prefix is the total
  __syncthreads();
  const int nh = total;
  if (t == 0) hlist[kSplitHeavy] = nh;
  for (int h = nh + t; h < kSplitHeavy; h += 1024) hlist[h] = -1;
}

// One wave per token: the token's heavy residuals summed per heavy channel
// (in LDS, fp32), scaled and split into the fp16 hi/lo row of the dense
// operand; the other live entries compacted in list order.
//   tscale == nullptr: the dense part runs on its own and the token's scale
//     is a power of two 2^E_i with |R 2^-E_i| < 2 (pow2[i] = 2^E_i).
//   tscale != nullptr: the dense part joins the main-branch GEMM, whose
//     epilogue multiplies by t_i, so the operand is R / t_i.  A channel whose
//     R / t_i is not below 2^15 in magnitude (or whose token has t_i = 0 and
//     R != 0) leaves the dense operand (0 there) and its entries join the
//     compacted lists, so any scale mode stays exact.
__global__ void __launch_bounds__(64) k_split_rows(CompArgs A, const int* __restrict__ slot,
                                                   const float* __restrict__ tscale,
                                                   float* __restrict__ pow2,
                                                   uint16_t* __restrict__ rh,
                                                   int32_t* __restrict__ spp,
                                                   float* __restrict__ spr,
                                                   int32_t* __restrict__ spc) {
  __shared__ float acc[kSplitHeavy];
  __shared__ int out[kSplitHeavy];  // heavy channel handled by the lists instead
  const int i = blockIdx.x, lane = threadIdx.x;
  const int E = 2 * A.k;
  for (int h = lane; h < kSplitHeavy; h += 64) {
    acc[h] = 0.0f;
    out[h] = 0;
  }
  __builtin_amdgcn_wave_barrier();
  for (int e0 = 0; e0 < E; e0 += 64) {
    const int e = e0 + lane;
    int p = -1;
    float r = 0.0f;
    if (e < E && split_entry(A, (size_t)i * E + e, p, r)) {
      const int sl = slot[p];
      if (sl >= 0) atomicAdd(&acc[sl], r);
    }
  }
  __builtin_amdgcn_wave_barrier();
  float down;
  if (tscale) {
    const float t = tscale[i];
    for (int h = lane; h < kSplitHeavy; h += 64) {
      const float v = acc[h];
      if (v == 0.0f) continue;
      const float q = t > 0.0f ? v / t : INFINITY;
      if (!(fabsf(q) < 32768.0f)) {
        out[h] = 1;
        acc[h] = 0.0f;
      } else {
        acc[h] = q;
      }
    }
    down = 1.0f;
  } else {
    // per-token power of two: |acc| * 2^-E < 2
    float m = 0.0f;
    for (int h = lane; h < kSplitHeavy; h += 64) m = fmaxf(m, fabsf(acc[h]));
    const float mx = __builtin_bit_cast(float, wave_max(__builtin_bit_cast(uint32_t, m)));
    const int ex = mx > 0.0f ? ilogbf(mx) : 0;
    down = ldexpf(1.0f, -ex);
    if (lane == 0) pow2[i] = ldexpf(1.0f, ex);
  }
  __builtin_amdgcn_wave_barrier();
  // the compacted lists: live entries of channels that are not heavy (or left
  // the dense operand), in list order
  uint32_t base = 0;
  for (int e0 = 0; e0 < E; e0 += 64) {
    const int e = e0 + lane;
    int p = -1;
    float r = 0.0f;
    bool sparse = false;
    if (e < E && split_entry(A, (size_t)i * E + e, p, r)) {
      const int sl = slot[p];
      sparse = sl < 0 || out[sl];
    }
    const uint64_t m = __ballot(sparse);
    const uint32_t before = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (sparse) {
      spp[(size_t)i * E + base + before] = p;
      spr[(size_t)i * E + base + before] = r;
    }
    base += (uint32_t)__popcll(m);
  }
  // lane l writes positions 8l .. 8l + 7 (heavy channels 4l .. 4l + 3)
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float v = acc[4 * lane + q] * down;
    const _Float16 hi = (_Float16)v;
    const _Float16 lo = (_Float16)(v - (float)hi);
    w[q] = (uint32_t)__builtin_bit_cast(uint16_t, hi) |
           ((uint32_t)__builtin_bit_cast(uint16_t, lo) << 16);
  }
  reinterpret_cast<uint4_t*>(rh + (size_t)i * kSplitPos)[lane] = uint4_t{w[0], w[1], w[2], w[3]};
  if (lane == 0) spc[i] = (int)base;
}

// Weight codes of the dense positions in the GEMM layout: word (q, j) holds
// positions 8q .. 8q + 7 of column j, i.e. heavy channels 4q .. 4q + 3 each
// twice (hi and lo); positions past the list get code 0 (their operand is 0).
__global__ void __launch_bounds__(256) k_split_wgather(const uint32_t* __restrict__ idx_w,
                                                       int d_out, const int* __restrict__ hlist,
                                                       uint32_t* __restrict__ idxh) {
  const int q = blockIdx.y;
  const int nh = hlist[kSplitHeavy];
  if (8 * q >= ((2 * nh + 63) / 64) * 64) return;  // beyond the blocks the kernel reads
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= d_out) return;
  uint32_t word = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = hlist[4 * q + u];
    uint32_t code = 0;
    if (c >= 0) code = (idx_w[(size_t)(c >> 3) * d_out + j] >> (4 * (c & 7))) & 15u;
    word |= (code | (code << 4)) << (8 * u);
  }
  idxh[(size_t)q * d_out + j] = word;
}

// Heavy channels, dense operand rows, heavy weight codes and compacted lists
// (tscale: see k_split_rows).
static hipError_t split_prepass(const CompArgs& a, const uint32_t* idx_w_gemm, void* ws,
                                const float* tscale, hipStream_t s) {
  const SplitLayout L = split_layout(a.n, a.d_in, a.d_out, a.k);
  char* base = static_cast<char*>(ws);
  int* count = reinterpret_cast<int*>(base + L.count);
  int* slot = reinterpret_cast<int*>(base + L.slot);
  int* hlist = reinterpret_cast<int*>(base + L.hlist);
  float* pow2 = reinterpret_cast<float*>(base + L.pow2);
  uint16_t* rh = reinterpret_cast<uint16_t*>(base + L.rh);
  uint32_t* idxh = reinterpret_cast<uint32_t*>(base + L.idxh);
  int32_t* spp = reinterpret_cast<int32_t*>(base + L.spp);
  float* spr = reinterpret_cast<float*>(base + L.spr);
  int32_t* spc = reinterpret_cast<int32_t*>(base + L.spc);

  hipError_t e = launch_fill_zero(reinterpret_cast<float*>(count), (size_t)a.d_in, s);
  if (e != hipSuccess) return e;
  const size_t tot = (size_t)a.n * 2 * a.k;
  if (a.d_in <= kSplitLdsBins) {
    // at most 64 workgroups of 1024 threads: each flushes the counts it
    // touched with global adds (the heavy channels' counters serialize).
    // Measured at 4096 x 8192 x 28672 (k = 64): 16 workgroups 22.6 us, 32
    // 13.4, 64 8.8, 128 8.5, 256 10.8; at 2048 tokens 64 was the fastest
    const unsigned cblocks = (unsigned)std::min<size_t>((tot + 1023) / 1024, 64);
    hipLaunchKernelGGL((k_split_count<true, 1024>), dim3(cblocks), dim3(1024), 0, s, a, count);
  } else {
    const unsigned cblocks = (unsigned)std::min<size_t>((tot + 255) / 256, 4096);
    hipLaunchKernelGGL((k_split_count<false, 256>), dim3(cblocks), dim3(256), 0, s, a, count);
  }
  const int thr = std::max(2, a.n / 8);
  hipLaunchKernelGGL(k_split_select, dim3(1), dim3(1024), 0, s, a.d_in, thr, count, slot, hlist);
  hipLaunchKernelGGL(k_split_rows, dim3(a.n), dim3(64), 0, s, a, slot, tscale, pow2, rh, spp,
                     spr, spc);
  hipLaunchKernelGGL(k_split_wgather, dim3((a.d_out + 255) / 256, kSplitPos / 8), dim3(256), 0, s,
                     idx_w_gemm, a.d_out, hlist, idxh);
  return hipGetLastError();
}

// The compacted lists of the workspace as the row-layout kernel's lists.
static CompArgs sparse_args(const CompArgs& a, void* ws, int accumulate) {
  const SplitLayout L = split_layout(a.n, a.d_in, a.d_out, a.k);
  char* base = static_cast<char*>(ws);
  CompArgs c = a;
  c.max_idx = reinterpret_cast<const int32_t*>(base + L.spp);
  c.min_idx = nullptr;
  c.residual = reinterpret_cast<const float*>(base + L.spr);
  c.cnt = reinterpret_cast<const int32_t*>(base + L.spc);
  c.accumulate = accumulate;
  return c;
}

hipError_t launch_compensate_split(const CompArgs& a, const uint32_t* idx_w_gemm, void* ws,
                                   hipStream_t s) {
  if (a.n == 0 || a.d_out == 0) return hipSuccess;
  if (a.k == 0) {
    if (a.accumulate) return hipSuccess;
    return launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
  }
  hipError_t e = split_prepass(a, idx_w_gemm, ws, nullptr, s);
  if (e != hipSuccess) return e;
  const SplitLayout L = split_layout(a.n, a.d_in, a.d_out, a.k);
  char* base = static_cast<char*>(ws);
  int* hlist = reinterpret_cast<int*>(base + L.hlist);
  float* pow2 = reinterpret_cast<float*>(base + L.pow2);
  uint16_t* rh = reinterpret_cast<uint16_t*>(base + L.rh);
  uint32_t* idxh = reinterpret_cast<uint32_t*>(base + L.idxh);

  // dense part: y (+)= 2^E_i * s_j * sum_q R~[i][q] C_W[w(q, j)]
  GemmArgs g{};
  g.idx_act = reinterpret_cast<const uint8_t*>(rh);
  g.act_scale = pow2;
  g.n = a.n;
  g.d_in = kSplitPos;
  g.idx_w = idxh;
  g.w_scale = a.w_scale;
  g.d_out = a.d_out;
  g.lut = a.lut;
  g.b_a = 4;
  g.b_w = a.b_w;
  g.y = a.y;
  g.accumulate = a.accumulate;
  g.kdyn = hlist + kSplitHeavy;
  g.a_row = 2 * kSplitPos;
  if ((e = launch_gemm_values(g, s)) != hipSuccess) return e;

  // the rest: y += Y' of the compacted lists
  return launch_compensate_wr(sparse_args(a, ws, 1), s);
}

// Main branch and compensation with the heavy channels inside the GEMM: the
// GEMM over the codes and the dense positions (y (+)= Y* + Y' of the heavy
// channels), then the compacted lists (y += their Y').  g: the main GEMM's
// arguments (n > 32 tokens, d_in % 64 == 0).
hipError_t launch_gemm_compensated_split(const GemmArgs& g, const CompArgs& a,
                                         const uint32_t* idx_w_gemm, void* ws, hipStream_t s) {
  hipError_t e = split_prepass(a, idx_w_gemm, ws, g.act_scale, s);
  if (e != hipSuccess) return e;
  // the GEMM (with the heavy channels) first, with the caller's accumulate;
  // the lists' kernel then adds into y.  That kernel hides the read of y
  // behind its arithmetic, where the GEMM's epilogue would wait for it.
  const SplitLayout L = split_layout(a.n, a.d_in, a.d_out, a.k);
  char* base = static_cast<char*>(ws);
  GemmArgs m = g;
  m.accumulate = a.accumulate;
  m.nheavy = reinterpret_cast<const int*>(base + L.hlist) + kSplitHeavy;
  m.hv = reinterpret_cast<const uint8_t*>(base + L.rh);
  m.hw = reinterpret_cast<const uint32_t*>(base + L.idxh);
  // (expanding the activation codes once, to fp16 values the GEMM reads,
  // measured slower: 3.29 vs 2.73 ms at 4096x8192x28672 - four times the
  // activation bytes through L2 for every column tile)
  if ((e = launch_gemm_heavy(m, s)) != hipSuccess) return e;
  return launch_compensate_wr(sparse_args(a, ws, 1), s);
}

// ----------------------------------------------------------------------------
// The same call without a caller workspace, for callers that cannot allocate
// (HIP graph capture, tight serving loops): the scratch is a file-scope device
// array of kScratchBytes that every GPU the library runs on holds until the
// process ends.  Its device address (per device, taken with that device
// current on the first call there) is what the kernels receive; the array's
// name in host code is only a stand-in for it.  Every call on one GPU shares
// the array: calls that overlap on a GPU race.  What must start at zero (the
// channel counts) is cleared by a fill kernel in every call.
// ----------------------------------------------------------------------------
constexpr size_t kScratchBytes = 32u << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (nullptr on error).
void* scratch_address() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

}  // namespace oasis

extern "C" int oasis_lut_gemm_compensated_split_noalloc(
    const uint8_t* idx_act, const float* act_scale, int n, int d_in, const uint32_t* idx_w,
    const uint32_t* idx_wr, const float* w_scale, int d_out, const oasis_lut_block* lut, int b_a,
    int b_w, const int32_t* max_idx, const int32_t* min_idx, const float* residual, int k,
    float* y, int accumulate, hipStream_t stream) {
  if (n < 0 || d_in < 0 || d_out < 0 || k < 0) return OASIS_ERR_SHAPE;
  if ((size_t)oasis_outlier_compensate_split_workspace(n, d_in, d_out, k) > oasis::kScratchBytes)
    return OASIS_ERR_TOO_LARGE;
  void* ws = oasis::scratch_address();
  if (!ws) return OASIS_ERR_LAUNCH;
  return oasis_lut_gemm_compensated_split(idx_act, act_scale, n, d_in, idx_w, idx_wr, w_scale,
                                          d_out, lut, b_a, b_w, max_idx, min_idx, residual, k, y,
                                          accumulate, ws, oasis::kScratchBytes, stream);
}
