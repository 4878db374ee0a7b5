// Per-token activation quantization with dynamic top-k outlier detection.
//
// One workgroup (256 threads, 4 waves) per token.  The token is staged in LDS
// once; then
//   * the per-token scale t = absmax (Sec. III-A),
//   * the cluster index of every channel by the mid-point boundary rule of the
//     Clustering Unit (Sec. IV-C): a = #{c : x >= fp32(t * b_c)},
//   * the k largest and k smallest channels (the job of the Orizuru engine,
//     Sec. IV-D) with ties to the lower channel, in pop order,
//   * the residual of every listed outlier (Sec. III-C2).
// The top-k is a two-pass radix select on order-preserving 16-bit keys
// (-0 folded into +0) shared by the max and min lists: pass 1 histograms the
// high byte, pass 2 the low byte inside the boundary bucket, which fixes the
// threshold key T and the count G of keys strictly beyond it.  Keys beyond T
// are ranked among themselves (G < k of them); keys equal to T are taken in
// channel order, which a block-wide scan provides.  The paper's tree pops in
// exactly this order; the select needs 2 histogram passes instead of k pops.
#include "common.h"

namespace oasis {

constexpr int QT = 256;

struct QuantSmem {
  uint32_t hist1[256];
  uint32_t hist2_max[256];
  uint32_t hist2_min[256];
  float ca[16];
  uint32_t scan_tmp[4];
  uint32_t red_tmp[4];
  uint32_t ctl[8];  // B1/G1 of max & min, then T/G/need
};

size_t quantize_lds_bytes(int d_in, int k) {
  size_t xs = ((size_t)d_in * 2 + 15) / 16 * 16;
  size_t bitmap = (((size_t)d_in + 31) / 32) * 4;
  size_t cand = (size_t)k * 4;
  return sizeof(QuantSmem) + xs + ((bitmap + 15) / 16) * 16 + cand;
}

__device__ __forceinline__ uint32_t ord_key(uint32_t bits) {
  if (bits == 0x8000u) bits = 0;  // -0 == +0
  return (bits & 0x8000u) ? (~bits & 0xFFFFu) : (bits | 0x8000u);
}

// Inclusive scan of one value per thread over the 256-thread block.
__device__ __forceinline__ uint32_t block_scan(uint32_t v, uint32_t* tmp) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    uint32_t u = __shfl_up(v, off, 64);
    if (lane >= off) v += u;
  }
  if (lane == 63) tmp[wid] = v;
  __syncthreads();
  uint32_t base = 0;
  for (int w = 0; w < wid; ++w) base += tmp[w];
  __syncthreads();
  return v + base;
}

__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* tmp) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, (uint32_t)__shfl_xor(v, off, 64));
  if (lane == 0) tmp[wid] = v;
  __syncthreads();
  uint32_t r = max(max(tmp[0], tmp[1]), max(tmp[2], tmp[3]));
  __syncthreads();
  return r;
}

__global__ void __launch_bounds__(QT) k_quantize(QuantArgs A) {
#pragma clang fp contract(off)
  extern __shared__ __align__(16) unsigned char smem_raw[];
  QuantSmem& S = *reinterpret_cast<QuantSmem*>(smem_raw);
  const int d_in = A.d_in, k = A.k;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem_raw + sizeof(QuantSmem));
  const size_t xs_bytes = ((size_t)d_in * 2 + 15) / 16 * 16;
  uint32_t* bitmap = reinterpret_cast<uint32_t*>(smem_raw + sizeof(QuantSmem) + xs_bytes);
  const int bm_words = (d_in + 31) / 32;
  uint32_t* cand = bitmap + ((bm_words + 3) / 4) * 4;

  const int tid = threadIdx.x;
  const int i = blockIdx.x;
  const uint16_t* xrow = A.x + (size_t)i * d_in;

  // ---- stage the token in LDS (coalesced 16-byte loads) and find absmax
  uint32_t amax = 0;
  const int nvec = d_in / 8;
  for (int v = tid; v < nvec; v += QT) {
    uint4 q = reinterpret_cast<const uint4*>(xrow)[v];
    reinterpret_cast<uint4*>(xs)[v] = q;
    uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      amax = max(amax, w[h] & 0x7FFFu);
      amax = max(amax, (w[h] >> 16) & 0x7FFFu);
    }
  }
  for (int b = tid; b < 256; b += QT) {
    S.hist1[b] = 0;
    S.hist2_max[b] = 0;
    S.hist2_min[b] = 0;
  }
  for (int w = tid; w < bm_words; w += QT) bitmap[w] = 0;
  if (tid < 16) S.ca[tid] = h2f(A.lut->cb_act[tid]);
  amax = block_max(amax, S.red_tmp);  // contains a barrier

  const float t = (A.scale_mode == OASIS_SCALE_NONE) ? 1.0f : h2f((uint16_t)amax);
  if (tid == 0) A.act_scale[i] = t;

  // ---- scaled cluster boundaries P_c = fp32(t * b_c), b_c = (c_c + c_{c+1}) * 0.5
  const int nb = (1 << A.b_a) - 1;
  float P[15];
#pragma unroll
  for (int c = 0; c < 15; ++c) {
    float bc = (S.ca[c] + S.ca[c + 1]) * 0.5f;
    P[c] = t * bc;
  }

  // ---- cluster index of every channel, packed 8 per word
  uint32_t* arow = reinterpret_cast<uint32_t*>(A.idx_act + (size_t)i * (d_in / 2));
  for (int v = tid; v < nvec; v += QT) {
    uint4 q = reinterpret_cast<const uint4*>(xs)[v];
    uint32_t w[4] = {q.x, q.y, q.z, q.w};
    uint32_t packed = 0;
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      float x = h2f((uint16_t)(w[h >> 1] >> (16 * (h & 1))));
      uint32_t a = 0;
#pragma unroll
      for (int c = 0; c < 15; ++c) a += (c < nb && x >= P[c]) ? 1u : 0u;
      packed |= a << (4 * h);
    }
    arow[v] = packed;
  }
  if (k == 0) return;  // uniform across the block
  if (tid == 0) {
    S.ctl[0] = 0; S.ctl[1] = 0; S.ctl[2] = 0; S.ctl[3] = 0;
    S.ctl[4] = 0; S.ctl[5] = 0; S.ctl[6] = 0; S.ctl[7] = 0;
  }

  // ---- pass 1: histogram of the key's high byte (shared by both lists)
  for (int p = tid; p < d_in; p += QT) atomicAdd(&S.hist1[ord_key(xs[p]) >> 8], 1u);
  __syncthreads();
  {
    const uint32_t h = S.hist1[tid];
    const uint32_t pre = block_scan(h, S.scan_tmp);  // # keys with high byte <= tid
    const uint32_t total = (uint32_t)d_in;
    const uint32_t suf_excl = total - pre;           // # keys with high byte > tid
    if (suf_excl < (uint32_t)k && (uint32_t)k <= suf_excl + h) {
      S.ctl[0] = tid;
      S.ctl[1] = suf_excl;
    }
    const uint32_t pre_excl = pre - h;
    if (pre_excl < (uint32_t)k && (uint32_t)k <= pre) {
      S.ctl[2] = tid;
      S.ctl[3] = pre_excl;
    }
  }
  __syncthreads();
  const uint32_t B1max = S.ctl[0], G1max = S.ctl[1], B1min = S.ctl[2], G1min = S.ctl[3];

  // ---- pass 2: low byte inside the two boundary buckets
  for (int p = tid; p < d_in; p += QT) {
    uint32_t key = ord_key(xs[p]);
    if ((key >> 8) == B1max) atomicAdd(&S.hist2_max[key & 255u], 1u);
    if ((key >> 8) == B1min) atomicAdd(&S.hist2_min[key & 255u], 1u);
  }
  __syncthreads();
  {
    const uint32_t hm = S.hist2_max[tid];
    const uint32_t pre_m = block_scan(hm, S.scan_tmp);
    const uint32_t tot_m = S.scan_tmp[0] + S.scan_tmp[1] + S.scan_tmp[2] + S.scan_tmp[3];
    const uint32_t kk = (uint32_t)k - G1max;
    const uint32_t suf_excl = tot_m - pre_m;
    const uint32_t hn = S.hist2_min[tid];
    __syncthreads();
    const uint32_t pre_n = block_scan(hn, S.scan_tmp);
    const uint32_t kn = (uint32_t)k - G1min;
    const uint32_t pre_excl = pre_n - hn;
    if (suf_excl < kk && kk <= suf_excl + hm) {
      S.ctl[4] = (B1max << 8) | tid;  // threshold key of the max list
      S.ctl[5] = G1max + suf_excl;    // keys strictly greater
    }
    if (pre_excl < kn && kn <= pre_n) {
      S.ctl[6] = (B1min << 8) | tid;  // threshold key of the min list
      S.ctl[7] = G1min + pre_excl;    // keys strictly smaller
    }
  }
  __syncthreads();
  // G < k holds by construction; the clamp only keeps every index in bounds.
  const uint32_t Tmax = S.ctl[4], Tmin = S.ctl[6];
  const uint32_t Gmax = min(S.ctl[5], (uint32_t)k - 1u), Gmin = min(S.ctl[7], (uint32_t)k - 1u);

  // Each thread owns a contiguous run of channels so ties are ranked in
  // channel order by one block scan.
  const int chunk = (d_in + QT - 1) / QT;
  const int p0 = min(d_in, tid * chunk), p1 = min(d_in, p0 + chunk);
  const size_t krow = (size_t)i * k;
  const size_t rrow = (size_t)i * 2 * k;

  auto residual_of = [&](int p) -> float {
    float x = h2f(xs[p]);
    uint32_t a = 0;
#pragma unroll
    for (int c = 0; c < 15; ++c) a += (c < nb && x >= P[c]) ? 1u : 0u;
    float xhat = t * S.ca[a];  // exact: a product of two fp16 values
    return x - xhat;
  };

  // ---- max list
  {
    uint32_t ties = 0;
    for (int p = p0; p < p1; ++p) ties += (ord_key(xs[p]) == Tmax) ? 1u : 0u;
    uint32_t tie_rank = block_scan(ties, S.scan_tmp) - ties;
    if (tid == 0) S.red_tmp[0] = 0;  // candidate counter
    __syncthreads();
    const uint32_t need = (uint32_t)k - Gmax;
    for (int p = p0; p < p1; ++p) {
      uint32_t key = ord_key(xs[p]);
      if (key > Tmax) {
        uint32_t slot = atomicAdd(&S.red_tmp[0], 1u);
        if (slot < Gmax) cand[slot] = (key << 16) | (0xFFFFu - (uint32_t)p);
      } else if (key == Tmax) {
        if (tie_rank < need) {
          uint32_t pos = Gmax + tie_rank;
          A.max_idx[krow + pos] = p;
          A.residual[rrow + pos] = residual_of(p);
          atomicOr(&bitmap[p >> 5], 1u << (p & 31));
        }
        ++tie_rank;
      }
    }
    __syncthreads();
    for (uint32_t s = tid; s < Gmax; s += QT) {
      const uint32_t key = cand[s];
      uint32_t rank = 0;
      for (uint32_t q = 0; q < Gmax; ++q) rank += (cand[q] > key) ? 1u : 0u;
      const int p = (int)(0xFFFFu - (key & 0xFFFFu));
      A.max_idx[krow + rank] = p;
      A.residual[rrow + rank] = residual_of(p);
      atomicOr(&bitmap[p >> 5], 1u << (p & 31));
    }
    __syncthreads();
  }

  // ---- min list (a channel already in the max list gets residual 0)
  {
    uint32_t ties = 0;
    for (int p = p0; p < p1; ++p) ties += (ord_key(xs[p]) == Tmin) ? 1u : 0u;
    uint32_t tie_rank = block_scan(ties, S.scan_tmp) - ties;
    if (tid == 0) S.red_tmp[1] = 0;
    __syncthreads();
    const uint32_t need = (uint32_t)k - Gmin;
    auto emit = [&](uint32_t pos, int p) {
      A.min_idx[krow + pos] = p;
      const bool dup = (bitmap[p >> 5] >> (p & 31)) & 1u;
      A.residual[rrow + k + pos] = dup ? 0.0f : residual_of(p);
    };
    for (int p = p0; p < p1; ++p) {
      uint32_t key = ord_key(xs[p]);
      if (key < Tmin) {
        uint32_t slot = atomicAdd(&S.red_tmp[1], 1u);
        if (slot < Gmin) cand[slot] = (key << 16) | (uint32_t)p;
      } else if (key == Tmin) {
        if (tie_rank < need) emit(Gmin + tie_rank, p);
        ++tie_rank;
      }
    }
    __syncthreads();
    for (uint32_t s = tid; s < Gmin; s += QT) {
      const uint32_t key = cand[s];
      uint32_t rank = 0;
      for (uint32_t q = 0; q < Gmin; ++q) rank += (cand[q] < key) ? 1u : 0u;
      emit(rank, (int)(key & 0xFFFFu));
    }
  }
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  size_t lds = quantize_lds_bytes(a.d_in, a.k);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k_quantize,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_quantize, dim3(a.n), dim3(QT), lds, s, a);
  return hipGetLastError();
}

}  // namespace oasis
