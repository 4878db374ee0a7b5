// Per-token activation quantization with dynamic top-k outlier detection.
//
// One workgroup per token.  The token is staged in LDS once; then
//   * the per-token scale t = absmax (Sec. III-A),
//   * the cluster index of every channel by the mid-point boundary rule of the
//     Clustering Unit (Sec. IV-C): a = #{c : x >= fp32(t * b_c)},
//   * the k largest and k smallest channels (the job of the Orizuru engine,
//     Sec. IV-D) with ties to the lower channel, in pop order,
//   * the residual of every listed outlier (Sec. III-C2).
// The top-k is a two-pass radix select on order-preserving 16-bit keys
// (-0 folded into +0) shared by the max and min lists: pass 1 histograms the
// high byte while the token is staged, pass 2 the low byte inside the boundary
// bucket, which fixes the
// threshold key T and the count G of keys strictly beyond it.  Keys beyond T
// (G < k of them) are ranked among themselves, one lane per candidate; keys
// equal to T are taken in channel order, which one block-wide scan provides.  The
// paper's tree pops in exactly this order; the select needs two histogram
// passes instead of k pops.
//
// Each thread owns a contiguous run of channels (a multiple of 8, read from
// LDS as 16-byte vectors), so channel order inside a tie is the order of the
// block scan; the pass that counts ties also writes the run's cluster codes.  Small batches use 512-thread workgroups (short runs, latency
// bound), large batches 256-thread ones (many tokens per CU).
#include "common.h"

namespace oasis {

template <int NT>
struct QuantSmem {
  uint32_t hist1[256];
  uint16_t bucket[256];  // per high byte of the key: first | last cluster index << 8
  float P[16];           // scaled boundaries
  uint32_t hist2_max[256];
  uint32_t hist2_min[256];
  float ca[16];
  uint64_t scan_tmp[3][NT / 64];  // one per block scan: no barrier between reuses
  uint32_t red_tmp[NT / 64];
  uint32_t ctl[8];    // B1/G1 of the max and min lists, then T/G of both
};

// Dynamic LDS after the fixed part: token (2 B per channel, 16-byte padded),
// max candidates (4 B each), min candidates (4 B + a 4-byte duplicate flag).
static size_t dyn_bytes(int d_in, int k) {
  size_t xs = ((size_t)d_in * 2 + 15) / 16 * 16;
  return xs + (size_t)k * 12;
}

size_t quantize_lds_bytes(int d_in, int k) {
  return sizeof(QuantSmem<1024>) + dyn_bytes(d_in, k);
}

__device__ __forceinline__ uint32_t ord_key(uint32_t bits) {
  if (bits == 0x8000u) bits = 0;  // -0 == +0
  return (bits & 0x8000u) ? (~bits & 0xFFFFu) : (bits | 0x8000u);
}

template <int NT>
__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* tmp) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, (uint32_t)__shfl_xor(v, off, 64));
  if (lane == 0) tmp[wid] = v;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) r = max(r, tmp[w]);
  return r;  // `tmp` is not reused: no trailing barrier
}

// CLUSTER: write scale and codes.  TOPK: write outlier lists and residuals.
template <int NT, bool CLUSTER, bool TOPK>
__global__ void __launch_bounds__(NT) k_quantize(QuantArgs A) {
#pragma clang fp contract(off)
  extern __shared__ __align__(16) unsigned char smem_raw[];
  QuantSmem<NT>& S = *reinterpret_cast<QuantSmem<NT>*>(smem_raw);
  const int d_in = A.d_in, k = A.k;
  unsigned char* dyn = smem_raw + sizeof(QuantSmem<NT>);
  uint16_t* xs = reinterpret_cast<uint16_t*>(dyn);
  const size_t xs_bytes = ((size_t)d_in * 2 + 15) / 16 * 16;
  uint32_t* cand_max = reinterpret_cast<uint32_t*>(dyn + xs_bytes);
  uint32_t* cand_min = cand_max + k;
  uint32_t* cand_dup = cand_min + k;

  const int tid = threadIdx.x;
  const int i = blockIdx.x;
  const uint16_t* xrow = A.x + (size_t)i * d_in;
  const uint4* xs4 = reinterpret_cast<const uint4*>(xs);

  const bool topk = TOPK && k > 0;                 // uniform across the block
  const bool fused_cluster = CLUSTER && topk;      // codes written by the count pass
  if (tid < 256) {
    S.hist1[tid] = 0;
    S.hist2_max[tid] = 0;
    S.hist2_min[tid] = 0;
  }
  if (tid < 16) S.ca[tid] = h2f(A.lut->cb_act[tid]);
  if (tid < 8) S.ctl[tid] = 0;
  __syncthreads();  // histograms cleared

  // ---- stage the token in LDS (coalesced 16-byte loads), find absmax and
  // build the histogram of the key's high byte (pass 1 of the top-k select)
  uint32_t amax = 0;
  const int nvec = d_in / 8;
  for (int v = tid; v < nvec; v += NT) {
    uint4 q = reinterpret_cast<const uint4*>(xrow)[v];
    reinterpret_cast<uint4*>(xs)[v] = q;
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) amax = max(amax, max(w[h] & 0x7FFFu, (w[h] >> 16) & 0x7FFFu));
    if (topk) {
#pragma unroll
      for (int h = 0; h < 8; ++h)
        atomicAdd(&S.hist1[ord_key((w[h >> 1] >> (16 * (h & 1))) & 0xFFFFu) >> 8], 1u);
    }
  }
  amax = block_max<NT>(amax, S.red_tmp);  // barrier: xs and hist1 complete

  const float t = (A.scale_mode == OASIS_SCALE_NONE) ? 1.0f : h2f((uint16_t)amax);
  if (CLUSTER && tid == 0) A.act_scale[i] = t;

  // ---- scaled cluster boundaries P_c = fp32(t * b_c), b_c = (c_c + c_{c+1}) * 0.5
  const int nb = (1 << A.b_a) - 1;
  float P[15];
#pragma unroll
  for (int c = 0; c < 15; ++c) {
    const float bc = (S.ca[c] + S.ca[c + 1]) * 0.5f;
    P[c] = t * bc;
  }
  auto cluster = [&](float x) -> uint32_t {
    uint32_t a = 0;
#pragma unroll
    for (int c = 0; c < 15; ++c) a += (c < nb && x >= P[c]) ? 1u : 0u;
    return a;
  };

  // ---- cluster index of every channel, packed 8 per word.  The index is
  // monotone in the order-preserving key, so the keys sharing a high byte span
  // a range [first, last] of indices; only the few buckets a boundary crosses
  // need compares: a = first + #{first <= c < last : x >= P_c}.  The table is
  // visible after the next barrier.
  if (CLUSTER) {
    if (tid < 16) S.P[tid] = tid < nb ? P[tid < 15 ? tid : 14] : 0.0f;
    if (tid < 256) {
      auto bits_of = [](uint32_t key) -> uint16_t {  // inverse of ord_key
        return (uint16_t)((key & 0x8000u) ? (key & 0x7FFFu) : (~key & 0xFFFFu));
      };
      const uint32_t lo = cluster(h2f(bits_of((uint32_t)tid << 8)));
      const uint32_t hi = cluster(h2f(bits_of(((uint32_t)tid << 8) | 0xFFu)));
      S.bucket[tid] = (uint16_t)(lo | (hi << 8));
    }
  }
  auto code8 = [&](const uint4& q) -> uint32_t {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    uint32_t packed = 0;
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const uint32_t bits = (w[h >> 1] >> (16 * (h & 1))) & 0xFFFFu;
      const uint32_t e = S.bucket[ord_key(bits) >> 8];
      uint32_t a = e & 0xFFu;
      const uint32_t last = e >> 8;
      if (a < last) {  // a boundary lies inside this bucket
        const float x = h2f((uint16_t)bits);
        uint32_t add = 0;
        for (uint32_t c = a; c < last; ++c) add += x >= S.P[c] ? 1u : 0u;
        a += add;
      }
      packed |= a << (4 * h);
    }
    return packed;
  };
  uint32_t* arow = reinterpret_cast<uint32_t*>(A.idx_act + (size_t)i * (d_in / 2));
  if (!topk) {
    if (CLUSTER) {
      __syncthreads();
      for (int v = tid; v < nvec; v += NT) arow[v] = code8(xs4[v]);  // coalesced
    }
    return;
  }

  // contiguous run of channels owned by this thread, in 8-channel vectors
  const int vpt = (nvec + NT - 1) / NT;
  const int v0 = min(nvec, tid * vpt), v1 = min(nvec, v0 + vpt);

  // ---- pass 1 (histogram built while staging): the high-byte buckets that
  // hold the k-th largest and the k-th smallest key
  {
    const uint32_t h = tid < 256 ? S.hist1[tid] : 0u;
    const uint32_t pre = (uint32_t)block_scan64<NT>(h, S.scan_tmp[0]);  // keys with byte <= tid
    if (tid < 256) {
      const uint32_t suf_excl = (uint32_t)d_in - pre;  // keys with high byte > tid
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
  }
  __syncthreads();
  const uint32_t B1max = S.ctl[0], G1max = S.ctl[1], B1min = S.ctl[2], G1min = S.ctl[3];

  // ---- pass 2: low byte inside the two boundary buckets
  for (int v = v0; v < v1; ++v) {
    const uint4 q = xs4[v];
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const uint32_t key = ord_key((w[h >> 1] >> (16 * (h & 1))) & 0xFFFFu);
      if ((key >> 8) == B1max) atomicAdd(&S.hist2_max[key & 255u], 1u);
      if ((key >> 8) == B1min) atomicAdd(&S.hist2_min[key & 255u], 1u);
    }
  }
  __syncthreads();
  {
    const uint32_t hm = tid < 256 ? S.hist2_max[tid] : 0u;
    const uint32_t hn = tid < 256 ? S.hist2_min[tid] : 0u;
    const uint64_t pre = block_scan64<NT>(((uint64_t)hn << 32) | hm, S.scan_tmp[1]);
    const uint32_t pre_m = (uint32_t)pre, pre_n = (uint32_t)(pre >> 32);
    if (tid < 256) {
      const uint32_t kk = (uint32_t)k - G1max;
      // keys of the max list's boundary bucket with a low byte above tid
      const uint32_t suf_excl = S.hist1[B1max] - pre_m;
      if (suf_excl < kk && kk <= suf_excl + hm) {
        S.ctl[4] = (B1max << 8) | tid;  // threshold key of the max list
        S.ctl[5] = G1max + suf_excl;    // keys strictly greater
      }
      const uint32_t kn = (uint32_t)k - G1min;
      const uint32_t pre_excl = pre_n - hn;
      if (pre_excl < kn && kn <= pre_n) {
        S.ctl[6] = (B1min << 8) | tid;  // threshold key of the min list
        S.ctl[7] = G1min + pre_excl;    // keys strictly smaller
      }
    }
  }
  __syncthreads();
  // G < k holds by construction; the clamp only keeps every index in bounds.
  const uint32_t Tmax = S.ctl[4], Tmin = S.ctl[6];
  const uint32_t Gmax = min(S.ctl[5], (uint32_t)k - 1u);
  const uint32_t Gmin = min(S.ctl[7], (uint32_t)k - 1u);
  const uint32_t need_max = (uint32_t)k - Gmax, need_min = (uint32_t)k - Gmin;

  // ---- per-thread counts, in channel order, of (max-list ties, min-list ties,
  // keys above Tmax, keys below Tmin), 16 bits each: one 64-bit block scan
  // gives every thread its tie ranks and its candidate slots.  (Exclusive
  // prefixes stay below 2^16 because d_in <= 65536.)  The same pass writes the
  // cluster codes of the thread's run.
  uint64_t cnt = 0;
  for (int v = v0; v < v1; ++v) {
    const uint4 q = xs4[v];
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const uint32_t key = ord_key((w[h >> 1] >> (16 * (h & 1))) & 0xFFFFu);
      cnt += (uint64_t)(key == Tmax) | ((uint64_t)(key == Tmin) << 16) |
             ((uint64_t)(key > Tmax) << 32) | ((uint64_t)(key < Tmin) << 48);
    }
    if (fused_cluster) arow[v] = code8(q);
  }
  const uint64_t excl = block_scan64<NT>(cnt, S.scan_tmp[2]) - cnt;
  uint32_t rank_max = (uint32_t)(excl & 0xFFFFu), rank_min = (uint32_t)((excl >> 16) & 0xFFFFu);
  uint32_t slot_max = (uint32_t)((excl >> 32) & 0xFFFFu), slot_min = (uint32_t)(excl >> 48);

  const size_t krow = (size_t)i * k;
  const size_t rrow = (size_t)i * 2 * k;
  auto residual_of = [&](float x) -> float {
    const float xhat = t * S.ca[cluster(x)];  // exact: a product of two fp16 values
    return x - xhat;
  };

  // ---- collect: direct output for threshold ties, candidate slots for the rest
  for (int v = v0; v < v1; ++v) {
    const uint4 q = xs4[v];
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const uint32_t bits = (w[h >> 1] >> (16 * (h & 1))) & 0xFFFFu;
      const uint32_t key = ord_key(bits);
      const int p = 8 * v + h;
      bool in_max = key > Tmax;
      if (key == Tmax) {
        in_max = rank_max < need_max;
        if (in_max) {
          const uint32_t pos = Gmax + rank_max;
          A.max_idx[krow + pos] = p;
          A.residual[rrow + pos] = residual_of(h2f((uint16_t)bits));
        }
        ++rank_max;
      } else if (in_max) {
        if (slot_max < Gmax) cand_max[slot_max] = (key << 16) | (0xFFFFu - (uint32_t)p);
        ++slot_max;
      }
      if (key == Tmin) {
        if (rank_min < need_min) {
          const uint32_t pos = Gmin + rank_min;
          A.min_idx[krow + pos] = p;
          A.residual[rrow + k + pos] = in_max ? 0.0f : residual_of(h2f((uint16_t)bits));
        }
        ++rank_min;
      } else if (key < Tmin) {
        if (slot_min < Gmin) {
          cand_min[slot_min] = (key << 16) | (uint32_t)p;
          cand_dup[slot_min] = in_max ? 1u : 0u;
        }
        ++slot_min;
      }
    }
  }
  __syncthreads();

  // ---- rank the candidates: one lane per candidate, counting the
  // candidates that pop before it (broadcast LDS reads, no serial chain)
  for (uint32_t c = tid; c < Gmax + Gmin; c += NT) {
    if (c < Gmax) {
      const uint32_t key = cand_max[c];
      uint32_t rank = 0;
#pragma unroll 4
      for (uint32_t q = 0; q < Gmax; ++q) rank += cand_max[q] > key ? 1u : 0u;
      const int p = (int)(0xFFFFu - (key & 0xFFFFu));
      A.max_idx[krow + rank] = p;
      A.residual[rrow + rank] = residual_of(h2f(xs[p]));
    } else {
      const uint32_t cm = c - Gmax;
      const uint32_t key = cand_min[cm];
      uint32_t rank = 0;
#pragma unroll 4
      for (uint32_t q = 0; q < Gmin; ++q) rank += cand_min[q] < key ? 1u : 0u;
      const int p = (int)(key & 0xFFFFu);
      A.min_idx[krow + rank] = p;
      A.residual[rrow + k + rank] = cand_dup[cm] ? 0.0f : residual_of(h2f(xs[p]));
    }
  }
}

template <int NT, bool CL, bool TK>
static hipError_t launch_nt(const QuantArgs& a, hipStream_t s) {
  const size_t lds = sizeof(QuantSmem<NT>) + dyn_bytes(a.d_in, TK ? a.k : 0);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k_quantize<NT, CL, TK>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_quantize<NT, CL, TK>), dim3(a.n), dim3(NT), lds, s, a);
  return hipGetLastError();
}

template <bool CL, bool TK>
static hipError_t launch_parts(const QuantArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  // few tokens: wide workgroups keep each token's serial phases short
  return a.n <= 64 ? launch_nt<512, CL, TK>(a, s) : launch_nt<256, CL, TK>(a, s);
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t s) { return launch_parts<true, true>(a, s); }
hipError_t launch_cluster(const QuantArgs& a, hipStream_t s) { return launch_parts<true, false>(a, s); }
hipError_t launch_outliers(const QuantArgs& a, hipStream_t s) {
  if (a.k == 0) return hipSuccess;
  return launch_parts<false, true>(a, s);
}

}  // namespace oasis
