// Per-token activation quantization with dynamic top-k outlier detection.
//
// One workgroup per token computes
//   * the per-token scale t = absmax (Sec. III-A),
//   * the cluster index of every channel by the mid-point boundary rule of the
//     Clustering Unit (Sec. IV-C): a = #{c : x >= fp32(t * b_c)},
//   * the k largest and k smallest channels (the job of the Orizuru engine,
//     Sec. IV-D) with ties to the lower channel, in pop order,
//   * the residual of every listed outlier (Sec. III-C2).
//
// Every fp16 value x becomes an order-preserving 16-bit key (-0 folded into
// +0).  Each thread holds VR runs of 8 consecutive channels in registers, so
// thread order is channel order; the raw token is also staged in LDS for the
// few channels the lists take.
//
// Clustering in key space: an fp16 x satisfies x >= P (P fp32) exactly when
// x >= Q, Q the smallest fp16 (or +-inf) not below P, i.e. when
// key(x) >= key(Q).  The 15 boundary keys are derived from the fp32 boundaries
// once per token, so the index is the number of boundary keys <= key(x): a
// 256-entry table over the key's high byte gives the count at the start of
// that bucket and the low byte of the first boundary inside it.  Unless two
// centroids are very close, at most one boundary falls inside a bucket; keys
// in a bucket with more take the full 15-compare count.  This is the fp32 rule
// of the oracle, bit for bit, at one LDS lookup per channel.
//
// Top-k is a radix select on the keys shared by the max and min lists: a
// histogram of the high byte fixes the bucket holding the k-th largest
// (smallest) key and the count G of keys in the buckets beyond it.  When the
// boundary bucket is small (G plus its size fits the list area) and the two
// candidate sets are disjoint, a list takes every key of the boundary bucket
// and beyond, and ranking them by (key, channel) - distinct per channel -
// keeps the first k.  Otherwise a histogram of the low byte inside the bucket
// gives the exact threshold key T, the count G < k of keys beyond it and the
// count N of keys equal to it; a list takes every key beyond T and, when N
// fits the k - G places left, every key equal to T, else the first k - G of
// those in channel order (a block-wide exclusive count ranks them).  The
// paper's trees pop in exactly this order; the select replaces k sequential
// pops by histogram passes.  Every wave scans the histograms itself (DPP
// prefix sums), so a level costs one barrier.
#include "common.h"

namespace oasis {

struct __align__(16) QuantSmem {
  uint32_t hist1[256];     // high byte of the key
  uint32_t hist2[2][256];  // low byte inside the max / min boundary bucket
  uint16_t bucket[256];    // first index | inside count << 4 | low byte << 8
  float ca[16];            // C_A in fp32
  uint32_t wmax[16];       // per-wave absmax
  uint32_t wtot[16];       // per-wave tie counts (max | min << 16), cut case only
  uint32_t nalloc;         // list slots handed out (max | min << 16)
};

// Entries a list area holds: k rounded up to 4, plus room for the keys of a
// boundary bucket beyond the k-th (a multiple of 4).
__host__ __device__ inline uint32_t list_cap(int k) {
  const uint32_t k4 = ((uint32_t)k + 3u) & ~3u;
  return k4 + (k4 / 2u > 32u ? ((k4 / 2u) & ~3u) : 32u);
}

// Dynamic LDS after the fixed part: the token (2 B per channel), then the two
// list areas, each list_cap(k) sort keys and as many cluster indices (max
// list, then min list).
static size_t dyn_bytes(int d_in, int k) { return (size_t)d_in * 2 + 16 * (size_t)list_cap(k); }

// Inlier scale computed in the same launch (top-k lists, no fixed
// thresholds): after the lists, a bitmap of the listed channels (d_in bits,
// whole 16-byte rows) and the 2k list entries (channel | 1 << 31 for a min
// entry whose channel is on the max list too).
__host__ __device__ inline uint32_t inlier_words(int d_in) {
  return (((uint32_t)d_in + 31u) / 32u + 3u) & ~3u;
}
static size_t inlier_bytes(int d_in, int k) { return 4 * (size_t)inlier_words(d_in) + 8 * (size_t)k; }

size_t quantize_lds_bytes(int d_in, int k, bool inlier) {
  return sizeof(QuantSmem) + dyn_bytes(d_in, k) + (inlier ? inlier_bytes(d_in, k) : 0);
}

// fp16 bits -> order-preserving key; -0 and +0 share key 0x8000.
__device__ __forceinline__ uint32_t ord_key(uint32_t bits) {
  if (bits == 0x8000u) bits = 0;
  return (bits & 0x8000u) ? (bits ^ 0xFFFFu) : (bits | 0x8000u);
}

template <int NT, int VR, bool CLUSTER, bool TOPK>
__global__ void __launch_bounds__(NT) k_quantize(QuantArgs A) {
#pragma clang fp contract(off)
  constexpr int NW = NT / 64;
  static_assert(NT >= 256 && NW <= 16, "256..1024 threads");
  static_assert(VR >= 1 && 8 * VR <= 64, "at most 64 channels per thread");
  extern __shared__ __align__(16) unsigned char smem_raw[];
  QuantSmem& S = *reinterpret_cast<QuantSmem*>(smem_raw);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i = blockIdx.x;
  const int d_in = A.d_in, k = A.k, nvec = d_in >> 3;
  const bool topk = TOPK && k > 0;  // uniform
  const uint32_t lcap = topk ? list_cap(k) : 0u;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem_raw + sizeof(QuantSmem));
  uint32_t* cmax = reinterpret_cast<uint32_t*>(xs + d_in);  // d_in % 8 == 0: 16-byte aligned
  uint32_t* amax_ = cmax + lcap;
  uint32_t* cmin = amax_ + lcap;
  uint32_t* amin_ = cmin + lcap;
  // inlier scale in this launch (uniform): see inlier_bytes
  const bool inl = topk && A.scale_mode == OASIS_SCALE_INLIER && !A.static_thr;
  uint32_t* lbits = amin_ + lcap;
  uint32_t* lent = lbits + inlier_words(d_in);

  // ---- the token into registers (runs tid*VR .. tid*VR + VR - 1)
  uint4 xv[VR];
  const uint4* xrow = reinterpret_cast<const uint4*>(A.x + (size_t)i * d_in);
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int v = tid * VR + u;
    xv[u] = v < nvec ? xrow[v] : make_uint4(0u, 0u, 0u, 0u);
  }
  if (tid < 256) {
    S.hist1[tid] = 0;
    S.hist2[0][tid] = 0;
    S.hist2[1][tid] = 0;
  }
  // C_A[lane] and C_A[lane + 1] (the boundary mid-points need both) from the
  // codebook arguments when the LUT is built in this launch, else from the
  // LUT block; requested now, used after the keys are made
  const bool build = A.lut_out != nullptr;  // uniform
  uint32_t cal = 0, cah = 0;
  if (lane < 16) cal = build ? A.cb.act[lane] : A.lut->cb_act[lane];
  if (lane < 15) cah = build ? A.cb.act[lane + 1] : A.lut->cb_act[lane + 1];
  // workgroup 0 of a building launch: the codebook entries of LUT entry tid
  const bool lut_writer = build && i == 0 && tid < 256;
  const int lut_e = tid, lut_a = tid >> A.b_w, lut_w = tid & ((1 << A.b_w) - 1);
  uint32_t lua = 0, luw = 0, lcw = 0;
  if (lut_writer && lut_e < (1 << (A.b_a + A.b_w))) {
    lua = A.cb.act[lut_a];
    luw = A.cb.wgt[lut_w];
  }
  if (lut_writer && tid < 16) lcw = A.cb.wgt[tid];
  if (tid < 256) {
    S.hist1[tid] = 0;
    S.hist2[0][tid] = 0;
    S.hist2[1][tid] = 0;
  }
  if (tid == 0) S.nalloc = 0;
  if (inl)
    for (uint32_t w = (uint32_t)tid; w < inlier_words(d_in); w += NT) lbits[w] = 0u;
  __syncthreads();  // histograms cleared

  // keys, two per word (even channel low)
  uint32_t key[VR][4];
  uint32_t amax = 0;
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const bool live = tid * VR + u < nvec;
    const uint32_t w[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = w[q] & 0xFFFFu, hi = w[q] >> 16;
      key[u][q] = ord_key(lo) | (ord_key(hi) << 16);
      amax = max(amax, max(lo & 0x7FFFu, hi & 0x7FFFu));
    }
    if (topk && live) {
      reinterpret_cast<uint4*>(xs)[tid * VR + u] = xv[u];
      if (!A.static_thr) {  // uniform: fixed thresholds need no histogram
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          atomicAdd(&S.hist1[(key[u][q] >> 8) & 0xFFu], 1u);
          atomicAdd(&S.hist1[key[u][q] >> 24], 1u);
        }
      }
    }
  }
  // boundary mid-points b_c = fp32(C_A[c] + C_A[c+1]) * 0.5 in lane c (they
  // do not depend on the token)
  const int nb = (1 << A.b_a) - 1;
  const float bc = lane < nb ? (h2f((uint16_t)cal) + h2f((uint16_t)cah)) * 0.5f : 0.0f;
  if (tid < 16) S.ca[tid] = h2f((uint16_t)cal);  // read after later barriers
  if (lut_writer) {
    // the LUT block (the contents oasis_build_lut writes); a product of two
    // fp16 values is exact in fp32
    A.lut_out->lut[lut_e] = lut_e < (1 << (A.b_a + A.b_w)) ? h2f((uint16_t)lua) * h2f((uint16_t)luw)
                                                          : 0.0f;
    if (tid < 16) {  // entries past 2^b are 0 in the arguments
      A.lut_out->cb_act[tid] = (uint16_t)cal;
      A.lut_out->cb_wgt[tid] = (uint16_t)lcw;
    }
  }
  amax = wave_max(amax);
  if (lane == 0) S.wmax[wave] = amax;
  __syncthreads();  // absmax partials, level-1 histogram

#pragma unroll
  for (int j = 0; j < NW / 4; ++j) {
    const uint4 m = reinterpret_cast<const uint4*>(S.wmax)[j];
    amax = max(amax, max(max(m.x, m.y), max(m.z, m.w)));
  }
  const float t = (A.scale_mode == OASIS_SCALE_NONE) ? 1.0f : h2f((uint16_t)amax);
  if (CLUSTER && !inl && tid == 0) A.act_scale[i] = t;

  // ---- boundary keys: lane c computes key(Q_c), Q_c = the smallest fp16 not
  // below P_c = fp32(ts * b_c)
  uint32_t kq_lane = 0x10000u;  // above every key: boundaries past the last one
  uint32_t KQ[15];
  auto boundaries = [&](float ts) {
    kq_lane = 0x10000u;
    if (lane < nb) {
      const float P = ts * bc;
      const _Float16 h = (_Float16)P;  // round to nearest even
      kq_lane = ord_key(__builtin_bit_cast(uint16_t, h)) + ((float)h < P ? 1u : 0u);
    }
#pragma unroll
    for (int c = 0; c < 15; ++c) KQ[c] = (uint32_t)__builtin_amdgcn_readlane((int)kq_lane, c);
  };
  boundaries(t);
  // cluster index by the full count
  auto code_full = [&](uint32_t kk) -> uint32_t {
    uint32_t a = 0;
#pragma unroll
    for (int c = 0; c < 15; ++c) a += kk >= KQ[c] ? 1u : 0u;
    return a;
  };
  auto build_bucket = [&]() {
    if (tid < 256) {  // bucket tid: keys tid*256 .. tid*256 + 255
      const uint32_t base = (uint32_t)tid << 8;
      uint32_t first = 0, upto = 0;
#pragma unroll
      for (int c = 0; c < 15; ++c) {
        first += KQ[c] <= base ? 1u : 0u;
        upto += KQ[c] <= base + 255u ? 1u : 0u;
      }
      // KQ[first], the first boundary inside if any, from lane `first` of this wave
      const uint32_t kf = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(first << 2), (int)kq_lane);
      S.bucket[tid] = (uint16_t)(first | ((upto - first) << 4) | ((kf & 0xFFu) << 8));
    }
  };
  build_bucket();
  // cluster index of one key from the table (visible after the next barrier);
  // `multi` flags a bucket with two or more boundaries (then use code_full)
  auto code_fast = [&](uint32_t kk, bool& multi) -> uint32_t {
    const uint32_t e = S.bucket[kk >> 8];
    const uint32_t nin = (e >> 4) & 15u;
    multi |= nin > 1u;
    return (e & 15u) + ((nin != 0u && (kk & 0xFFu) >= (e >> 8)) ? 1u : 0u);
  };
  // packed cluster indices of the thread's runs (8 per word, channel 8v + h in
  // bits 4h..4h+3); 0 for runs past d_in
  uint32_t codes[VR];
  auto make_codes = [&]() {
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      bool multi = false;
      uint32_t packed = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        packed |= code_fast(key[u][q] & 0xFFFFu, multi) << (8 * q);
        packed |= code_fast(key[u][q] >> 16, multi) << (8 * q + 4);
      }
      if (multi) {
        packed = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          packed |= (code_full(key[u][q] & 0xFFFFu) << (8 * q)) |
                    (code_full(key[u][q] >> 16) << (8 * q + 4));
      }
      codes[u] = tid * VR + u < nvec ? packed : 0u;
    }
  };
  uint32_t* arow = reinterpret_cast<uint32_t*>(A.idx_act + (size_t)i * (d_in / 2));
  auto store_codes = [&]() {
#pragma unroll
    for (int u = 0; u < VR; ++u)
      if (tid * VR + u < nvec) arow[tid * VR + u] = codes[u];
  };
  if (!topk) {
    if (CLUSTER) {
      __syncthreads();  // bucket table
      make_codes();
      store_codes();
    }
    return;
  }
  const size_t krow = (size_t)i * k;
  const size_t rrow = (size_t)i * 2 * k;
  // one bit per channel of the thread: 32-bit masks while they suffice
  using mask_t = typename std::conditional<(8 * VR <= 32), uint32_t, uint64_t>::type;

  if (A.static_thr) {  // uniform
    // ---- OASIS-S: the outliers are the channels at or beyond two fixed
    // thresholds, listed in channel order, at most k per side; the places
    // left are padded with channel -1 and residual 0.  x >= thr_hi exactly
    // when key(x) >= key(Q), Q the smallest fp16 (or +inf) not below thr_hi;
    // x <= thr_lo when key(x) <= key(Q'), Q' the largest fp16 not above it.
    const _Float16 fh = (_Float16)A.thr_hi, fl = (_Float16)A.thr_lo;  // nearest even
    const uint32_t KH = ord_key(__builtin_bit_cast(uint16_t, fh)) + ((float)fh < A.thr_hi ? 1u : 0u);
    const uint32_t KL = ord_key(__builtin_bit_cast(uint16_t, fl)) - ((float)fl > A.thr_lo ? 1u : 0u);
    __syncthreads();  // bucket table
    make_codes();
    if (CLUSTER) store_codes();
    mask_t mmax = 0, mmin = 0;
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (tid * VR + u < nvec) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t kk = (key[u][q] >> (16 * hh)) & 0xFFFFu;
            mmax |= (mask_t)(kk >= KH ? 1u : 0u) << (8 * u + 2 * q + hh);
            mmin |= (mask_t)(kk <= KL ? 1u : 0u) << (8 * u + 2 * q + hh);
          }
        }
      }
    }
    // channel-order ranks: block exclusive scans of the per-thread counts
    // (two scans: a side may hold all 65536 channels)
    const uint32_t cmx = (uint32_t)__builtin_popcountll((uint64_t)mmax);
    const uint32_t cmn = (uint32_t)__builtin_popcountll((uint64_t)mmin);
    const uint32_t imx = wave_incl_scan(cmx), imn = wave_incl_scan(cmn);
    uint32_t* wtot_min = S.hist2[0];  // the level-2 histograms are unused here
    if (lane == 63) {
      S.wtot[wave] = imx;
      wtot_min[wave] = imn;
    }
    __syncthreads();  // wave totals
    uint32_t smax = imx - cmx, smin = imn - cmn, totmax = 0, totmin = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t a = S.wtot[w], b = wtot_min[w];
      smax += w < wave ? a : 0u;
      smin += w < wave ? b : 0u;
      totmax += a;
      totmin += b;
    }
    mask_t m = mmax | mmin;
    const uint32_t p0 = 8u * (uint32_t)(tid * VR);
    while (m) {
      const int e = __builtin_ctzll((uint64_t)m);
      m &= m - 1;
      uint32_t cw = codes[0];
#pragma unroll
      for (int u = 1; u < VR; ++u) cw = (e >> 3) == u ? codes[u] : cw;
      const uint32_t a = (cw >> (4 * (e & 7))) & 15u;
      const uint32_t p = p0 + (uint32_t)e;
      // t * C_A[a] is exact, a product of two fp16 values
      const float r = h2f(xs[p]) - t * S.ca[a];
      const bool im = ((mmax >> e) & 1u) != 0u, in = ((mmin >> e) & 1u) != 0u;
      const bool listed_max = im && smax < (uint32_t)k;
      if (listed_max) {
        A.max_idx[krow + smax] = (int)p;
        A.residual[rrow + smax] = r;
      }
      if (in && smin < (uint32_t)k) {
        A.min_idx[krow + smin] = (int)p;
        A.residual[rrow + k + smin] = listed_max ? 0.0f : r;  // compensated once
      }
      smax += im ? 1u : 0u;
      smin += in ? 1u : 0u;
    }
    for (int e = tid; e < k; e += NT) {
      if ((uint32_t)e >= totmax) {
        A.max_idx[krow + e] = -1;
        A.residual[rrow + e] = 0.0f;
      }
      if ((uint32_t)e >= totmin) {
        A.min_idx[krow + e] = -1;
        A.residual[rrow + k + e] = 0.0f;
      }
    }
    return;
  }

  // ---- level 1: the high-byte buckets holding the k-th largest and k-th
  // smallest key (each wave scans the histogram itself)
  uint32_t B1max, G1max, B1min, G1min, H1max, H1min;  // H1: keys in the bucket
  {
    const uint4 h = *reinterpret_cast<const uint4*>(&S.hist1[4 * lane]);
    const uint32_t hs[4] = {h.x, h.y, h.z, h.w};
    const uint32_t sum = h.x + h.y + h.z + h.w;
    uint32_t pre = wave_incl_scan(sum) - sum;  // keys in buckets below 4*lane
    uint32_t fmax = 0, gmax = 0, fmin = 0, gmin = 0, hmx = 0, hmn = 0;
    bool hit_max = false, hit_min = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t below = pre, upto = pre + hs[q];
      const uint32_t above = (uint32_t)d_in - upto;  // keys in buckets above
      const bool hm = above < (uint32_t)k && (uint32_t)k <= above + hs[q];
      const bool hn = below < (uint32_t)k && (uint32_t)k <= upto;
      fmax = hm ? (uint32_t)(4 * lane + q) : fmax;
      gmax = hm ? above : gmax;
      fmin = hn ? (uint32_t)(4 * lane + q) : fmin;
      gmin = hn ? below : gmin;
      hmx = hm ? hs[q] : hmx;
      hmn = hn ? hs[q] : hmn;
      hit_max |= hm;
      hit_min |= hn;
      pre = upto;
    }
    // exactly one bucket holds each threshold; the guard keeps lanes < 64
    const int lm = __builtin_ctzll(__ballot(hit_max) | (1ull << 63));
    const int ln = __builtin_ctzll(__ballot(hit_min) | (1ull << 63));
    B1max = __builtin_amdgcn_readlane(fmax, lm);
    G1max = __builtin_amdgcn_readlane(gmax, lm);
    B1min = __builtin_amdgcn_readlane(fmin, ln);
    G1min = __builtin_amdgcn_readlane(gmin, ln);
    H1max = __builtin_amdgcn_readlane(hmx, lm);
    H1min = __builtin_amdgcn_readlane(hmn, ln);
  }
  // One level suffices when both lists fit every key of their boundary bucket
  // and the two candidate sets are disjoint: the lists then take all those
  // keys and the ranking by (key, channel) keeps the first k of each.
  const bool one_level = G1max + H1max <= lcap && G1min + H1min <= lcap && B1max > B1min;
  // ---- level 2: low bytes inside the two boundary buckets
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    if (!one_level && tid * VR + u < nvec) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const uint32_t kk = (key[u][q] >> (16 * hh)) & 0xFFFFu;
          if ((kk >> 8) == B1max) atomicAdd(&S.hist2[0][kk & 0xFFu], 1u);
          if ((kk >> 8) == B1min) atomicAdd(&S.hist2[1][kk & 0xFFu], 1u);
        }
      }
    }
  }
  __syncthreads();  // level-2 histograms, bucket table

  // thresholds: keys >= Tmax enter the max list, keys <= Tmin the min list;
  // L entries each (one level: the whole boundary buckets; two levels: k)
  uint32_t Tmax, Tmin, Lmax, Lmin;
  bool cut = false;
  uint32_t need_max = 0, need_min = 0;
  if (one_level) {
    Tmax = B1max << 8;
    Tmin = (B1min << 8) | 0xFFu;
    Lmax = G1max + H1max;
    Lmin = G1min + H1min;
  } else {
    uint32_t Gmax, Gmin, Nmax, Nmin;  // N: keys equal to the threshold
    {
      const uint4 hm = *reinterpret_cast<const uint4*>(&S.hist2[0][4 * lane]);
      const uint4 hn = *reinterpret_cast<const uint4*>(&S.hist2[1][4 * lane]);
      const uint32_t ms[4] = {hm.x, hm.y, hm.z, hm.w}, ns[4] = {hn.x, hn.y, hn.z, hn.w};
      const uint32_t summ = hm.x + hm.y + hm.z + hm.w, sumn = hn.x + hn.y + hn.z + hn.w;
      uint32_t prem = wave_incl_scan(summ) - summ, pren = wave_incl_scan(sumn) - sumn;
      const uint32_t totm = S.hist1[B1max];
      const uint32_t kk = (uint32_t)k - G1max, kn = (uint32_t)k - G1min;
      uint32_t tm = 0, gm = 0, tn = 0, gn = 0, nm = 0, nn = 0;
      bool hit_max = false, hit_min = false;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t uptom = prem + ms[q];
        const uint32_t above = totm - uptom;  // keys of the bucket with a higher low byte
        const bool hmq = above < kk && kk <= above + ms[q];
        tm = hmq ? ((B1max << 8) | (uint32_t)(4 * lane + q)) : tm;
        gm = hmq ? G1max + above : gm;
        nm = hmq ? ms[q] : nm;
        const uint32_t upton = pren + ns[q];
        const bool hnq = pren < kn && kn <= upton;
        tn = hnq ? ((B1min << 8) | (uint32_t)(4 * lane + q)) : tn;
        gn = hnq ? G1min + pren : gn;
        nn = hnq ? ns[q] : nn;
        hit_max |= hmq;
        hit_min |= hnq;
        prem = uptom;
        pren = upton;
      }
      const int lm = __builtin_ctzll(__ballot(hit_max) | (1ull << 63));
      const int ln = __builtin_ctzll(__ballot(hit_min) | (1ull << 63));
      Tmax = __builtin_amdgcn_readlane(tm, lm);
      Gmax = __builtin_amdgcn_readlane(gm, lm);
      Tmin = __builtin_amdgcn_readlane(tn, ln);
      Gmin = __builtin_amdgcn_readlane(gn, ln);
      Nmax = __builtin_amdgcn_readlane(nm, lm);
      Nmin = __builtin_amdgcn_readlane(nn, ln);
    }
    // G < k holds by construction; the clamp only keeps every index in bounds.
    Gmax = min(Gmax, (uint32_t)k - 1u);
    Gmin = min(Gmin, (uint32_t)k - 1u);
    need_max = (uint32_t)k - Gmax;
    need_min = (uint32_t)k - Gmin;
    // a key equal to a threshold enters its list unless the value occurs more
    // often than the list has room for: then only the first `need` such keys
    // in channel order do, ranked by a block-wide exclusive count
    cut = Nmax > need_max || Nmin > need_min;
    Lmax = Lmin = (uint32_t)k;
  }
  // pad both lists to a multiple of 4 with entries that never rank first
  // (sort keys are compared after XOR with 0 for the max list and with ~0 for
  // the min list, which turns a pad into 0)
  if (tid < 4) {
    if (Lmax + (uint32_t)tid < lcap) cmax[Lmax + tid] = 0u;
    if (Lmin + (uint32_t)tid < lcap) cmin[Lmin + tid] = 0xFFFFFFFFu;
  }

  make_codes();
  if (CLUSTER && !inl) store_codes();

  // ---- list membership, one bit per channel
  mask_t mmax = 0, mmin = 0;
  if (!cut) {
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (tid * VR + u < nvec) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t kk = (key[u][q] >> (16 * hh)) & 0xFFFFu;
            mmax |= (mask_t)(kk >= Tmax ? 1u : 0u) << (8 * u + 2 * q + hh);
            mmin |= (mask_t)(kk <= Tmin ? 1u : 0u) << (8 * u + 2 * q + hh);
          }
        }
      }
    }
  } else {
    uint32_t c_tie = 0;  // (max ties, min ties), 16 bits each: < 65536 channels
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (tid * VR + u < nvec) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t kk = (key[u][q] >> (16 * hh)) & 0xFFFFu;
            c_tie += (kk == Tmax ? 1u : 0u) + (kk == Tmin ? 0x10000u : 0u);
          }
        }
      }
    }
    const uint32_t inc = wave_incl_scan(c_tie);
    if (lane == 63) S.wtot[wave] = inc;
    __syncthreads();  // wave tie totals
    uint32_t ex = inc - c_tie;
    {
      uint32_t wt[NW];
#pragma unroll
      for (int j = 0; j < NW / 4; ++j) {
        const uint4 v = reinterpret_cast<const uint4*>(S.wtot)[j];
        wt[4 * j] = v.x;
        wt[4 * j + 1] = v.y;
        wt[4 * j + 2] = v.z;
        wt[4 * j + 3] = v.w;
      }
#pragma unroll
      for (int w = 0; w < NW; ++w) ex += w < wave ? wt[w] : 0u;
    }
    uint32_t rm = ex & 0xFFFFu, rn = ex >> 16;
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      if (tid * VR + u < nvec) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t kk = (key[u][q] >> (16 * hh)) & 0xFFFFu;
            const bool em = kk == Tmax, en = kk == Tmin;
            const bool im = kk > Tmax || (em && rm < need_max);
            const bool in = kk < Tmin || (en && rn < need_min);
            mmax |= (mask_t)(im ? 1u : 0u) << (8 * u + 2 * q + hh);
            mmin |= (mask_t)(in ? 1u : 0u) << (8 * u + 2 * q + hh);
            rm += em ? 1u : 0u;
            rn += en ? 1u : 0u;
          }
        }
      }
    }
  }

  // ---- each list holds exactly L entries; slots in any order (the ranking
  // sorts them), a block-wide count through one LDS counter
  const uint32_t cnt = (uint32_t)__builtin_popcountll((uint64_t)mmax) |
                       ((uint32_t)__builtin_popcountll((uint64_t)mmin) << 16);
  // wave prefix, then one LDS atomic per wave (lane 63 holds the wave total)
  const uint32_t inc = wave_incl_scan(cnt);
  uint32_t wbase = 0;
  if (lane == 63) wbase = atomicAdd(&S.nalloc, inc);
  const uint32_t slot = (uint32_t)__builtin_amdgcn_readlane((int)wbase, 63) + inc - cnt;
  uint32_t smax = slot & 0xFFFFu, smin = slot >> 16;
  mask_t m = mmax | mmin;
  const uint32_t p0 = 8u * (uint32_t)(tid * VR);
  while (m) {
    const int e = __builtin_ctzll((uint64_t)m);
    m &= m - 1;
    uint32_t w = key[0][0];
#pragma unroll
    for (int j = 1; j < 4 * VR; ++j) w = (e >> 1) == j ? key[j >> 2][j & 3] : w;
    const uint32_t kk = (w >> (16 * (e & 1))) & 0xFFFFu;
    uint32_t cw = codes[0];
#pragma unroll
    for (int u = 1; u < VR; ++u) cw = (e >> 3) == u ? codes[u] : cw;
    const uint32_t a = (cw >> (4 * (e & 7))) & 15u;
    const uint32_t p = p0 + (uint32_t)e;
    const bool im = ((mmax >> e) & 1u) != 0u, in = ((mmin >> e) & 1u) != 0u;
    if (im && smax < Lmax) {
      cmax[smax] = (kk << 16) | (0xFFFFu - p);
      amax_[smax] = a;
    }
    if (in && smin < Lmin) {
      cmin[smin] = (kk << 16) | p;
      amin_[smin] = a | (im ? 16u : 0u);  // 16: the channel is on the max list too
    }
    smax += im ? 1u : 0u;
    smin += in ? 1u : 0u;
  }
  __syncthreads();  // both lists

  // ---- rank: the first half of the waves the max list, the second half the
  // min list.  P lanes share an entry, each counting the entries that pop
  // before it over every P-th quad; a DPP sum combines the P counts.  Sort
  // keys (key, channel) are distinct, so the ranks are the list positions.
  {
    constexpr int HALF = NT / 2;
    const bool is_max = wave < NW / 2;  // uniform
    const uint32_t flip = is_max ? 0u : 0xFFFFFFFFu;
    const uint32_t* cand = is_max ? cmax : cmin;
    const uint32_t* aux = is_max ? amax_ : amin_;
    const uint4* c4 = reinterpret_cast<const uint4*>(cand);
    const uint32_t L = is_max ? Lmax : Lmin;
    const uint32_t nq = (L + 3u) / 4u;
    uint32_t P = 1;  // uniform
    while (P < 8u && P < nq && 2u * P * L <= (uint32_t)HALF) P *= 2u;
    const uint32_t lt = (uint32_t)tid & (uint32_t)(HALF - 1), part = lt & (P - 1u);
    for (uint32_t c = lt / P; c < L; c += (uint32_t)HALF / P) {
      const uint32_t mine = cand[c] ^ flip;
      const uint32_t ax = aux[c];
      const uint32_t p = is_max ? 0xFFFFu - (mine & 0xFFFFu) : (~mine & 0xFFFFu);
      // two independent LDS reads: the raw value and its centroid; t * C_A[a]
      // is exact, a product of two fp16 values
      const uint32_t bits = xs[p];
      const float xhat = t * S.ca[ax & 15u];
      uint32_t rank = 0;
      for (uint32_t qq = part; qq < nq; qq += P) {
        const uint4 o = c4[qq];  // the same 16 bytes in every lane of the group
        rank += ((o.x ^ flip) > mine ? 1u : 0u) + ((o.y ^ flip) > mine ? 1u : 0u) +
                ((o.z ^ flip) > mine ? 1u : 0u) + ((o.w ^ flip) > mine ? 1u : 0u);
      }
      rank = group_sum(rank, P);
      if (part == 0u && rank < (uint32_t)k) {
        const float r = (ax & 16u) ? 0.0f : h2f((uint16_t)bits) - xhat;
        if (is_max) {
          A.max_idx[krow + rank] = (int)p;
          if (!inl) A.residual[rrow + rank] = r;
        } else {
          A.min_idx[krow + rank] = (int)p;
          if (!inl) A.residual[rrow + k + rank] = r;
        }
        if (inl) {  // the residual waits for the inlier scale
          lent[(is_max ? 0u : (uint32_t)k) + rank] = p | ((ax & 16u) ? 0x80000000u : 0u);
          atomicOr(&lbits[p >> 5], 1u << (p & 31u));
        }
      }
    }
  }
  if (!inl) return;

  // ---- inlier scale: t = max |x| over the channels in neither list (0 when
  // every channel is listed), then the codes under t and the residuals of
  // the listed channels (by the same boundary rule)
  __syncthreads();  // lists, bitmap
  uint32_t mi = 0;
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int v = tid * VR + u;
    if (v >= nvec) continue;
    const uint32_t lst = (lbits[v >> 2] >> (8 * (v & 3))) & 0xFFu;  // channels 8v .. 8v + 7
    const uint4 xw = reinterpret_cast<const uint4*>(xs)[v];
    const uint32_t w[4] = {xw.x, xw.y, xw.z, xw.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {  // |x| of finite fp16 values orders like its 15 low bits
      if (!((lst >> (2 * q)) & 1u)) mi = max(mi, w[q] & 0x7FFFu);
      if (!((lst >> (2 * q + 1)) & 1u)) mi = max(mi, (w[q] >> 16) & 0x7FFFu);
    }
  }
  mi = wave_max(mi);
  if (lane == 0) S.wmax[wave] = mi;
  __syncthreads();  // inlier maxima
#pragma unroll
  for (int j = 0; j < NW / 4; ++j) {
    const uint4 mm = reinterpret_cast<const uint4*>(S.wmax)[j];
    mi = max(mi, max(max(mm.x, mm.y), max(mm.z, mm.w)));
  }
  const float ti = h2f((uint16_t)mi);
  if (CLUSTER && tid == 0) A.act_scale[i] = ti;
  boundaries(ti);
  build_bucket();
  __syncthreads();  // bucket table
  if (CLUSTER) {
#pragma unroll
    for (int u = 0; u < VR; ++u) {
      const int v = tid * VR + u;
      if (v >= nvec) continue;
      const uint4 xw = reinterpret_cast<const uint4*>(xs)[v];
      const uint32_t w[4] = {xw.x, xw.y, xw.z, xw.w};
      bool multi = false;
      uint32_t packed = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        packed |= code_fast(ord_key(w[q] & 0xFFFFu), multi) << (8 * q);
        packed |= code_fast(ord_key(w[q] >> 16), multi) << (8 * q + 4);
      }
      if (multi) {
        packed = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          packed |= (code_full(ord_key(w[q] & 0xFFFFu)) << (8 * q)) |
                    (code_full(ord_key(w[q] >> 16)) << (8 * q + 4));
      }
      arow[v] = packed;
    }
  }
  // t * C_A[a] is exact, a product of two fp16 values
  for (int e = tid; e < 2 * k; e += NT) {
    const uint32_t ent = lent[e], p = ent & 0x7FFFFFFFu;
    const uint32_t bits = xs[p];
    const float r = (ent >> 31) ? 0.0f : h2f((uint16_t)bits) - ti * S.ca[code_full(ord_key(bits))];
    A.residual[rrow + e] = r;
  }
}

template <int NT, int VR, bool CL, bool TK>
static hipError_t launch_nt(const QuantArgs& a, hipStream_t s) {
  const bool inl = TK && a.k > 0 && a.scale_mode == OASIS_SCALE_INLIER && !a.static_thr;
  const size_t lds = sizeof(QuantSmem) + (TK ? dyn_bytes(a.d_in, a.k) : 0) +
                     (inl ? inlier_bytes(a.d_in, a.k) : 0);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k_quantize<NT, VR, CL, TK>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_quantize<NT, VR, CL, TK>), dim3(a.n), dim3(NT), lds, s, a);
  return hipGetLastError();
}

// Runs of 8 channels per thread (VR) for NT threads.
template <int NT, bool CL, bool TK>
static hipError_t launch_vr(const QuantArgs& a, int nvec, hipStream_t s) {
  if (nvec <= NT) return launch_nt<NT, 1, CL, TK>(a, s);
  if (nvec <= 2 * NT) return launch_nt<NT, 2, CL, TK>(a, s);
  if (nvec <= 4 * NT) return launch_nt<NT, 4, CL, TK>(a, s);
  return launch_nt<NT, 8, CL, TK>(a, s);
}

template <bool CL, bool TK>
static hipError_t launch_parts(const QuantArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  const int nvec = a.d_in / 8;
  // few tokens: short runs per thread (latency); many: 256 threads per token
  // while runs of 4 vectors suffice (register pressure), then wider
  if (a.n <= 64) {
    if (nvec <= 512) return launch_vr<512, CL, TK>(a, nvec, s);
    return launch_vr<1024, CL, TK>(a, nvec, s);
  }
  if (nvec <= 4 * 256) return launch_vr<256, CL, TK>(a, nvec, s);
  if (nvec <= 4 * 512) return launch_vr<512, CL, TK>(a, nvec, s);
  return launch_vr<1024, CL, TK>(a, nvec, s);
}

// ----------------------------------------------------------------------------
// Inlier scale, a second pass once the lists exist: per token (one workgroup
// of 256 threads), t = max |x| over the channels in neither list (0 when all
// are listed), the cluster index of every channel under that t by the same
// boundary rule, and the residuals of the listed channels.  The token (VR
// vectors of 8 channels per thread), its list entries and C_A are requested
// together at the start; the token is also staged in LDS for the residuals.
// LDS: the token (2 B per channel), then two bitmaps of d_in bits (listed;
// in the max list).
// ----------------------------------------------------------------------------
struct InlierBounds {
  float p[15];  // P_c, +inf past the last boundary
};

struct InlierCb {
  float c[16];  // C_A in fp32
};

__device__ __forceinline__ float inlier_centroid(const InlierCb cb, uint32_t a) {
  float v = cb.c[0];
#pragma unroll
  for (int q = 1; q < 16; ++q) v = a == (uint32_t)q ? cb.c[q] : v;
  return v;
}

__device__ __forceinline__ uint32_t inlier_code(const InlierBounds b, float xf) {
  uint32_t a = 0;
#pragma unroll
  for (int c = 0; c < 15; ++c) a += xf >= b.p[c] ? 1u : 0u;
  return a;
}

template <int VR>
__global__ void __launch_bounds__(256) k_inlier_codes(QuantArgs A) {
#pragma clang fp contract(off)
  extern __shared__ __align__(16) unsigned char ismem[];
  __shared__ uint32_t wmax[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = blockIdx.x;
  const int d_in = A.d_in, k = A.k, nw = (d_in + 31) / 32, nvec = d_in / 8;
  uint16_t* xs = reinterpret_cast<uint16_t*>(ismem);
  uint32_t* listed = reinterpret_cast<uint32_t*>(ismem + 2 * (size_t)d_in);
  uint32_t* inmax = listed + nw;
  // ---- requests: the token, the list entries, C_A
  const uint4* xrow = reinterpret_cast<const uint4*>(A.x + (size_t)i * d_in);
  uint4 xv[VR];
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int v = tid + 256 * u;
    xv[u] = v < nvec ? xrow[v] : make_uint4(0u, 0u, 0u, 0u);
  }
  const int32_t* mx = A.max_idx + (size_t)i * k;
  const int32_t* mn = A.min_idx + (size_t)i * k;
  constexpr int EPT = 4;  // list entries per thread per pass
  int pe[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int e = tid + 256 * u;
    pe[u] = e < 2 * k ? (e < k ? mx[e] : mn[e - k]) : -1;
  }
  InlierCb ca;
#pragma unroll
  for (int c = 0; c < 16; ++c) ca.c[c] = h2f(A.lut->cb_act[c]);
  for (int w = tid; w < 2 * nw; w += 256) listed[w] = 0u;
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int v = tid + 256 * u;
    if (v < nvec) reinterpret_cast<uint4*>(xs)[v] = xv[u];
  }
  __syncthreads();
  for (int e = tid, u = 0; e < 2 * k; e += 256, ++u) {
    const int p = u < EPT ? pe[u < EPT ? u : 0] : (e < k ? mx[e] : mn[e - k]);
    if (p >= 0 && p < d_in) {
      atomicOr(&listed[p >> 5], 1u << (p & 31));
      if (e < k) atomicOr(&inmax[p >> 5], 1u << (p & 31));
    }
  }
  __syncthreads();
  // ---- t: |x| of finite fp16 values orders like its 15 low bits
  uint32_t m = 0;
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int v = tid + 256 * u;
    if (v >= nvec) continue;
    const uint32_t lst = (listed[v >> 2] >> (8 * (v & 3))) & 0xFFu;  // channels 8v .. 8v + 7
    const uint32_t w[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (!((lst >> (2 * c)) & 1u)) m = max(m, w[c] & 0x7FFFu);
      if (!((lst >> (2 * c + 1)) & 1u)) m = max(m, (w[c] >> 16) & 0x7FFFu);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o, 64));
  if (lane == 0) wmax[wave] = m;
  __syncthreads();
  m = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
  const float t = h2f((uint16_t)m);
  if (tid == 0) A.act_scale[i] = t;
  // ---- scaled boundaries P_c = fp32(t * b_c), b_c = fp32(C_A[c] + C_A[c+1]) * 0.5
  const int nb = (1 << A.b_a) - 1;
  InlierBounds P;
#pragma unroll
  for (int c = 0; c < 15; ++c)
    P.p[c] = c < nb ? t * ((ca.c[c] + ca.c[c + 1]) * 0.5f) : __builtin_inff();
  uint32_t* arow = reinterpret_cast<uint32_t*>(A.idx_act + (size_t)i * (d_in / 2));
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    const int v = tid + 256 * u;
    if (v >= nvec) continue;
    const uint32_t w[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
    uint32_t packed = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      packed |= inlier_code(P, h2f((uint16_t)(w[c] & 0xFFFFu))) << (8 * c);
      packed |= inlier_code(P, h2f((uint16_t)(w[c] >> 16))) << (8 * c + 4);
    }
    arow[v] = packed;
  }
  // ---- residuals: r = fp32(x - fp32(t * C_A[a])); a min entry also in the max list gets 0
  for (int e = tid, u = 0; e < 2 * k; e += 256, ++u) {
    const int p = u < EPT ? pe[u < EPT ? u : 0] : (e < k ? mx[e] : mn[e - k]);
    if (p < 0 || p >= d_in) continue;  // an unused place keeps its 0
    const float xf = h2f(xs[p]);
    const float c = inlier_centroid(ca, inlier_code(P, xf));
    const bool dup = e >= k && ((inmax[p >> 5] >> (p & 31)) & 1u);
    A.residual[(size_t)i * 2 * k + e] = dup ? 0.0f : xf - t * c;
  }
}

hipError_t launch_inlier_codes(const QuantArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  const int nvec = a.d_in / 8;
  const size_t lds = 2 * (size_t)a.d_in + 2 * (size_t)((a.d_in + 31) / 32) * 4;
  auto go = [&](auto kern) {
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute((const void*)kern,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(a.n), dim3(256), lds, s, a);
    return hipGetLastError();
  };
  if (nvec <= 256) return go(k_inlier_codes<1>);
  if (nvec <= 512) return go(k_inlier_codes<2>);
  if (nvec <= 1024) return go(k_inlier_codes<4>);
  if (nvec <= 2048) return go(k_inlier_codes<8>);
  if (nvec <= 4096) return go(k_inlier_codes<16>);
  return go(k_inlier_codes<32>);
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t s) { return launch_parts<true, true>(a, s); }
hipError_t launch_cluster(const QuantArgs& a, hipStream_t s) { return launch_parts<true, false>(a, s); }
hipError_t launch_outliers(const QuantArgs& a, hipStream_t s) {
  if (a.k == 0) return hipSuccess;
  return launch_parts<false, true>(a, s);
}

}  // namespace oasis
