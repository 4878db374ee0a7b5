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
// Top-k is a two-level radix select on the keys shared by the max and min
// lists: a histogram of the high byte fixes the bucket holding the k-th
// largest (smallest) key, a histogram of the low byte inside it the exact
// threshold key T and the count G < k of keys strictly beyond it.  Keys equal
// to T are taken in channel order (a block-wide exclusive count gives each its
// rank); the G keys beyond T are ranked among themselves.  The paper's trees
// pop in exactly this order; the select replaces k sequential pops by two
// histogram passes.  Every wave scans the histograms itself (DPP prefix sums),
// so a level costs one barrier, and only the keys at or beyond a threshold
// are visited after the counts.
#include "common.h"

namespace oasis {

struct __align__(16) QuantSmem {
  uint32_t hist1[256];     // high byte of the key
  uint32_t hist2[2][256];  // low byte inside the max / min boundary bucket
  uint16_t bucket[256];    // first index | inside count << 4 | low byte << 8
  float ca[16];            // C_A in fp32
  uint32_t wmax[16];       // per-wave absmax
  uint32_t wtot[2][16];    // per-wave totals of the two packed count pairs
};

// Dynamic LDS after the fixed part: the token (2 B per channel), then G < k
// candidates per list, each a sort key and its residual (max list, then min
// list), padded to a multiple of 4.
static size_t dyn_bytes(int d_in, int k) {
  const size_t k4 = ((size_t)k + 3) & ~(size_t)3;
  return (size_t)d_in * 2 + 16 * k4;
}

size_t quantize_lds_bytes(int d_in, int k) { return sizeof(QuantSmem) + dyn_bytes(d_in, k); }

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
  const uint32_t k4 = ((uint32_t)k + 3u) & ~3u;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem_raw + sizeof(QuantSmem));
  uint32_t* cmax = reinterpret_cast<uint32_t*>(xs + d_in);  // d_in % 8 == 0: 16-byte aligned
  float* rmax = reinterpret_cast<float*>(cmax + k4);
  uint32_t* cmin = reinterpret_cast<uint32_t*>(rmax + k4);
  float* rmin = reinterpret_cast<float*>(cmin + k4);

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
  if (tid < 16) S.ca[tid] = h2f(A.lut->cb_act[tid]);
  __syncthreads();  // histograms cleared, C_A staged

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
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        atomicAdd(&S.hist1[(key[u][q] >> 8) & 0xFFu], 1u);
        atomicAdd(&S.hist1[key[u][q] >> 24], 1u);
      }
    }
  }
  amax = wave_max(amax);
  if (lane == 0) S.wmax[wave] = amax;
  __syncthreads();  // absmax partials, level-1 histogram

#pragma unroll
  for (int w = 0; w < NW; ++w) amax = max(amax, S.wmax[w]);
  const float t = (A.scale_mode == OASIS_SCALE_NONE) ? 1.0f : h2f((uint16_t)amax);
  if (CLUSTER && tid == 0) A.act_scale[i] = t;

  // ---- boundary keys: lane c computes key(Q_c), Q_c = the smallest fp16 not
  // below P_c = fp32(t * b_c), b_c = fp32(C_A[c] + C_A[c+1]) * 0.5
  const int nb = (1 << A.b_a) - 1;
  uint32_t kq_lane = 0x10000u;  // above every key: boundaries past the last one
  if (lane < nb) {
    const float bc = (S.ca[lane] + S.ca[lane + 1]) * 0.5f;
    const float P = t * bc;
    const _Float16 h = (_Float16)P;  // round to nearest even
    kq_lane = ord_key(__builtin_bit_cast(uint16_t, h)) + ((float)h < P ? 1u : 0u);
  }
  uint32_t KQ[15];
#pragma unroll
  for (int c = 0; c < 15; ++c) KQ[c] = (uint32_t)__builtin_amdgcn_readlane((int)kq_lane, c);
  // cluster index by the full count
  auto code_full = [&](uint32_t kk) -> uint32_t {
    uint32_t a = 0;
#pragma unroll
    for (int c = 0; c < 15; ++c) a += kk >= KQ[c] ? 1u : 0u;
    return a;
  };
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

  // ---- level 1: the high-byte buckets holding the k-th largest and k-th
  // smallest key (each wave scans the histogram itself)
  uint32_t B1max, G1max, B1min, G1min;
  {
    const uint4 h = *reinterpret_cast<const uint4*>(&S.hist1[4 * lane]);
    const uint32_t hs[4] = {h.x, h.y, h.z, h.w};
    const uint32_t sum = h.x + h.y + h.z + h.w;
    uint32_t pre = wave_incl_scan(sum) - sum;  // keys in buckets below 4*lane
    uint32_t fmax = 0, gmax = 0, fmin = 0, gmin = 0;
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
  }
  // ---- level 2: low bytes inside the two boundary buckets
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    if (tid * VR + u < nvec) {
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

  uint32_t Tmax, Gmax, Tmin, Gmin;
  {
    const uint4 hm = *reinterpret_cast<const uint4*>(&S.hist2[0][4 * lane]);
    const uint4 hn = *reinterpret_cast<const uint4*>(&S.hist2[1][4 * lane]);
    const uint32_t ms[4] = {hm.x, hm.y, hm.z, hm.w}, ns[4] = {hn.x, hn.y, hn.z, hn.w};
    const uint32_t summ = hm.x + hm.y + hm.z + hm.w, sumn = hn.x + hn.y + hn.z + hn.w;
    uint32_t prem = wave_incl_scan(summ) - summ, pren = wave_incl_scan(sumn) - sumn;
    const uint32_t totm = S.hist1[B1max];
    const uint32_t kk = (uint32_t)k - G1max, kn = (uint32_t)k - G1min;
    uint32_t tm = 0, gm = 0, tn = 0, gn = 0;
    bool hit_max = false, hit_min = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t uptom = prem + ms[q];
      const uint32_t above = totm - uptom;  // keys of the bucket with a higher low byte
      const bool hmq = above < kk && kk <= above + ms[q];
      tm = hmq ? ((B1max << 8) | (uint32_t)(4 * lane + q)) : tm;
      gm = hmq ? G1max + above : gm;
      const uint32_t upton = pren + ns[q];
      const bool hnq = pren < kn && kn <= upton;
      tn = hnq ? ((B1min << 8) | (uint32_t)(4 * lane + q)) : tn;
      gn = hnq ? G1min + pren : gn;
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
  }
  // G < k holds by construction; the clamp only keeps every index in bounds.
  Gmax = min(Gmax, (uint32_t)k - 1u);
  Gmin = min(Gmin, (uint32_t)k - 1u);
  const uint32_t need_max = (uint32_t)k - Gmax, need_min = (uint32_t)k - Gmin;

  // ---- codes; per-thread counts in channel order of (max-list ties, min-list
  // ties) and (keys above Tmax, keys below Tmin), 16 bits each; the keys at
  // or beyond a threshold (the only ones a list can take)
  make_codes();
  if (CLUSTER) store_codes();
  uint32_t c_tie = 0, c_out = 0;
  uint64_t special = 0;
#pragma unroll
  for (int u = 0; u < VR; ++u) {
    if (tid * VR + u < nvec) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const uint32_t kk = (key[u][q] >> (16 * hh)) & 0xFFFFu;
          c_tie += (kk == Tmax ? 1u : 0u) + (kk == Tmin ? 0x10000u : 0u);
          c_out += (kk > Tmax ? 1u : 0u) + (kk < Tmin ? 0x10000u : 0u);
          special |= (uint64_t)((kk >= Tmax) | (kk <= Tmin)) << (8 * u + 2 * q + hh);
        }
      }
    }
  }
  // block-wide exclusive prefix: wave scan, wave totals through LDS.  A
  // prefix counts keys before this thread, < 65536, so the fields never carry.
  const uint32_t inc_tie = wave_incl_scan(c_tie), inc_out = wave_incl_scan(c_out);
  if (lane == 63) {
    S.wtot[0][wave] = inc_tie;
    S.wtot[1][wave] = inc_out;
  }
  // pad the candidate lists to a multiple of 4 with entries that never rank
  // first (sort keys are compared after XOR with 0 for the max list and with
  // ~0 for the min list, which turns a pad into 0)
  if (tid < 4) {
    if (Gmax + (uint32_t)tid < k4) cmax[Gmax + tid] = 0u;
    if (Gmin + (uint32_t)tid < k4) cmin[Gmin + tid] = 0xFFFFFFFFu;
  }
  __syncthreads();  // wave totals
  uint32_t ex_tie = inc_tie - c_tie, ex_out = inc_out - c_out;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    if (w < wave) {
      ex_tie += S.wtot[0][w];
      ex_out += S.wtot[1][w];
    }
  }
  uint32_t rank_max = ex_tie & 0xFFFFu, rank_min = ex_tie >> 16;
  uint32_t slot_max = ex_out & 0xFFFFu, slot_min = ex_out >> 16;

  const size_t krow = (size_t)i * k;
  const size_t rrow = (size_t)i * 2 * k;
  // ---- collect, in channel order: threshold ties go straight to their list
  // position, the keys beyond the thresholds to candidate slots
  while (special) {
    const int e = __builtin_ctzll(special);
    special &= special - 1;
    const int p = 8 * (tid * VR + (e >> 3)) + (e & 7);
    uint32_t cw = codes[0];
#pragma unroll
    for (int u = 1; u < VR; ++u) cw = (e >> 3) == u ? codes[u] : cw;
    const uint32_t a = (cw >> (4 * (e & 7))) & 15u;
    // two independent LDS reads: the raw value (staged by this thread) and its
    // centroid; t * C_A[a] is exact, a product of two fp16 values
    const uint32_t bits = xs[p];
    const float xhat = t * S.ca[a];
    const uint32_t kk = ord_key(bits);
    const float r = h2f((uint16_t)bits) - xhat;
    const bool tie_max = kk == Tmax && rank_max < need_max;
    const bool in_max = kk > Tmax || tie_max;
    if (tie_max) {
      A.max_idx[krow + Gmax + rank_max] = p;
      A.residual[rrow + Gmax + rank_max] = r;
    }
    if (kk > Tmax && slot_max < Gmax) {
      cmax[slot_max] = (kk << 16) | (0xFFFFu - (uint32_t)p);
      rmax[slot_max] = r;
    }
    if (kk == Tmin && rank_min < need_min) {
      A.min_idx[krow + Gmin + rank_min] = p;
      A.residual[rrow + k + Gmin + rank_min] = in_max ? 0.0f : r;
    }
    if (kk < Tmin && slot_min < Gmin) {
      cmin[slot_min] = (kk << 16) | (uint32_t)p;
      rmin[slot_min] = in_max ? 0.0f : r;
    }
    rank_max += kk == Tmax ? 1u : 0u;
    slot_max += kk > Tmax ? 1u : 0u;
    rank_min += kk == Tmin ? 1u : 0u;
    slot_min += kk < Tmin ? 1u : 0u;
  }
  __syncthreads();  // candidates

  // ---- rank the candidates: the first half of the waves the max list, the
  // second half the min list; each counts the candidates that pop before it
  {
    constexpr int HALF = NT / 2;
    const bool is_max = wave < NW / 2;  // uniform
    const uint32_t G = is_max ? Gmax : Gmin;
    const uint32_t flip = is_max ? 0u : 0xFFFFFFFFu;
    const uint32_t* cand = is_max ? cmax : cmin;
    const uint4* c4 = reinterpret_cast<const uint4*>(cand);
    const uint32_t nq = (G + 3u) / 4u;
    for (uint32_t c = (uint32_t)(tid & (HALF - 1)); c < G; c += HALF) {
      const uint32_t mine = cand[c] ^ flip;
      uint32_t rank = 0;
#pragma unroll 4
      for (uint32_t q = 0; q < nq; ++q) {
        const uint4 o = c4[q];  // the same 16 bytes in every lane
        rank += ((o.x ^ flip) > mine ? 1u : 0u) + ((o.y ^ flip) > mine ? 1u : 0u) +
                ((o.z ^ flip) > mine ? 1u : 0u) + ((o.w ^ flip) > mine ? 1u : 0u);
      }
      if (is_max) {
        A.max_idx[krow + rank] = (int)(0xFFFFu - (mine & 0xFFFFu));
        A.residual[rrow + rank] = rmax[c];
      } else {
        A.min_idx[krow + rank] = (int)(~mine & 0xFFFFu);
        A.residual[rrow + k + rank] = rmin[c];
      }
    }
  }
}

template <int NT, int VR, bool CL, bool TK>
static hipError_t launch_nt(const QuantArgs& a, hipStream_t s) {
  const size_t lds = sizeof(QuantSmem) + (TK ? dyn_bytes(a.d_in, a.k) : 0);
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

hipError_t launch_quantize(const QuantArgs& a, hipStream_t s) { return launch_parts<true, true>(a, s); }
hipError_t launch_cluster(const QuantArgs& a, hipStream_t s) { return launch_parts<true, false>(a, s); }
hipError_t launch_outliers(const QuantArgs& a, hipStream_t s) {
  if (a.k == 0) return hipSuccess;
  return launch_parts<false, true>(a, s);
}

}  // namespace oasis
