// Error compensation of the outlier branch (Sec. III-C2):
//   Y'[i][j] = s_j * sum_e r_ie * C_W[w(p_ie, j)].
// Each listed outlier channel p fetches input channel p of the weight codes
// (one contiguous row of words in the input-channel-major layout), the codes
// are dequantized with the weight codebook (the Dequant Unit) and multiplied
// by the residual (the MAC units), then merged into the main-branch output.
//
// Two kernels.  k_compensate (few tokens): one workgroup per (token, 64 or
// 256 output columns); its 4 waves split the token's 2k listed channels and
// are summed through LDS.  A lane owns one or four columns and issues the word
// loads of 16 listed channels before using any of them.  Channel ids and
// residuals are wave-uniform; zero residuals (channels already compensated
// through the max list) are skipped.
//
// k_compensate_rows (many tokens): a 32-bit word of the codes holds 8 input
// channels, so fetching it for one outlier uses 4 of its 32 bits.  A workgroup
// takes a tile of tokens, counting-sorts their listed outliers by word row in
// LDS and fetches every touched row once for all the tile's outliers in it;
// outlier channels recur across tokens, so rows are shared.
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


// ----------------------------------------------------------------------------
// Row-grouped compensation.  Workgroup = (tile of up to TT tokens,
// NW * 64 * CPL output columns); lane l of wave w owns CPL consecutive columns
// and one register accumulator per (token, column).  The tile's live entries
// (nonzero residual) are sorted by word row, then channel, then token: a run
// of entries on one channel needs one codebook lookup per column for all its
// tokens, and every sum is taken in a fixed order.  Every wave walks all
// touched rows for its own columns.  A run's token mask drives an unrolled
// loop over the tile's tokens, so each accumulator stays in a fixed register.
//
// Entry meta word: token (bits 0-4), channel within the row (5-7); the first
// entry of a run also carries the run's token mask (8-15), bit 16 and the
// run's length (17-29).
// ----------------------------------------------------------------------------
constexpr int ROW_TT = 4;       // tokens per tile, at most (<= 8: token mask)
constexpr int ROW_EMAX = 4096;  // listed entries of a tile held in LDS
constexpr int ROW_PF = 4;       // rows of codes in flight per wave

// LDS bytes of one workgroup: codebook, per-row counters, entries (meta and
// residual), touched-row list and row starts.
static size_t rows_lds_bytes(int d_in, int tt, int k) {
  const size_t R = (size_t)d_in / 8, emax = (size_t)tt * 2 * k;
  const size_t rmax = R < emax ? R : emax;
  return 64 + 4 * R + 8 * emax + 4 * rmax + 4 * (rmax + 1) + 16;
}

template <int TT, int CPL, int NW>
__global__ void __launch_bounds__(NW * 64) k_compensate_rows(CompArgs A, int tt, int ncol_tiles,
                                                             int ntok_tiles) {
  constexpr int NT = NW * 64;
  static_assert(TT >= 1 && TT <= 8, "the run token mask has 8 bits");
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ uint64_t scan_tmp[NW];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int d_in = A.d_in, d_out = A.d_out, k = A.k, E2 = 2 * k;
  const int R = d_in >> 3;
  const int emax = tt * E2;
  const int rmax = min(R, emax);
  float* cwf = reinterpret_cast<float*>(smem);                    // 16
  uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + 64);         // R: count, then fill
  uint32_t* meta = cnt + R;                                       // emax
  float* rv = reinterpret_cast<float*>(meta + emax);              // emax
  uint32_t* rowlist = reinterpret_cast<uint32_t*>(rv + emax);     // rmax
  uint32_t* rowbeg = rowlist + rmax;                              // rmax + 1
  uint32_t* nrow_s = rowbeg + rmax + 1;

  // token tiles fastest, so one XCD sweeps every token tile of a column slab
  // while the slab's rows sit in its L2
  const int tile = xcd_tile(blockIdx.x, ncol_tiles * ntok_tiles);
  const int tk = tile % ntok_tiles, ct = tile / ntok_tiles;
  const int tok0 = tk * tt;
  const int ntok = min(tt, A.n - tok0);
  const int e_tot = ntok * E2;

  if (tid < 16) cwf[tid] = h2f(A.lut->cb_wgt[tid]);
  for (int r = tid; r < R; r += NT) cnt[r] = 0u;
  __syncthreads();

  // entry f of the tile: token tok0 + f / 2k, list position f % 2k
  auto entry = [&](int f, int& t, int& e, int& p, float& r) -> bool {
    t = f / E2;
    e = f - t * E2;
    const size_t i = (size_t)(tok0 + t);
    p = e < k ? A.max_idx[i * k + e] : A.min_idx[i * k + (e - k)];
    r = A.residual[i * E2 + e];
    return r != 0.0f && p >= 0 && p < d_in;
  };
  for (int f = tid; f < e_tot; f += NT) {
    int t, e, p;
    float r;
    if (entry(f, t, e, p, r)) atomicAdd(&cnt[p >> 3], 1u);
  }
  __syncthreads();

  // exclusive scan over the rows (each thread a contiguous run): entry
  // offsets, and the ascending list of touched rows
  {
    const int rpt = (R + NT - 1) / NT;
    const int r0 = min(R, tid * rpt), r1 = min(R, r0 + rpt);
    uint64_t loc = 0;
    for (int r = r0; r < r1; ++r) loc += (uint64_t)cnt[r] | ((uint64_t)(cnt[r] != 0u) << 32);
    const uint64_t excl = block_scan64<NT>(loc, scan_tmp) - loc;
    uint32_t off = (uint32_t)excl, nr = (uint32_t)(excl >> 32);
    for (int r = r0; r < r1; ++r) {
      const uint32_t c = cnt[r];
      if (c) {
        rowlist[nr] = (uint32_t)r;
        rowbeg[nr] = off;
        ++nr;
      }
      cnt[r] = off;  // fill pointer
      off += c;
    }
    if (tid == NT - 1) {
      rowbeg[nr] = off;
      *nrow_s = nr;
    }
  }
  __syncthreads();
  for (int f = tid; f < e_tot; f += NT) {
    int t, e, p;
    float r;
    if (entry(f, t, e, p, r)) {
      const uint32_t pos = atomicAdd(&cnt[p >> 3], 1u);
      meta[pos] = ((uint32_t)(p & 7) << 5) | (uint32_t)t;
      rv[pos] = r;
    }
  }
  __syncthreads();
  const uint32_t nrow = *nrow_s;
  // each row: insertion sort by (channel, token) - atomics placed the entries
  // in arbitrary order; a (channel, token) pair occurs once - then mark the
  // runs of one channel with their token masks
  for (uint32_t j = tid; j < nrow; j += NT) {
    const uint32_t b = rowbeg[j], e_end = rowbeg[j + 1];
    for (uint32_t q = b + 1; q < e_end; ++q) {
      const uint32_t m = meta[q];
      const float v = rv[q];
      uint32_t z = q;
      while (z > b && meta[z - 1] > m) {
        meta[z] = meta[z - 1];
        rv[z] = rv[z - 1];
        --z;
      }
      meta[z] = m;
      rv[z] = v;
    }
    for (uint32_t q = b; q < e_end;) {
      const uint32_t ch = meta[q] >> 5;
      uint32_t tm = 0, z = q, w = q;
      for (; z < e_end && (meta[z] >> 5) == ch; ++z) {
        const uint32_t t = meta[z] & 31u;
        if (tm & (1u << t)) {
          rv[w - 1] += rv[z];  // a token listing the channel twice: one entry
        } else {
          tm |= 1u << t;
          meta[w] = meta[z];
          rv[w] = rv[z];
          ++w;
        }
      }
      // live entries [q, w) in token order; [w, z) are never read
      meta[q] |= (tm << 8) | (1u << 16) | ((z - q) << 17);
      q = z;
    }
  }
  __syncthreads();

  // ---- accumulate: every wave walks all touched rows for its columns.
  // Row data and entries are read 64 at a time into lanes (lane u holds
  // item base + u) and handed out as scalars with readlane, so no LDS read
  // sits on the per-row path.  A row's offset into the codes is the scalar
  // offset of its buffer loads.
  const int j0 = ct * (NW * 64 * CPL) + wave * 64 * CPL + lane * CPL;
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(A.idx_w), 0, (int)((uint32_t)R * (uint32_t)d_out * 4u), 0x00020000);
  const uint32_t voff = (uint32_t)j0 * 4u;
  const uint32_t row_bytes = (uint32_t)d_out * 4u;
  auto window = [&](const uint32_t* src, uint32_t first, uint32_t count, uint32_t fill) {
    return first + lane < count ? src[first + lane] : fill;
  };
  // load stream: rows [lw0, lw0 + 64) of the list in lanes.  The row's offset
  // is added to the lane's (the descriptor's size check then covers the whole
  // offset: columns past d_out in the last row read zeros)
  uint32_t lw0 = 0, lw_row = window(rowlist, 0, nrow, 0u);
  auto load_batch = [&](uint32_t base, uint32_t (&w)[ROW_PF][CPL]) {
    if (base >= lw0 + 64) {  // batches are 64-aligned: slide the window
      lw0 += 64;
      lw_row = window(rowlist, lw0, nrow, 0u);
    }
#pragma unroll
    for (int d = 0; d < ROW_PF; ++d) {
      const uint32_t j = base + d;
      const uint32_t row = (uint32_t)__builtin_amdgcn_readlane((int)lw_row, (int)(j - lw0));
      // rows past the list read row 0 (in bounds) and are never used
      const uint32_t roff = j < nrow ? row * row_bytes : 0u;
      if constexpr (CPL % 4 == 0) {
#pragma unroll
        for (int h = 0; h < CPL / 4; ++h) {
          const uint4_t v = __builtin_bit_cast(
              uint4_t, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(roff + voff + 16u * h), 0, 0));
          w[d][4 * h] = v[0]; w[d][4 * h + 1] = v[1]; w[d][4 * h + 2] = v[2]; w[d][4 * h + 3] = v[3];
        }
      } else {
        w[d][0] = __builtin_amdgcn_raw_buffer_load_b32(rw, (int)(roff + voff), 0, 0);
      }
    }
  };
  float acc[TT][CPL];
#pragma unroll
  for (int t = 0; t < TT; ++t)
#pragma unroll
    for (int c = 0; c < CPL; ++c) acc[t][c] = 0.0f;

  // processing stream: rows [pw0, pw0 + 64) and entries [ew0, ew0 + 64)
  uint32_t pw0 = 0;
  uint32_t pw_beg = window(rowbeg, 0, nrow + 1, 0u), pw_end = window(rowbeg, 1, nrow + 1, 0u);
  uint32_t ew0 = 0;
  uint32_t ew_m = window(meta, 0, emax, 0u);
  float ew_r = __builtin_bit_cast(float, window(reinterpret_cast<const uint32_t*>(rv), 0, emax, 0u));

  uint32_t wv[2][ROW_PF][CPL];
  load_batch(0, wv[0]);
  for (uint32_t jb = 0; jb < nrow; jb += 2 * ROW_PF) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t base = jb + h * ROW_PF;
      load_batch(base + ROW_PF, wv[h ^ 1]);  // next batch in flight
#pragma unroll
      for (int d = 0; d < ROW_PF; ++d)  // wait for this batch only
#pragma unroll
        for (int c = 0; c < CPL; ++c) asm volatile("" : "+v"(wv[h][d][c]));
      if (base >= pw0 + 64) {
        pw0 += 64;
        pw_beg = window(rowbeg, pw0, nrow + 1, 0u);
        pw_end = window(rowbeg, pw0 + 1, nrow + 1, 0u);
      }
#pragma unroll
      for (int d = 0; d < ROW_PF; ++d) {
        const uint32_t j = base + d;
        // rows past the list: an empty range
        const int u = (int)(j - pw0);
        const uint32_t b = j < nrow ? (uint32_t)__builtin_amdgcn_readlane((int)pw_beg, u) : 0u;
        const uint32_t e_end = j < nrow ? (uint32_t)__builtin_amdgcn_readlane((int)pw_end, u) : 0u;
        for (uint32_t q = b; q < e_end;) {
          // a run: one channel, at most TT entries, in token order
          if (q + TT > ew0 + 64) {  // entries are consumed in order: slide
            ew0 = q;
            ew_m = window(meta, ew0, emax, 0u);
            ew_r = __builtin_bit_cast(float, window(reinterpret_cast<const uint32_t*>(rv), ew0, emax, 0u));
          }
          const uint32_t m = (uint32_t)__builtin_amdgcn_readlane((int)ew_m, (int)(q - ew0));
          const uint32_t tm = (m >> 8) & 0xFFu;
          const uint32_t sh = ((m >> 5) & 7u) * 4u;
          float cv[CPL];
#pragma unroll
          for (int c = 0; c < CPL; ++c) cv[c] = cwf[(wv[h][d][c] >> sh) & 15u];
          int pos = (int)(q - ew0);
#pragma unroll
          for (int T = 0; T < TT; ++T) {
            if (tm & (1u << T)) {
              const float r = __builtin_bit_cast(
                  float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ew_r), pos));
              ++pos;
#pragma unroll
              for (int c = 0; c < CPL; ++c) acc[T][c] = fmaf(r, cv[c], acc[T][c]);
            }
          }
          q += max(1u, (m >> 17) & 0x1FFFu);  // the run's length (>= 1 always advances)
        }
      }
    }
  }

  // ---- merge: y (+)= s_j * acc
  float sw[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) sw[c] = (j0 + c < d_out) ? A.w_scale[j0 + c] : 0.0f;
#pragma unroll
  for (int t = 0; t < TT; ++t) {
    float* dst = A.y + (size_t)(tok0 + t) * d_out + j0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      if (t < ntok && j0 + c < d_out) {
        const float v = sw[c] * acc[t][c];
        dst[c] = A.accumulate ? dst[c] + v : v;
      }
    }
  }
}

// ----------------------------------------------------------------------------
// Compensation from the row layout: idx_wr uint32 [d_in][wn], wn =
// ceil(d_out / 8), word m of row p holds the codes of input channel p for
// output columns 8m .. 8m + 7 (column 8m + c in bits 4c .. 4c + 3).  One
// listed outlier reads exactly its own row, d_out / 2 bytes.
//
// Workgroup = 16 waves over a slab of 64 words (512 columns) and a tile of
// tt tokens; wave w takes tokens w, w + 16, ... of the tile.  Lane l owns
// word 64 * slab + l and 8 fp32 accumulators per token.  A token's listed
// entries are wave-uniform: lane e holds entry e, readlane hands out the
// channels and a broadcast LDS read the residuals, in list order, and each
// entry fetches one word per lane (one contiguous
// 256-byte piece of row p per wave, 3 * WR_U entries in flight).  A word's four
// bytes become four pairs of weight centroids through a 64 KiB LDS table -
// row `byte` holds 32 copies of the pair as two fp32 values, lane l reads
// copy l mod 32, so the 8-byte reads are conflict free and the offset is one
// v_perm_b32 - and each centroid meets the residual in one v_fma_f32 (the
// fp16-operand v_fma_mix_f32 issues at half its rate; fp32 pairs: 712 ->
// 680 us at 4096 x 8192 x 28672).  Sixteen waves share the table (128 KiB of LDS with their
// lists): four waves per SIMD hide the row loads, where 4-wave workgroups
// with their own table fit two (64 copies) or three (32 copies, one more
// shift per lookup) on a CU.
// ----------------------------------------------------------------------------
constexpr int WR_U = 16;    // entries per unit of word loads
constexpr int WR_C = 512;   // list entries per wave held in LDS at a time
constexpr int WR_W = 16;    // waves per workgroup

__global__ void __launch_bounds__(64 * WR_W) k_compensate_wr(CompArgs A, int wn, int nslab,
                                                        int ntile, int tt) {
  // the pair table at a fixed LDS address; dynamic LDS: per wave WR_C
  // channels and WR_C residuals of its lists
  __shared__ uint32_t tab[256 * 64];
  extern __shared__ __align__(16) unsigned char smem_wr[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int* lp = reinterpret_cast<int*>(smem_wr) + wave * WR_C;
  float* lr = reinterpret_cast<float*>(smem_wr + 4 * WR_W * WR_C) + wave * WR_C;
  const int r = xcd_tile(blockIdx.x, nslab * ntile);
  const int slab = r / ntile, tile = r % ntile;  // token tiles of a slab on one XCD
  const int k = A.k, E = 2 * k, d_in = A.d_in, d_out = A.d_out;

  // ---- this wave's tokens, in units of WR_U entries
  const int tok0 = tile * tt;
  const int tw = tok0 + wave;  // first token of this wave; then every WR_W-th
  const int tend = min(A.n, tok0 + tt);
  const int ntw = tw < tend ? (tend - tw + WR_W - 1) / WR_W : 0;
  // units per token: the whole list, or with compacted lists the token's own
  // entries (at least one unit when y is overwritten: a token's last unit
  // writes y; none for a token without entries when adding into y).  Lane
  // j < ntw holds the first unit past token tw + 4j (inclusive prefix sum);
  // units are numbered over the wave's tokens in order.
  const int nch = (E + WR_U - 1) / WR_U;
  int nu = 0;
  if (lane < ntw) {
    nu = nch;
    if (A.cnt) {
      nu = (min(max(A.cnt[tw + WR_W * lane], 0), E) + WR_U - 1) / WR_U;
      if (!A.accumulate) nu = max(1, nu);
    }
  }
  const int uend = (int)wave_incl_scan((uint32_t)nu);
  const int U = __builtin_amdgcn_readlane(uend, 63);
  // token slot j of unit u (the first j whose end exceeds u) and its first unit
  auto unit_token = [&](int u, int& j, int& ubeg) {
    j = 0;
    ubeg = 0;
    for (int q = 0; q + 1 < ntw; ++q) {
      const int endq = __builtin_amdgcn_readlane(uend, q);
      if (u >= endq) {
        j = q + 1;
        ubeg = endq;
      }
    }
  };
  // copy the lists of units [c0, c1) into this wave's LDS area, validated:
  // dead entries (past the lists, duplicates with residual 0, channels out of
  // range) get channel -1 and residual 0.  LDS operations of one wave run in
  // order, so the wave reads its area without a barrier.
  auto fill = [&](int c0, int c1) {
    constexpr int PER = WR_C / 64;
    int pv[PER];
    float rv[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {  // every load first, then the checks
      const int f = lane + 64 * j;
      const int u = c0 + f / WR_U;
      int slot_j, ubeg;
      unit_token(u, slot_j, ubeg);
      const int i = tw + WR_W * slot_j, e = WR_U * (u - ubeg) + f % WR_U;
      pv[j] = -1;
      rv[j] = 0.0f;
      if (f < (c1 - c0) * WR_U && e < E) {
        if (A.cnt) {  // compacted: max_idx rows hold the channels, 2k long
          if (e < A.cnt[i]) {
            pv[j] = A.max_idx[(size_t)i * E + e];
            rv[j] = A.residual[(size_t)i * E + e];
          }
        } else {
          const int32_t* src =
              e < k ? A.max_idx + (size_t)i * k + e : A.min_idx + (size_t)i * k + (e - k);
          pv[j] = *src;
          rv[j] = A.residual[(size_t)i * E + e];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const bool live = pv[j] >= 0 && pv[j] < d_in && rv[j] != 0.0f;
      lp[lane + 64 * j] = live ? pv[j] : -1;
      lr[lane + 64 * j] = live ? rv[j] : 0.0f;
    }
  };
  fill(0, min(U, WR_C / WR_U));  // the first chunk's loads overlap the table build

  // pair table, 64 KiB: row `byte` holds 32 copies of the fp32 pair
  // (C_W[byte & 15], C_W[byte >> 4]).  Thread t writes chunks c = t + 1024 s
  // (s < 4) of 16 bytes: row c / 16 (low code (t / 16) mod 16, high code
  // t / 256 + 4 s), copies 2 (c mod 16) and 2 (c mod 16) + 1
  {
    static_assert(WR_W == 16, "the table build takes 1024 threads");
    const uint16_t* cb = A.lut->cb_wgt;
    const uint32_t lo = __builtin_bit_cast(uint32_t, h2f(cb[(tid >> 4) & 15]));
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint32_t hi = __builtin_bit_cast(uint32_t, h2f(cb[(tid >> 8) + 4 * s]));
      const uint32_t c = (uint32_t)tid + 1024u * (uint32_t)s;
      *reinterpret_cast<uint4_t*>(&tab[(c >> 4) * 64u + (c & 15u) * 4u]) = uint4_t{lo, hi, lo, hi};
    }
  }

  const uint32_t m = (uint32_t)slab * 64u + (uint32_t)lane;  // this lane's word
  // lanes past the row end read its last word (never stored), so a load stays
  // inside its row whatever part of the offset the size check covers
  const uint32_t voff = min(m, (uint32_t)wn - 1u) * 4u;
  const uint32_t row_bytes = (uint32_t)wn * 4u;
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(A.idx_w), 0, (int)((uint32_t)d_in * row_bytes), 0x00020000);
  // the offset of byte b's entry, b * 256 + (lane mod 32) * 8, is one
  // v_perm_b32 (a ds_read_b64 serves 16 lanes at a time: 32 copies keep
  // every group of 16 on distinct banks)
  const uint32_t loff = (uint32_t)(lane & 31) * 8u;
  const char* tb = reinterpret_cast<const char*>(tab);
  float sw[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const uint32_t j = 8u * m + (uint32_t)c;
    sw[c] = j < (uint32_t)d_out ? A.w_scale[j] : 0.0f;
  }
  const bool vec = (d_out & 3) == 0 && ((reinterpret_cast<uintptr_t>(A.y) & 15u) == 0) &&
                   8u * m + 8u <= (uint32_t)d_out;
  __syncthreads();  // pair table

  // ---- chunks of WR_C entries; inside a chunk three units of word loads
  // stay in flight: step v reads the lists of unit v + 2 from LDS, requests
  // its words (one per lane per entry), then consumes unit v.  Only word
  // loads are in flight, and they retire in order, so each wait covers just
  // the unit consumed.
  auto issue = [&](int pl, uint32_t (&w)[WR_U]) {
#pragma unroll
    for (int e = 0; e < WR_U; ++e) {
      const int pe = __builtin_amdgcn_readlane(pl, e);
      // a dead entry reads row 0 (in bounds); its residual is 0
      const int soff = pe >= 0 ? (int)((uint32_t)pe * row_bytes) : 0;
      w[e] = __builtin_amdgcn_raw_buffer_load_b32(rw, (int)voff, soff, 0);
    }
  };
  float acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = 0.0f;
  // adding into y: the token's y words are requested at its first unit and
  // used at its last (a load right before the store would wait for memory)
  float4 yv[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
  // rl: the unit's residuals, lane e holding entry e (for the skip test);
  // lrv: the same in LDS, read as one broadcast word per entry (a readlane
  // per entry was one VALU instruction of about fourteen: 747 -> 710 us at
  // 4096 x 8192 x 28672)
  auto consume = [&](int u, float rl, const uint32_t (&w)[WR_U], const float* lrv) {
    int slot_j, ubeg;
    unit_token(u, slot_j, ubeg);
    if (A.accumulate && vec && u == ubeg) {
      const float4* s4 = reinterpret_cast<const float4*>(A.y + (size_t)(tw + WR_W * slot_j) * d_out + 8u * m);
      yv[0] = s4[0];
      yv[1] = s4[1];
    }
    // a unit without a live entry (the unused places of OASIS-S lists sit at
    // the end of each list) adds nothing: skip its products
    if (__ballot(rl != 0.0f) != 0) {
#pragma unroll
      for (int e = 0; e < WR_U; ++e) {
        const float re = lrv[e];  // the same LDS word in every lane
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const uint32_t off = __builtin_amdgcn_perm(w[e], loff, 0x0C0C0000u | ((4u + b) << 8));
          const uint2 pr = *reinterpret_cast<const uint2*>(tb + off);
          acc[2 * b] = fmaf(re, __builtin_bit_cast(float, pr.x), acc[2 * b]);
          acc[2 * b + 1] = fmaf(re, __builtin_bit_cast(float, pr.y), acc[2 * b + 1]);
        }
      }
    }
    if (u != __builtin_amdgcn_readlane(uend, slot_j) - 1) return;
    // the token's last unit: y (+)= s_j * acc
    const int i = tw + WR_W * slot_j;
    float* dst = A.y + (size_t)i * d_out + 8u * m;
    if (vec) {
      float4* d4 = reinterpret_cast<float4*>(dst);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float4 o = make_float4(sw[4 * h] * acc[4 * h], sw[4 * h + 1] * acc[4 * h + 1],
                               sw[4 * h + 2] * acc[4 * h + 2], sw[4 * h + 3] * acc[4 * h + 3]);
        if (A.accumulate) {
          o.x += yv[h].x;
          o.y += yv[h].y;
          o.z += yv[h].z;
          o.w += yv[h].w;
        }
        d4[h] = o;
      }
    } else {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        if (8u * m + (uint32_t)c < (uint32_t)d_out) {
          const float v = sw[c] * acc[c];
          dst[c] = A.accumulate ? dst[c] + v : v;
        }
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = 0.0f;
  };

  for (int c0 = 0; c0 < U; c0 += WR_C / WR_U) {
    const int c1 = min(U, c0 + WR_C / WR_U), V = c1 - c0;
    if (c0 > 0) fill(c0, c1);
    __builtin_amdgcn_wave_barrier();
    // lane e < WR_U: entry e of chunk unit v
    auto rd = [&](int v, int& pl, float& rl) {
      pl = -1;
      rl = 0.0f;
      if (v < V && lane < WR_U) {
        pl = lp[v * WR_U + lane];
        rl = lr[v * WR_U + lane];
      }
    };
    int p0, p1, p2;
    float r0, r1, r2;
    uint32_t w0[WR_U], w1[WR_U], w2[WR_U];
    rd(0, p0, r0);
    rd(1, p1, r1);
    issue(p0, w0);
    if (V > 1) issue(p1, w1);
    // (ra, wa): unit v; unit v + 2's lists go to (pc, rc), its words to wc
    auto step = [&](int v, float& ra, uint32_t (&wa)[WR_U], int& pc, float& rc,
                    uint32_t (&wc)[WR_U]) {
      const float ru = ra;
      rd(v + 2, pc, rc);
      if (v + 2 < V) issue(pc, wc);
      consume(c0 + v, ru, wa, lr + v * WR_U);
    };
    for (int v = 0; v < V; v += 3) {
      step(v, r0, w0, p2, r2, w2);
      if (v + 1 < V) step(v + 1, r1, w1, p0, r0, w0);
      if (v + 2 < V) step(v + 2, r2, w2, p1, r1, w1);
    }
    __builtin_amdgcn_wave_barrier();  // the next fill overwrites the area
  }
}

hipError_t launch_compensate_wr(const CompArgs& a, hipStream_t s) {
  if (a.n == 0 || a.d_out == 0) return hipSuccess;
  if (a.k == 0) {
    if (a.accumulate) return hipSuccess;
    return launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
  }
  const int wn = (a.d_out + 7) / 8;
  // tokens per tile: every wave's lists fit its LDS area at once (one copy,
  // no pipeline drain) when 2k <= WR_C / 8 ... WR_C; at most 8 per wave
  const int E = 2 * a.k;
  const int tt = WR_W * max(1, min(8, WR_C / E));
  const int nslab = (wn + 63) / 64, ntile = (a.n + tt - 1) / tt;
  const size_t lds = 8 * WR_W * WR_C;  // dynamic part: the lists
  hipError_t e = hipFuncSetAttribute((const void*)k_compensate_wr,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_compensate_wr, dim3(nslab * ntile), dim3(64 * WR_W), lds, s, a, wn, nslab,
                     ntile, tt);
  return hipGetLastError();
}

hipError_t launch_compensate(const CompArgs& a, hipStream_t s) {
  if (a.n == 0 || a.d_out == 0) return hipSuccess;
  if (a.k == 0) {
    if (a.accumulate) return hipSuccess;
    return launch_fill_zero(a.y, (size_t)a.n * a.d_out, s);
  }
  // many tokens: row-grouped, as long as a tile's lists fit in LDS
  const int tt = a.k <= ROW_EMAX / 2 ? min(ROW_TT, ROW_EMAX / (2 * a.k)) : 0;
  if (a.n > 64 && tt >= 1) {
    constexpr int NW = 4;
    const size_t lds = rows_lds_bytes(a.d_in, tt, a.k);
    const int ntok_tiles = (a.n + tt - 1) / tt;
    auto go = [&](auto kern, int cols) -> hipError_t {
      if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)kern,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
      }
      const int ncol_tiles = (a.d_out + cols - 1) / cols;
      hipLaunchKernelGGL(kern, dim3(ncol_tiles * ntok_tiles), dim3(NW * 64), lds, s, a, tt,
                         ncol_tiles, ntok_tiles);
      return hipGetLastError();
    };
    if ((a.d_out & 3) == 0) return go(k_compensate_rows<ROW_TT, 8, NW>, NW * 64 * 8);
    return go(k_compensate_rows<ROW_TT, 1, NW>, NW * 64);
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
