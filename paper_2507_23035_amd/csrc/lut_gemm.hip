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
// selects a packed pair from an LDS table) and fed to
// v_mfma_f32_16x16x32_f16.  Every product equals its LUT entry bit for bit;
// only the fp32 summation order differs from the literal scheme.
//
// MFMA operand mapping (16x16x32): A = weight codes (row m = output column),
// B = activation codes (column = token).  Lane (g, m), g = lane / 16, holds the
// 8 codes of one 32-bit word.  Within a block of 16 words (128 channels) lane
// group g and step s use word 4g + s on both sides, so the weight rows are read
// as contiguous segments and each token's 4 words as one 16-byte load; the
// order in which channels enter the MFMA is irrelevant to the sum.
#include <atomic>

#include "common.h"

namespace oasis {

// ----------------------------------------------------------------------------
// shared helpers
// ----------------------------------------------------------------------------

// Dual decode table in LDS (64 KiB): row `byte` (256 bytes) holds 32 copies of
// the weight entry pair(C_W, byte), then 32 copies of the activation entry
// pair(C_A, byte), pair(C, b) = C[b & 15] | C[b >> 4] << 16 (fp16 bits).  Lane
// l reads copy l mod 32, so the byte offset of an entry is
// byte * 256 + (l mod 32) * 4 (+ 128 for activations): one v_perm_b32 per byte,
// and the 32 lanes of a half-wave always hit 32 different banks.
// Written with 16-byte stores by the first four waves only (16 stores per
// lane): wave w, lane l, step j writes chunk c = 1024 w + l + 64 j, i.e. row
// c / 16, side (l / 8) mod 2, low code (l / 16 + 4 j) mod 16 and high code
// 4 w + j / 4.  The codebooks come in through scalar loads - four waves per
// workgroup rather than all of them ask for the same 64 bytes - off the vector
// memory queue that the weight stream fills; every code index is then a
// compile-time constant or lane / 16.
struct DualTableLoader {
  uint32_t cw[8], ca[8];  // C_W, C_A as fp16 pairs (SGPRs)
  uint32_t hw[2], ha[2];  // the pairs holding codes 4w .. 4w + 3
  // wave < 4 only
  __device__ __forceinline__ void load(const oasis_lut_block* lut, uint32_t wave) {
    // constant address space: scalar loads, also through a pointer the compiler
    // cannot trace back to a kernel argument
    using cu32 = const __attribute__((address_space(4))) uint32_t;
    cu32* w32 = (cu32*)reinterpret_cast<const uint32_t*>(lut->cb_wgt);
    cu32* a32 = (cu32*)reinterpret_cast<const uint32_t*>(lut->cb_act);
    // readfirstlane keeps every value a scalar load: without it the compiler
    // may turn the per-lane choice between the two codebooks into a choice of
    // address, i.e. a vector load that waits behind the weight stream
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      cw[q] = __builtin_amdgcn_readfirstlane(w32[q]);
      ca[q] = __builtin_amdgcn_readfirstlane(a32[q]);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      hw[q] = __builtin_amdgcn_readfirstlane(w32[2 * wave + q]);
      ha[q] = __builtin_amdgcn_readfirstlane(a32[2 * wave + q]);
    }
  }
  // ACT_ONLY: the weight half is written elsewhere (per-column codebooks)
  template <bool ACT_ONLY = false>
  __device__ __forceinline__ void store(uint32_t* tab, uint32_t wave, int lane) const {
    const bool act = (lane >> 3) & 1;
    if (ACT_ONLY && !act) return;
    const int lq = lane >> 4;
    auto half = [](uint32_t pair, int h) -> uint32_t { return (pair >> (16 * h)) & 0xFFFFu; };
    // low code of step j: lane / 16 + 4 (j mod 4); high code: 4w + j / 4
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      uint32_t lw = 0, la = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int code = u + 4 * jj;
        lw = lq == u ? half(cw[code >> 1], code & 1) : lw;
        la = lq == u ? half(ca[code >> 1], code & 1) : la;
      }
      lo[jj] = act ? la : lw;
      hi[jj] = (act ? half(ha[jj >> 1], jj & 1) : half(hw[jj >> 1], jj & 1)) << 16;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t v = lo[j & 3] | hi[j >> 2];
      reinterpret_cast<uint4_t*>(tab)[1024u * wave + (uint32_t)lane + 64u * (uint32_t)j] =
          uint4_t{v, v, v, v};
    }
  }
};

// Eight codes -> eight fp16 centroid values (VGPR v holds the two channels of
// byte v): the table offset of byte v is assembled by one v_perm_b32 from the
// code word and the lane's offset `lane4` (< 256).
__device__ __forceinline__ half8_t expand_dual(uint32_t w, const char* tab, uint32_t lane4) {
  uint4_t r;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t off = __builtin_amdgcn_perm(w, lane4, 0x0C0C0000u | ((4u + b) << 8));
    r[b] = *reinterpret_cast<const uint32_t*>(tab + off);
  }
  return __builtin_bit_cast(half8_t, r);
}

// C_W[code] from the weight half of the dual table (row `code` holds
// pair(C_W, code), whose low half is C_W[code]).
__device__ __forceinline__ float weight_centroid(const char* tab, uint32_t code, uint32_t lane4) {
  return h2f((uint16_t)*reinterpret_cast<const uint32_t*>(tab + ((code << 8) | lane4)));
}

// Raw codes of one block of 16 words for one wave: the activation words of
// its tokens (4 consecutive words per lane) and, for each of the 4 steps, CW
// consecutive weight words (CW output columns) per lane.
template <int CW, int TF>
struct BlockCodes {
  uint4_t av[TF];
  uint32_t wv[4][CW];
};

// Buffer loads of a block of codes for the GEMV kernel.  Per-lane byte offsets
// are computed once and the block's offset is added to them, so the whole
// offset is in the per-lane operand that the descriptor's size check covers:
// a read past the end returns 0 instead of faulting.  Columns past d_out or
// tokens past n only feed outputs that are never stored, the words of a last,
// partial K block are masked in mma_block, and a block past the last one
// (index clamped to nblk) reads zeros.
struct GemvAddr {
  __amdgpu_buffer_rsrc_t rw, ra;
  uint32_t woff[4];  // byte offset of (row 4g + s, column j0 + CW*m) in block 0
  uint32_t aoff;     // byte offset of (token m, word 4g) in block 0
  uint32_t wblk;     // bytes per block of 16 weight rows
  uint32_t astride;  // bytes between token tiles (16 tokens)
  uint32_t nblk;     // blocks of 16 weight rows (the last may be partial)
};

template <int CW>
__device__ __forceinline__ GemvAddr gemv_addr(const GemmArgs& A, int j0) {
  const int lane = threadIdx.x & 63, g = lane >> 4, m = lane & 15;
  const uint32_t KB = (uint32_t)(A.d_in >> 3);
  GemvAddr ad;
  ad.rw = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(A.idx_w), 0,
                                            (int)(KB * (uint32_t)A.d_out * 4u), 0x00020000);
  ad.ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(A.idx_act), 0,
                                            (int)((uint32_t)A.n * KB * 4u), 0x00020000);
#pragma unroll
  for (int s = 0; s < 4; ++s)
    ad.woff[s] = ((uint32_t)(4 * g + s) * (uint32_t)A.d_out + (uint32_t)(j0 + CW * m)) * 4u;
  ad.aoff = ((uint32_t)m * KB + 4u * g) * 4u;
  ad.wblk = 16u * (uint32_t)A.d_out * 4u;
  ad.astride = 16u * KB * 4u;
  ad.nblk = (KB + 15u) / 16u;
  return ad;
}

template <int CW, int TF>
__device__ __forceinline__ void load_block_buf(const GemvAddr& ad, int blk,
                                               BlockCodes<CW, TF>& bc) {
  const uint32_t b = min((uint32_t)blk, ad.nblk);
  const uint32_t wb = b * ad.wblk, ab = b * 64u;
#pragma unroll
  for (int f = 0; f < TF; ++f)
    bc.av[f] = __builtin_bit_cast(uint4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                               ad.ra, (int)(ad.aoff + f * ad.astride + ab), 0, 0));
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int o = (int)(ad.woff[s] + wb);
    if constexpr (CW == 4) {
      const uint4_t v =
          __builtin_bit_cast(uint4_t, __builtin_amdgcn_raw_buffer_load_b128(ad.rw, o, 0, 0));
      bc.wv[s][0] = v[0]; bc.wv[s][1] = v[1]; bc.wv[s][2] = v[2]; bc.wv[s][3] = v[3];
    } else if constexpr (CW == 3) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b96(ad.rw, o, 0, 0);
      bc.wv[s][0] = v[0]; bc.wv[s][1 % CW] = v[1]; bc.wv[s][2 % CW] = v[2];
    } else if constexpr (CW == 2) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(ad.rw, o, 0, 0);
      bc.wv[s][0] = v[0]; bc.wv[s][CW - 1] = v[1];
    } else {
      bc.wv[s][0] = __builtin_amdgcn_raw_buffer_load_b32(ad.rw, o, 0, 0);
    }
  }
}

// Expand the codes of one block to fp16 centroid values and run its MFMAs:
// CW column tiles (tile c holds columns j0 + CW*m + c) by TF token tiles.
// Steps are taken SB at a time: all their table reads are issued before the
// first MFMA, so the LDS latency is paid once per batch.  Tokens past n read
// code words of zero (buffer loads past the end) and are expanded like the
// others: they only reach MFMA output columns that are never stored.  MASK
// zeroes the words past d_in of a partial last block.
template <int CW, int TF, bool MASK>
__device__ __forceinline__ void mma_block(int KB, int blk, const BlockCodes<CW, TF>& bc,
                                          const char* tab, uint32_t l4w, uint32_t l4a,
                                          float4_t (&acc)[CW][TF]) {
  constexpr int SB = CW * TF >= 4 ? 2 : 4;
  const int g = (threadIdx.x & 63) >> 4;
  const int kw0 = blk * 16 + 4 * g;
  const half8_t zero = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int s0 = 0; s0 < 4; s0 += SB) {
    half8_t af[SB][CW], bf[SB][TF];
#pragma unroll
    for (int s = 0; s < SB; ++s)
#pragma unroll
      for (int c = 0; c < CW; ++c) af[s][c] = expand_dual(bc.wv[s0 + s][c], tab, l4w);
#pragma unroll
    for (int f = 0; f < TF; ++f)
#pragma unroll
      for (int s = 0; s < SB; ++s) bf[s][f] = expand_dual(bc.av[f][s0 + s], tab, l4a);
    if constexpr (MASK) {  // words past the end contribute nothing
#pragma unroll
      for (int s = 0; s < SB; ++s)
        if (kw0 + s0 + s >= KB)
#pragma unroll
          for (int f = 0; f < TF; ++f) bf[s][f] = zero;
    }
#pragma unroll
    for (int s = 0; s < SB; ++s)
#pragma unroll
      for (int c = 0; c < CW; ++c)
#pragma unroll
        for (int f = 0; f < TF; ++f)
          acc[c][f] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[s][c], bf[s][f], acc[c][f], 0, 0, 0);
  }
}

// Blocks blk_begin, blk_begin + stride, ... < blk_end of one GEMV wave with
// PF blocks' codes in flight (buffer loads): after a block is expanded and
// multiplied its registers are refilled with the block PF strides ahead.
// `buf` holds the codes of the first PF blocks (loaded before the table was
// built).  The refills are unconditional (past the end they read zeros
// through the buffer descriptors): a conditional load would make the compiler
// count it as absent on one path and wait for every load before using a block.
template <int CW, int TF, int PF, bool FULLK>
__device__ __forceinline__ void gemv_blocks(int KB, const GemvAddr& ad, int blk_begin,
                                            int blk_end, int blk_stride,
                                            BlockCodes<CW, TF> (&buf)[PF], const char* tab,
                                            uint32_t l4w, uint32_t l4a, float4_t (&acc)[CW][TF]) {
  if (blk_end <= blk_begin + PF * blk_stride) {  // the preloaded blocks are all: no refills
#pragma unroll
    for (int d = 0; d < PF; ++d)
      if (blk_begin + d * blk_stride < blk_end)
        mma_block<CW, TF, !FULLK>(KB, blk_begin + d * blk_stride, buf[d], tab, l4w, l4a, acc);
    return;
  }
  for (int blk = blk_begin; blk < blk_end; blk += PF * blk_stride) {
#pragma unroll
    for (int d = 0; d < PF; ++d) {
      const int b = blk + d * blk_stride;
      if (b < blk_end) {
        mma_block<CW, TF, !FULLK>(KB, b, buf[d], tab, l4w, l4a, acc);
        load_block_buf<CW, TF>(ad, b + PF * blk_stride, buf[d]);
      }
    }
  }
}

// Output of tile (c, f): lane (g, tc) holds rows m = 4g + r, i.e. output
// column j0 + CW*(4g + r) + c of token tok0 + 16f + tc.
__device__ __forceinline__ void store_out(const GemmArgs& A, int tok, int j, float v) {
  if (tok >= A.n || j >= A.d_out) return;
  float* dst = A.y + (size_t)tok * A.d_out + j;
  const float val = A.act_scale[tok] * A.w_scale[j] * v;
  if (A.accumulate)
    *dst += val;
  else
    *dst = val;
}

// Outlier compensation of one column tile (fused variant).  Every listed
// outlier (token i, channel p, residual r) reads the words of input channel p
// for the tile's columns - rows this workgroup streams, so mostly L2 hits -
// and adds r * C_W[code] per column.  Thread t owns token t / T (T = threads
// per token), four consecutive columns and a slice of the token's entries; B
// entries' row loads are issued before any is used.  With PRE the first B
// entries of the slice come preloaded (`first`).
template <int B>
struct CompEntries {
  int p[B];
  float r[B];
};

// All B entries are requested before any is checked: a check placed next to
// its load makes the compiler wait for that load, and then only two or three
// entries are in flight whatever B is.
template <int B>
__device__ __forceinline__ void comp_entries(const GemmArgs& A, int i, int e0, int nslices,
                                             CompEntries<B>& ce) {
  const int k = A.k, E = 2 * k;
  const float* res = A.residual + (size_t)i * E;
  const int32_t* mx = A.max_idx + (size_t)i * k;
  const int32_t* mn = A.min_idx + (size_t)i * k;
  int praw[B];
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const int e = min(e0 + b * nslices, E - 1);
    praw[b] = e < k ? mx[e] : mn[e - k];
    ce.r[b] = res[e];
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const bool live = e0 + b * nslices < E;
    ce.p[b] = live && praw[b] >= 0 && praw[b] < A.d_in ? praw[b] : -1;
  }
}

// Row words of the tile's columns for B entries (buffer loads; entries with
// p < 0 get an offset past the buffer, which reads zeros without a memory
// access, and a zero residual).
template <int B>
__device__ __forceinline__ void comp_rows(const GemmArgs& A, const GemvAddr& ad, uint32_t col4,
                                          const CompEntries<B>& ce, uint4_t (&w)[B]) {
  const uint32_t d_out = (uint32_t)A.d_out;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const uint32_t o = ce.p[b] >= 0 ? ((uint32_t)ce.p[b] >> 3) * d_out * 4u + col4 : 0xFFFFFFF0u;
    w[b] = __builtin_bit_cast(uint4_t, __builtin_amdgcn_raw_buffer_load_b128(ad.rw, (int)o, 0, 0));
  }
}

// PERCOL: the weight half of row `code` holds two copies of each tile
// column's own pair(C_W[j], code) (position 2 * column + copy), so column jl
// reads position 2 jl + (slice & 1) there.
template <int COLS, int B, bool PRE, bool PERCOL = false>
__device__ __forceinline__ void tile_compensation(const GemmArgs& A, const GemvAddr& ad, uint32_t col4,
                                                  const char* tab, int nslices, int i, int slice,
                                                  const CompEntries<B>& first,
                                                  const uint4_t (&first_rows)[B], float (&acc)[4],
                                                  uint32_t jl0 = 0) {
  const int E = 2 * A.k;
  uint32_t l4c[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
    l4c[c] = PERCOL ? ((jl0 + (uint32_t)c) * 2u + ((uint32_t)slice & 1u)) * 4u
                    : (uint32_t)(threadIdx.x & 31) * 4u;
  for (int e0 = slice; e0 < E; e0 += B * nslices) {
    CompEntries<B> ce;
    uint4_t w[B];
    if (PRE && e0 == slice) {
      ce = first;
#pragma unroll
      for (int b = 0; b < B; ++b) w[b] = first_rows[b];
    } else {
      comp_entries<B>(A, i, e0, nslices, ce);
      comp_rows<B>(A, ad, col4, ce, w);
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const uint32_t sh = ce.p[b] >= 0 ? 4u * ((uint32_t)ce.p[b] & 7u) : 0u;
      const float r = ce.p[b] >= 0 ? ce.r[b] : 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] += r * weight_centroid(tab, (w[b][c] >> sh) & 15u, l4c[c]);
    }
  }
}

// The same from the row layout: thread owns 8 consecutive columns (one word
// of each row), so an entry costs one 4-byte load, four pair lookups in the
// weight half of the decode table (row `byte` holds pair(C_W, byte)) and
// eight FMAs.
template <int B>
__device__ __forceinline__ void comp_rows_wr(__amdgpu_buffer_rsrc_t rwr, uint32_t row_bytes,
                                             uint32_t woff, const CompEntries<B>& ce,
                                             uint32_t (&w)[B]) {
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const uint32_t o = ce.p[b] >= 0 ? (uint32_t)ce.p[b] * row_bytes + woff : 0xFFFFFFF0u;
    w[b] = __builtin_amdgcn_raw_buffer_load_b32(rwr, (int)o, 0, 0);
  }
}

template <int B, bool PRE>
__device__ __forceinline__ void tile_compensation_wr(const GemmArgs& A,
                                                     __amdgpu_buffer_rsrc_t rwr,
                                                     uint32_t row_bytes, uint32_t woff,
                                                     const char* tab, int nslices, int i,
                                                     int slice, const CompEntries<B>& first,
                                                     const uint32_t (&first_rows)[B],
                                                     float (&acc)[8]) {
  const int E = 2 * A.k;
  const uint32_t l4 = (uint32_t)(threadIdx.x & 31) * 4u;
  for (int e0 = slice; e0 < E; e0 += B * nslices) {
    CompEntries<B> ce;
    uint32_t w[B];
    if (PRE && e0 == slice) {
      ce = first;
#pragma unroll
      for (int b = 0; b < B; ++b) w[b] = first_rows[b];
    } else {
      comp_entries<B>(A, i, e0, nslices, ce);
      comp_rows_wr<B>(rwr, row_bytes, woff, ce, w);
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const float r = ce.p[b] >= 0 ? ce.r[b] : 0.0f;
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const uint32_t off = __builtin_amdgcn_perm(w[b], l4, 0x0C0C0000u | ((4u + bb) << 8));
        const uint32_t pr = *reinterpret_cast<const uint32_t*>(tab + off);
        acc[2 * bb] = fmaf(r, h2f((uint16_t)(pr & 0xFFFFu)), acc[2 * bb]);
        acc[2 * bb + 1] = fmaf(r, h2f((uint16_t)(pr >> 16)), acc[2 * bb + 1]);
      }
    }
  }
}

// ----------------------------------------------------------------------------
// MFMA kernel, few tokens (GEMV-like): one workgroup per 16*CW output
// columns, its NW waves interleave the K blocks and are summed through LDS,
// so every output is written once, without atomics.  With outlier lists
// (B > 0, k > 0) the workgroup also adds the compensation of its columns; each
// wave starts its share as soon as its own blocks are done.
//
// Prologue: the scales and the first outlier entries, then the weight codes,
// then the codebooks (scalar loads, issued after the vector loads so that no
// wait for them delays the weight stream); building the table waits only for
// the codebooks, and the entries are checked after the table barrier, behind
// the weight loads in flight.
// ----------------------------------------------------------------------------
// One column tile (columns j0 .. j0 + 16 CW - 1) of the few-token kernels;
// `tab` is the workgroup's 64 KiB decode table, reused for the reduction.
template <int CW, int TF, int NW, int PF, bool FULLK, int B, bool ROWS, bool PERCOL>
__device__ __forceinline__ void gemv_tile(const GemmArgs& A, const int j0, uint32_t* tab) {
  static_assert(!PERCOL || (CW == 1 && !ROWS), "per-column codebooks: 16-column tiles, GEMM layout");
  constexpr int NT = NW * 64;
  constexpr int SLOTS = 16 * TF, COLS = 16 * CW;
  constexpr int CG = ROWS ? 8 : 4;  // columns per compensation thread
  constexpr int GROUPS = COLS / CG;  // compensation threads per token and slice
  static_assert(NT / SLOTS >= GROUPS, "a token's threads cover its columns");
  // threads per token NT / SLOTS: NSLICES * GROUPS of them compensate
  constexpr int NSLICES = (NT / SLOTS) / GROUPS;
  constexpr int RED_FLOATS = 4 * NW * CW * TF * 64;
  constexpr int PART_FLOATS = SLOTS * NSLICES * COLS;
  static_assert(4 * (RED_FLOATS + PART_FLOATS) <= 64 * 1024, "reduction buffers fit in the table");
  constexpr int EPT = (SLOTS * COLS + NT - 1) / NT;  // outputs per thread in the epilogue
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  const int KB = A.d_in >> 3;
  const int nblk = (KB + 15) / 16;
  constexpr bool fused = B > 0;  // B = 0: no outlier lists (k = 0)
  constexpr int BE = B > 0 ? B : 1;

  // ---- prologue: codebooks (scalar loads), scales, outlier entries, weight
  // codes.  Without outlier lists every kernel argument the vector loads need
  // is made resident in SGPRs first (the empty asm, on which the codebook
  // address depends): a scalar-load wait cannot single out one load, so none
  // is fetched after the codebook loads and no weight load waits for them;
  // the weight loads are unconditional (a block past the end reads zeros), so
  // the wait before each block covers that block only.  With lists the
  // entries are loaded and checked first and only the blocks that exist are
  // requested: measured, that order is the faster one there (the list wait
  // is short, and the row words that follow would otherwise queue behind
  // the whole weight stream).
  const GemvAddr ad = gemv_addr<CW>(A, j0);
  const oasis_lut_block* lutp = A.lut;
  if constexpr (!fused)
    asm("" : "+s"(lutp)
        : "s"(A.idx_w), "s"(A.idx_act), "s"(A.w_scale), "s"(A.act_scale), "s"(A.n),
          "s"(A.d_in), "s"(A.d_out));
  DualTableLoader dt;
  if (wave < 4) dt.load(lutp, (uint32_t)wave);
  if constexpr (!fused) __builtin_amdgcn_sched_barrier(0);
  // per-column codebooks: thread t writes position t % 32 (tile column
  // (t % 32) / 2, copy t % 2) of rows t / 32 + 32 i (i < 8) of the weight half,
  // i.e. low code (t / 32) % 16 and high codes t / 512 + 2 i of that column
  static_assert(!PERCOL || NT == 1024, "the per-column table takes 8 entries per thread");
  // (the column's 32-byte codebook in two 16-byte loads; t / 512 is
  // wave-uniform, so the high codes are one half of every word)
  uint32_t pc_lo = 0, pc_hi[8];
  if constexpr (PERCOL) {
    const int col = min(j0 + (tid & 31) / 2, A.d_out - 1);
    const uint4_t* cb = reinterpret_cast<const uint4_t*>(A.cb_cols + (size_t)col * 16);
    const uint4_t c0 = cb[0], c1 = cb[1];
    const uint32_t cw[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
    const uint32_t e = ((uint32_t)tid >> 5) & 15u, hs = 16u * ((uint32_t)tid >> 9);
    uint32_t d = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) d = (e >> 1) == (uint32_t)q ? cw[q] : d;
    pc_lo = (d >> (16u * (e & 1u))) & 0xFFFFu;
#pragma unroll
    for (int i = 0; i < 8; ++i) pc_hi[i] = (cw[i] >> hs) & 0xFFFFu;
  }
  float ts[EPT];   // t_i of this thread's epilogue outputs
  float swj[EPT];  // s_j of the same
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int o = tid + NT * q;
    const int tok = min(o / COLS, A.n - 1), j = min(j0 + o % COLS, A.d_out - 1);
    swj[q] = A.w_scale[j];
    ts[q] = A.act_scale[tok];
  }
  const int T = NT / SLOTS;  // threads per token
  const int ci = tid / T, cu = tid - ci * T;
  const int cquad = cu % GROUPS, cslice = cu / GROUPS;  // column group, slice
  const bool cact = cslice < NSLICES;  // a compensating thread
  // a few entries are worth holding through the main loop, many are not
  constexpr bool PRE = fused && B <= 4 && TF == 1 && CW <= 2;
  CompEntries<BE> ce0;
  if (PRE && cact && ci < A.n) comp_entries<BE>(A, ci, cslice, NSLICES, ce0);
  BlockCodes<CW, TF> buf[PF];
#pragma unroll
  for (int d = 0; d < PF; ++d)
    if (!fused || PERCOL || wave + d * NW < nblk) load_block_buf<CW, TF>(ad, wave + d * NW, buf[d]);
  if constexpr (!fused) __builtin_amdgcn_sched_barrier(0);
  if (wave < 4) dt.store<PERCOL>(tab, (uint32_t)wave, lane);
  if constexpr (PERCOL) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      tab[(((uint32_t)tid >> 5) + 32u * (uint32_t)i) * 64u + ((uint32_t)tid & 31u)] =
          pc_lo | (pc_hi[i] << 16);
  }
  __syncthreads();  // decode table

  float4_t acc[CW][TF];
#pragma unroll
  for (int c = 0; c < CW; ++c)
#pragma unroll
    for (int f = 0; f < TF; ++f) acc[c][f] = float4_t{0.f, 0.f, 0.f, 0.f};
  const char* tb = reinterpret_cast<const char*>(tab);
  // weight entries: copy lane mod 32 of the shared codebook, or (per column)
  // position 2 m + (g mod 2) of lane (g, m)'s column m
  const uint32_t l4a = (uint32_t)(lane & 31) * 4u + 128u;
  const uint32_t l4w = PERCOL ? ((uint32_t)(lane & 15) * 2u + ((uint32_t)(lane >> 4) & 1u)) * 4u
                              : (uint32_t)(lane & 31) * 4u;
  // the preloaded entries' row words, in flight during the main loop
  const uint32_t ccol4 = (uint32_t)(j0 + CG * cquad) * 4u;
  // row layout: word (j0 + 8 cquad) / 8 of each row
  const uint32_t wr_row = (uint32_t)((A.d_out + 7) / 8) * 4u;
  const uint32_t wr_off = (uint32_t)(j0 / 8 + cquad) * 4u;
  __amdgpu_buffer_rsrc_t rwr = ad.rw;
  if constexpr (ROWS)
    rwr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(A.idx_wr), 0,
                                            (int)((uint32_t)A.d_in * wr_row), 0x00020000);
  uint4_t crow0[ROWS ? 1 : BE];
  uint32_t crw0[ROWS ? BE : 1];
  if (PRE && cact && ci < A.n) {
    if constexpr (ROWS) comp_rows_wr<BE>(rwr, wr_row, wr_off, ce0, crw0);
    else comp_rows<BE>(A, ad, ccol4, ce0, crow0);
  }
  if (wave < nblk)
    gemv_blocks<CW, TF, PF, FULLK>(KB, ad, wave, nblk, NW, buf, tb, l4w, l4a, acc);

  // outlier branch: reads only rows 0..15 of the table (weight centroids),
  // which nothing overwrites before the next barrier
  float cacc[CG];
#pragma unroll
  for (int c = 0; c < CG; ++c) cacc[c] = 0.0f;
  if (fused && cact && ci < A.n) {
    if constexpr (ROWS)
      tile_compensation_wr<BE, PRE>(A, rwr, wr_row, wr_off, tb, NSLICES, ci, cslice, ce0, crw0,
                                   cacc);
    else
      tile_compensation<COLS, BE, PRE, PERCOL>(A, ad, ccol4, tb, NSLICES, ci, cslice, ce0, crow0,
                                               cacc, (uint32_t)(CG * cquad));
  }
  __syncthreads();  // every wave is done with the table: reuse it for the reduction
  float4_t (*red)[CW * TF][64] = reinterpret_cast<float4_t (*)[CW * TF][64]>(tab);
  float* part = reinterpret_cast<float*>(tab) + RED_FLOATS;  // compensation partials
#pragma unroll
  for (int c = 0; c < CW; ++c)
#pragma unroll
    for (int f = 0; f < TF; ++f) red[wave][c * TF + f][lane] = acc[c][f];
  if (fused && cact && ci < SLOTS) {
#pragma unroll
    for (int c = 0; c < CG; ++c) part[(ci * NSLICES + cslice) * COLS + CG * cquad + c] = cacc[c];
  }
  __syncthreads();

  // ---- epilogue: thread -> output (token o / COLS, column j0 + o % COLS)
  const float* redf = reinterpret_cast<const float*>(tab);
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int o = tid + NT * q;
    const int tok = o / COLS, jl = o % COLS;
    const int j = j0 + jl;
    if (o >= SLOTS * COLS || tok >= A.n || j >= A.d_out) continue;
    const int c = jl % CW, mrow = jl / CW;
    const int t = c * TF + (tok >> 4);
    const int ln = (mrow >> 2) * 16 + (tok & 15);
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) v += redf[((w * CW * TF + t) * 64 + ln) * 4 + (mrow & 3)];
    float val = ts[q] * swj[q] * v;
    if (fused) {
      float cs = 0.0f;
      for (int sl = 0; sl < NSLICES; ++sl) cs += part[(tok * NSLICES + sl) * COLS + jl];
      val += swj[q] * cs;
    }
    float* dst = A.y + (size_t)tok * A.d_out + j;
    *dst = A.accumulate ? *dst + val : val;
  }
}

template <int CW, int TF, int NW, int PF, bool FULLK, int B, bool ROWS, bool PERCOL = false>
__global__ void __launch_bounds__(NW * 64) k_gemm_mfma_gemv(GemmArgs A, int ntiles) {
  __shared__ uint32_t tab[256 * 64];  // 64 KiB decode table; after the main loop the reduction
  gemv_tile<CW, TF, NW, PF, FULLK, B, ROWS, PERCOL>(A, xcd_tile(blockIdx.x, ntiles) * 16 * CW,
                                                    tab);
}

// Two tile widths in one launch, so that the columns spread evenly over the
// CUs: the first na workgroups (one per CU) take 16*CWA columns each, the
// other nb take 16*CWB.  Workgroups start in id order and the first na fill
// every CU once, so each CU ends up with one tile of each width (at 28672
// columns: 64 + 48 per CU instead of two 64-column tiles on 192 CUs).
template <int CWA, int CWB, int NW, int PF, bool FULLK, int B, bool ROWS>
__global__ void __launch_bounds__(NW * 64) k_gemm_mfma_gemv2(GemmArgs A, int na, int nb) {
  __shared__ uint32_t tab[256 * 64];
  const int b = blockIdx.x;
  if (b < na)
    gemv_tile<CWA, 1, NW, PF, FULLK, B, ROWS, false>(A, xcd_tile(b, na) * 16 * CWA, tab);
  else
    gemv_tile<CWB, 1, NW, PF, FULLK, B, ROWS, false>(
        A, na * 16 * CWA + xcd_tile(b - na, nb) * 16 * CWB, tab);
}

// ----------------------------------------------------------------------------
// MFMA kernel, prefill tiling: WX x WY waves, each 16*CW columns x 16*TF
// tokens over the whole reduction; tiles ordered column-major over the XCDs
// so that one XCD's L2 holds few weight columns.
//
// Both pair tables share one 64 KiB region: row `byte` (256 bytes) holds 32
// copies of the weight entry, then 32 of the activation entry, so the byte
// offset of either is byte * 256 + (lane mod 32) * 4 (+ 128 for activations)
// - one v_perm_b32 per byte, and 32 lanes read 32 different banks.
// ----------------------------------------------------------------------------

// Per-lane byte offsets of the codes of one wave (block 0); a block's offset
// is added to them (the descriptor's size check covers the whole offset), so
// reads past either tensor return 0.  Weight lane m of
// column tile c holds column j0 + 16c + m, so the MFMA's output rows 4g..4g+3
// are 4 consecutive columns: each lane stores 16 contiguous bytes.
template <int CW, int TF>
struct PrefillAddr {
  __amdgpu_buffer_rsrc_t rw, ra;
  uint32_t woff[4];   // row 4g + s, column j0 + m (tile c: + 64c bytes)
  uint32_t aoff[TF];  // token tok0 + 16f + m, word 4g
  uint32_t wblk;      // bytes per block of 16 weight rows
};

template <int CW, int TF>
__device__ __forceinline__ void load_block_pf(const PrefillAddr<CW, TF>& ad, int blk,
                                              BlockCodes<CW, TF>& bc) {
  const uint32_t wb = (uint32_t)blk * ad.wblk, ab = (uint32_t)blk * 64u;
#pragma unroll
  for (int f = 0; f < TF; ++f)
    bc.av[f] = __builtin_bit_cast(
        uint4_t, __builtin_amdgcn_raw_buffer_load_b128(ad.ra, (int)(ad.aoff[f] + ab), 0, 0));
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int c = 0; c < CW; ++c)
      bc.wv[s][c] =
          __builtin_amdgcn_raw_buffer_load_b32(ad.rw, (int)(ad.woff[s] + wb + 64u * c), 0, 0);
}

// KMASK: zero the activation operand of words past the end of the reduction
// (only the last block can hold them; they would read the next token's codes).
template <int CW, int TF, bool KMASK>
__device__ __forceinline__ void mma_block_pf(int blk, int KB, const BlockCodes<CW, TF>& bc,
                                             const char* tab, uint32_t l4w, uint32_t l4a,
                                             float4_t (&acc)[CW][TF]) {
  const int g = (threadIdx.x & 63) >> 4;
  const int kw0 = blk * 16 + 4 * g;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    half8_t bf[TF];
#pragma unroll
    for (int f = 0; f < TF; ++f) {
      bf[f] = expand_dual(bc.av[f][s], tab, l4a);
      if (KMASK && kw0 + s >= KB) bf[f] = half8_t{0, 0, 0, 0, 0, 0, 0, 0};
    }
#pragma unroll
    for (int c = 0; c < CW; ++c) {
      const half8_t af = expand_dual(bc.wv[s][c], tab, l4w);
#pragma unroll
      for (int f = 0; f < TF; ++f)
        acc[c][f] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf[f], acc[c][f], 0, 0, 0);
    }
  }
}

template <int CW, int TF, int WX, int WY, bool FULLK>
__global__ void __launch_bounds__(WX * WY * 64) k_gemm_mfma_prefill(GemmArgs A, int ncx, int nty) {
  constexpr int NT = WX * WY * 64;
  __shared__ uint32_t tab[256 * 64];  // 64 KiB dual decode table
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, m = lane & 15;

  const int r = xcd_tile(blockIdx.x, ncx * nty);
  const int cx = r / nty, ty = r % nty;
  const int j0 = (cx * WX + wave % WX) * 16 * CW;
  const int tok0 = (ty * WY + wave / WX) * 16 * TF;
  const int KB = A.d_in >> 3;
  const int nblk = (KB + 15) / 16;

  PrefillAddr<CW, TF> ad;
  ad.rw = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(A.idx_w), 0,
                                            (int)((uint32_t)KB * (uint32_t)A.d_out * 4u), 0x00020000);
  ad.ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(A.idx_act), 0,
                                            (int)((uint32_t)A.n * (uint32_t)KB * 4u), 0x00020000);
#pragma unroll
  for (int s = 0; s < 4; ++s)
    ad.woff[s] = ((uint32_t)(4 * g + s) * (uint32_t)A.d_out + (uint32_t)(j0 + m)) * 4u;
#pragma unroll
  for (int f = 0; f < TF; ++f)
    ad.aoff[f] = ((uint32_t)(tok0 + 16 * f + m) * (uint32_t)KB + 4u * g) * 4u;
  ad.wblk = 16u * (uint32_t)A.d_out * 4u;

  // codebooks (scalar loads), then the first block's codes
  DualTableLoader dt;
  const uint32_t uwave = (uint32_t)__builtin_amdgcn_readfirstlane(wave);
  if (uwave < 4) dt.load(A.lut, uwave);
  BlockCodes<CW, TF> buf[2];
  load_block_pf<CW, TF>(ad, 0, buf[0]);
  if (uwave < 4) dt.store(tab, uwave, lane);
  __syncthreads();

  float4_t acc[CW][TF];
#pragma unroll
  for (int c = 0; c < CW; ++c)
#pragma unroll
    for (int f = 0; f < TF; ++f) acc[c][f] = float4_t{0.f, 0.f, 0.f, 0.f};

  const char* tb = reinterpret_cast<const char*>(tab);
  const uint32_t l4w = (uint32_t)(lane & 31) * 4u, l4a = l4w + 128u;
  // full blocks; a partial last block (FULLK false) is peeled off and masked
  const int nfull = FULLK ? nblk : nblk - 1;
  for (int blk = 0; blk < nfull; blk += 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const int b = blk + d;
      if (b < nfull) {
        if (b + 1 < nblk) load_block_pf<CW, TF>(ad, b + 1, buf[d ^ 1]);
        mma_block_pf<CW, TF, false>(b, KB, buf[d], tb, l4w, l4a, acc);
      }
    }
  }
  if constexpr (!FULLK) {
    if (nfull & 1)
      mma_block_pf<CW, TF, true>(nfull, KB, buf[1], tb, l4w, l4a, acc);
    else
      mma_block_pf<CW, TF, true>(nfull, KB, buf[0], tb, l4w, l4a, acc);
  }

  // lane (g, tc) of tile (c, f): token tok0 + 16f + tc, columns
  // j0 + 16c + 4g .. + 3
  const int tc = lane & 15;
  // 16-byte loads and stores only where y and the scales allow them (the
  // boundary promises 4-byte alignment)
  const bool vec = (A.d_out & 3) == 0 && (reinterpret_cast<uintptr_t>(A.y) & 15u) == 0 &&
                   (reinterpret_cast<uintptr_t>(A.w_scale) & 15u) == 0;
#pragma unroll
  for (int c = 0; c < CW; ++c) {
    const int j = j0 + 16 * c + 4 * g;
    if (vec && j + 3 < A.d_out) {
      const float4_t sw = *reinterpret_cast<const float4_t*>(A.w_scale + j);
#pragma unroll
      for (int f = 0; f < TF; ++f) {
        const int tok = tok0 + 16 * f + tc;
        if (tok >= A.n) continue;
        float4_t* dst = reinterpret_cast<float4_t*>(A.y + (size_t)tok * A.d_out + j);
        const float4_t v = A.act_scale[tok] * sw * acc[c][f];
        *dst = A.accumulate ? *dst + v : v;
      }
    } else {
#pragma unroll
      for (int f = 0; f < TF; ++f)
#pragma unroll
        for (int q = 0; q < 4; ++q) store_out(A, tok0 + 16 * f + tc, j + q, acc[c][f][q]);
    }
  }
}

// ----------------------------------------------------------------------------
// MFMA kernel, many tokens: v_mfma_f32_32x32x16_f16 (A = weights, 32 output
// columns; B = activations, 32 tokens; 16 channels), every wave expanding its
// own operands from the codes through the dual table.
//
// A wave owns 32*CW columns x 32*FT tokens (CW * FT accumulator tiles of 16
// registers); WX x WY waves form the workgroup tile.  An expanded operand
// (32 rows x 16 channels, 1 KiB, four ds_read_b32 per lane) feeds CW or FT
// MFMAs, so the LDS traffic per MFMA is 1 KiB * (1/CW + 1/FT): with 4 x 2
// that is 3/4 of what the LDS delivers (128 B/clk per CU for these reads)
// while the matrix cores run at their peak (one 32x32x16 MFMA per 8 clk per
// CU), with 4 x 4 one half.
//
// Channel order inside the MFMA: lane (r, h) (r = lane mod 32, h = lane / 32)
// of step s (0..3) takes word 4h + s of a block of 8 words (64 channels) on
// both operands; a token's four words of one lane are one 16-byte load, a
// weight word one 4-byte load (32 lanes: 128 contiguous bytes of a row).
//
// Output: lane (r, h), register v of tile (c, f) holds column
// j0 + 32 c + 8 (v / 4) + 4 h + (v mod 4) of token t0 + 32 f + r.
// ----------------------------------------------------------------------------
typedef float float16_t __attribute__((ext_vector_type(16)));

// Tile t of ncx x nty (column x token tiles) in groups of kTileGroup token
// tiles: inside a group the token tile runs fastest, then the column tile.
// The tiles an XCD holds at once (consecutive ones, see xcd_tile) then span
// a few column and a few token tiles: at 4096 x 8192 x 28672 one round of an
// XCD read 16 token tiles' activation codes and 2 column tiles' weight codes
// with the token tile fastest over all 16, 8 and 4 in groups of 8 (12 MB
// instead of 18 MB of operands per round and XCD).
constexpr int kTileGroup = 8;
__device__ __forceinline__ void tile_xy(int t, int ncx, int nty, int& cx, int& ty) {
  const int gb = t / (kTileGroup * ncx) * kTileGroup;  // the group's first token tile
  const int gt = min(kTileGroup, nty - gb);              // its token tiles
  const int r = t - gb * ncx;
  cx = r / gt;
  ty = gb + r % gt;
}

// BV: the B operand is an fp16 value matrix (GemmArgs::kdyn), one 16-byte load
// per lane, step and token group, instead of activation codes.
template <int CW, int FT, bool BV>
struct TileCodes {
  uint32_t w[4][CW];        // weight word 4h + s of column group c
  uint4_t a[BV ? 4 : 1][FT];  // codes: words 4h .. 4h + 3 of token group f;
                              // values: positions 8 (4h + s) .. + 7 of step s
};

// HV: after the codes, the blocks of the value operand A.hv with the codes
// A.hw (the heavy channels of the split compensation).
//
// Persistent: workgroup b takes tiles b, b + G, b + 2G, ... (G = gridDim.x,
// at most what the CUs hold at once).  The decode table is built once; the
// codes of a workgroup's next tile are requested right after the current
// tile's stores.  Requested before them, they were live through the
// epilogue, where the compiler then kept about twice as many values in
// scratch, and every reload there waited for those loads (the heavy-block
// GEMM at 4096 x 8192 x 28672: 1733 -> 1648 us with them moved).  The tile's
// scales are requested at its start and kept in registers (the column
// scales pass through a 512-byte LDS row per wave in the epilogue).
//
// QL (one workgroup per CU, d_in a multiple of 512): the activation codes
// pass through LDS.  A token's codes for 4 blocks are 128 contiguous bytes;
// loaded straight into LDS (buffer_load_dwordx4 ... lds, full 128-byte
// pieces of 8 rows per instruction) they cost a quarter of the L2 requests
// of per-lane 16-byte loads, which touch 32 rows x 32 bytes each.  Two
// buffers of 4 blocks (quads) per token group; the waves of a group each
// load half of its rows, so one barrier per quad publishes a quad (after
// each wave's own wait for its copies).  16-byte chunk c of row R sits at
// chunk c ^ ((R >> 1) & 7): the 16 lanes of a ds_read_b128 then hit 16
// distinct bank groups.  With the activation words read from LDS one block
// ahead, the weight words are requested three blocks ahead (four slots):
// with one block of lead the table lookups waited for them (a variant whose
// lookups did not depend on the loaded words ran 15 % faster).
template <int CW, int FT, int WX, int WY, bool BV, bool HV = false, bool QL = false>
__global__ void __launch_bounds__(WX * WY * 64, (CW * FT > 8 || BV || WX * WY > 4 ? 1 : 2))
    k_gemm_mfma_tile(GemmArgs A, int ncx, int nty) {
  static_assert(CW == 4, "the column scales of a wave are two per lane");
  static_assert(!QL || (!BV && WX == 2 && (FT == 4 || FT == 2)), "quad staging: 2 loaders a group");
  __shared__ uint32_t tab[256 * 64];          // 64 KiB dual decode table
  __shared__ float wsc[WX * WY][32 * CW];     // column scales of each wave's tile
  constexpr int QB = QL ? WY * 32 * FT * 128 : 16;  // bytes of one quad buffer
  __shared__ __align__(16) unsigned char actq0[QB], actq1[QB];
  const char* tb = reinterpret_cast<const char*>(tab);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31, h = lane >> 5;
  const int T = ncx * nty;

  const uint32_t KB = (uint32_t)(A.d_in >> 3);  // words per token row = weight rows
  // blocks of 8 words (64 channels); with a value operand, of 64 positions up
  // to the device-side length
  const int nblk = BV ? (2 * __builtin_amdgcn_readfirstlane(*A.kdyn) + 63) / 64 : (int)(KB >> 3);
  const uint32_t arow = BV ? (uint32_t)A.a_row : KB * 4u;  // bytes per token row
  const uint32_t d_out = (uint32_t)A.d_out;

  // The blocks past the last one are requested too (every refill is
  // unconditional) and read zeros (see load_from); columns and tokens past
  // the end are clamped to the last one (their outputs are never stored).
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(A.idx_w), 0, (int)(KB * d_out * 4u), 0x00020000);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(A.idx_act), 0, (int)((uint32_t)A.n * arow), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(A.w_scale), 0, (int)(d_out * 4u), 0x00020000);
  const __amdgpu_buffer_rsrc_t rst = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(A.act_scale), 0, (int)((uint32_t)A.n * 4u), 0x00020000);
  int j0 = 0, t0 = 0;
  uint32_t woff[CW], aoff[FT];
  // QL: byte offsets of this lane's 16-byte pieces of the quad copies (8 per
  // wave: rows 64 gx + 8 i + lane / 8 of the group), for this tile and the
  // workgroup's next one
  constexpr int RPW = 32 * FT / WX;              // rows of a group each of its waves copies
  constexpr int NDMA = QL ? RPW / 8 : 1;
  uint32_t dcur[NDMA], dnext[NDMA];
  auto dma_offsets = [&](int u, uint32_t (&d)[NDMA]) {
    if constexpr (QL) {
      int cx, ty;
      tile_xy(xcd_tile(min(u, T - 1), T), ncx, nty, cx, ty);
      const int tg = (ty * WY + wave / WX) * 32 * FT;
#pragma unroll
      for (int i = 0; i < NDMA; ++i) {
        const int R = RPW * (wave % WX) + 8 * i + (lane >> 3);
        const uint32_t c = (uint32_t)(lane & 7) ^ (uint32_t)((R >> 1) & 7);
        d[i] = (uint32_t)min(tg + R, A.n - 1) * arow + 16u * c;
      }
    }
  };
  // origin and per-lane code offsets of tile u
  auto place = [&](int u) {
    int cx, ty;
    tile_xy(xcd_tile(u, T), ncx, nty, cx, ty);
    j0 = (cx * WX + wave % WX) * 32 * CW;
    t0 = (ty * WY + wave / WX) * 32 * FT;
#pragma unroll
    for (int c = 0; c < CW; ++c)
      woff[c] = ((uint32_t)(4 * h) * d_out + (uint32_t)min(j0 + 32 * c + r32, A.d_out - 1)) * 4u;
#pragma unroll
    for (int f = 0; f < FT; ++f)
      aoff[f] = (uint32_t)min(t0 + 32 * f + r32, A.n - 1) * arow + (BV ? 64u : 16u) * (uint32_t)h;
    dma_offsets(u, dcur);
    dma_offsets(u + (int)gridDim.x, dnext);
  };
  const uint32_t wrow = d_out * 4u, wblk = 8u * d_out * 4u;

  // Code and value loads take the per-lane part of the offset in the VGPR
  // and the block's uniform part in soffset (no VALU add per load: two per
  // load were an eighth of the main loop's VALU instructions).  A block past
  // the tensor's last (index bl), which the loops request but never
  // multiply, goes through rz, a descriptor of size 0, at soffset 0: it
  // returns zeros without touching memory, whatever part of the offset the
  // range check covers.
  const __amdgpu_buffer_rsrc_t rz = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(A.idx_w), 0, 0, 0x00020000);
  auto sblk = [](int blk, int bl) { return blk <= bl ? (uint32_t)max(0, blk) : 0u; };
  // codes (or values) of block blk from the descriptors rwx / rax at the
  // per-lane offsets aoffx; the type of tc says which operand B is
  auto load_from = [&](int blk, int bl, auto& tc, __amdgpu_buffer_rsrc_t rwx,
                       __amdgpu_buffer_rsrc_t rax, const uint32_t (&aoffx)[FT]) {
    constexpr bool VALS = sizeof(tc.a) / sizeof(tc.a[0]) == 4;
    const uint32_t bc = sblk(blk, bl);
    if (blk > bl) rwx = rax = rz;
#pragma unroll
    for (int f = 0; f < FT; ++f) {
      if constexpr (VALS) {
#pragma unroll
        for (int st = 0; st < 4; ++st)
          tc.a[st][f] = __builtin_bit_cast(
              uint4_t, __builtin_amdgcn_raw_buffer_load_b128(
                           rax, (int)aoffx[f], (int)(bc * 128u + 16u * (uint32_t)st), 0));
      } else {
        tc.a[0][f] = __builtin_bit_cast(uint4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                     rax, (int)aoffx[f], (int)(bc * 32u), 0));
      }
    }
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int c = 0; c < CW; ++c)
        tc.w[st][c] = __builtin_amdgcn_raw_buffer_load_b32(
            rwx, (int)woff[c], (int)(bc * wblk + (uint32_t)st * wrow), 0);
  };
  auto load = [&](int blk, auto& tc) { load_from(blk, nblk - 1, tc, rw, ra, aoff); };
  // QL: copy a quad (8 pieces per lane, at offsets d + qoff; qoff uniform,
  // in soffset) into buffer q
  const uint32_t gbase = (uint32_t)(wave / WX) * (uint32_t)(32 * FT * 128);
  auto dma = [&](unsigned char* q, const uint32_t (&d)[NDMA], uint32_t qoff) {
    if constexpr (QL) {
#pragma unroll
      for (int i = 0; i < NDMA; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            ra, (__attribute__((address_space(3))) void*)(q + gbase + ((uint32_t)RPW * (uint32_t)(wave % WX) + 8u * (uint32_t)i) * 128u),
            16, (int)d[i], (int)qoff, 0, 0);
    }
  };
  // QL: lane (r, h) reads chunk 2 bq + h of rows 32 f + r of its group (aload4)
  const uint32_t xr = (uint32_t)((r32 >> 1) & 7);
  const uint32_t rbase = gbase + (uint32_t)r32 * 128u;
  // QL: wait for this wave's quad copy (issued four blocks of weight loads
  // ago; the last two blocks' 32 loads may stay in flight), then for every
  // wave's
  auto publish = [&]() {
    // s_waitcnt vmcnt(32): vmcnt bits [3:0] = 0 and [15:14] = 2, expcnt 7, lgkmcnt 15
    __builtin_amdgcn_s_waitcnt(0x8F70);
    __builtin_amdgcn_s_barrier();
  };
  struct WCodes {
    uint32_t w[4][CW];  // weight word 4h + s of column group c
  };
  struct ACodes {
    uint4_t a[FT];  // words 4h .. 4h + 3 of token group f
  };
  auto wload4 = [&](int blk, WCodes& wc) {
    const uint32_t sb = sblk(blk, nblk - 1) * wblk;
    const __amdgpu_buffer_rsrc_t rwb = blk < nblk ? rw : rz;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int c = 0; c < CW; ++c)
        wc.w[st][c] = __builtin_amdgcn_raw_buffer_load_b32(
            rwb, (int)woff[c], (int)(sb + (uint32_t)st * wrow), 0);
  };
  auto aload4 = [&](const unsigned char* q, int bq, ACodes& ac) {
    const uint32_t co = (((uint32_t)(2 * bq + h)) ^ xr) * 16u;
#pragma unroll
    for (int f = 0; f < FT; ++f)
      ac.a[f] = *reinterpret_cast<const uint4_t*>(q + rbase + co + 4096u * (uint32_t)f);
  };

  float16_t acc[CW][FT];
  const uint32_t l4w = (uint32_t)r32 * 4u, l4a = l4w + 128u;
  // operands of step st (every block is full: d_in is a multiple of 64)
  // The MFMAs of a step run token group by token group (all column groups
  // of b[0], then of b[1], ...), and the table reads of the next step are
  // issued in the order their MFMAs need them: a[0], b[0], a[1..], b[1..].
  // Each operand then has at least CW + FT + 1 MFMAs between its last read
  // and its first use (with a[] first and the MFMAs column by column, the
  // last-read b[] were needed within four MFMAs of the step start).
  auto operands = [&](const auto& tc, int st, half8_t (&a)[CW], half8_t (&b)[FT]) {
    constexpr bool VALS = sizeof(tc.a) / sizeof(tc.a[0]) == 4;
    auto bop = [&](int f) {
      if constexpr (VALS) b[f] = __builtin_bit_cast(half8_t, tc.a[st][f]);
      else b[f] = expand_dual(tc.a[0][f][st], tb, l4a);
    };
    a[0] = expand_dual(tc.w[st][0], tb, l4w);
    bop(0);
#pragma unroll
    for (int c = 1; c < CW; ++c) a[c] = expand_dual(tc.w[st][c], tb, l4w);
#pragma unroll
    for (int f = 1; f < FT; ++f) bop(f);
  };
  auto mma = [&](const half8_t (&a)[CW], const half8_t (&b)[FT]) {
#pragma unroll
    for (int f = 0; f < FT; ++f)
#pragma unroll
      for (int c = 0; c < CW; ++c)
        acc[c][f] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[c], b[f], acc[c][f], 0, 0, 0);
  };
  // Instruction order of one step: each MFMA keeps the matrix unit busy for
  // 32 cycles, and the wave issues in order, so the table lookups of the next
  // step (VALU v_perm + ds_read) and the code loads are spread between the
  // MFMAs instead of being issued as a burst after them.
  constexpr int NM = CW * FT;                     // MFMAs per step
  constexpr int NX = 4 * (CW + (BV ? 0 : FT));    // perms (= table reads) per step
  constexpr int PX = (NX + NM - 1) / NM;          // per MFMA
  constexpr int NL = (BV ? 4 : 1) * FT + 4 * CW;  // loads per block
  auto interleave = [&](bool with_loads) {
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, PX, 0);  // VALU
      __builtin_amdgcn_sched_group_barrier(0x100, PX, 0);  // DS read
      if (with_loads) __builtin_amdgcn_sched_group_barrier(0x020, (NL + NM - 1) / NM, 0);
    }
  };
  // One block on the codes in `cur`; a0/b0 hold its step 0 operands on entry
  // and the step 0 operands of the block in `nxt` on exit.  The registers of
  // `cur` are refilled with block `refill` during the last step, once its
  // step 3 operands are expanded.
  half8_t a0[CW], b0[FT], a1[CW], b1[FT];
  auto block_with = [&](const auto& cur, const auto& nxt, auto& refill_into, int refill,
                        auto&& loadfn) {
    operands(cur, 1, a1, b1);
    mma(a0, b0);
    interleave(false);
    __builtin_amdgcn_sched_barrier(0);
    operands(cur, 2, a0, b0);
    mma(a1, b1);
    interleave(false);
    __builtin_amdgcn_sched_barrier(0);
    operands(cur, 3, a1, b1);
    mma(a0, b0);
    interleave(false);
    __builtin_amdgcn_sched_barrier(0);
    operands(nxt, 0, a0, b0);
    loadfn(refill, refill_into);
    mma(a1, b1);
    interleave(true);
    __builtin_amdgcn_sched_barrier(0);
  };
  auto block = [&](const auto& cur, const auto& nxt, auto& refill_into, int refill) {
    block_with(cur, nxt, refill_into, refill, load);
  };
  // QL: operands of step st from a weight slot and an activation slot
  auto qoperands = [&](const WCodes& wc, const ACodes& ac, int st, half8_t (&a)[CW],
                       half8_t (&b)[FT]) {
    a[0] = expand_dual(wc.w[st][0], tb, l4w);
    b[0] = expand_dual(ac.a[0][st], tb, l4a);
#pragma unroll
    for (int c = 1; c < CW; ++c) a[c] = expand_dual(wc.w[st][c], tb, l4w);
#pragma unroll
    for (int f = 1; f < FT; ++f) b[f] = expand_dual(ac.a[f][st], tb, l4a);
  };
  // QL: one block on (wc, ac); the next block's activation words are read
  // from quad buffer qn (chunk pair bqn) into an during step 0 (three steps
  // before their first use: read right before it, the wait for them drained
  // the table reads issued in between), its step 0 operands expanded from
  // (wn, an) in the last step, where slot wr is refilled with the weights of
  // block rblk
  auto qblock = [&](const WCodes& wc, const ACodes& ac, const WCodes& wn, ACodes& an,
                    const unsigned char* qn, int bqn, WCodes& wr, int rblk) {
    aload4(qn, bqn, an);
    qoperands(wc, ac, 1, a1, b1);
    mma(a0, b0);
    interleave(false);
    __builtin_amdgcn_sched_barrier(0);
    qoperands(wc, ac, 2, a0, b0);
    mma(a1, b1);
    interleave(false);
    __builtin_amdgcn_sched_barrier(0);
    qoperands(wc, ac, 3, a1, b1);
    mma(a0, b0);
    interleave(false);
    __builtin_amdgcn_sched_barrier(0);
    qoperands(wn, an, 0, a0, b0);
    wload4(rblk, wr);
    mma(a1, b1);
    interleave(true);
    __builtin_amdgcn_sched_barrier(0);
  };
  // QL: quad Q of this tile, or from nq on the workgroup's next tile
  auto dma_quad = [&](unsigned char* q, int Q, int nq) {
    uint32_t dq[NDMA];
    const bool nxt = Q >= nq;
#pragma unroll
    for (int i = 0; i < NDMA; ++i) dq[i] = nxt ? dnext[i] : dcur[i];
    dma(q, dq, (uint32_t)(nxt ? Q - nq : Q) * 128u);
  };

  // ---- prologue: the first tile's first two blocks requested, then the table
  TileCodes<CW, FT, BV> c0, c1;
  WCodes W0, W1, W2, W3;
  ACodes A0, A1;
  place(blockIdx.x);
  if constexpr (QL) {
    dma(actq0, dcur, 0u);
    dma(actq1, dcur, 128u);
    wload4(0, W0);
    wload4(1, W1);
    wload4(2, W2);
    wload4(3, W3);
  } else {
    load(0, c0);
    load(1, c1);
  }
  if (wave < 4) {
    DualTableLoader dt;
    dt.load(A.lut, (uint32_t)wave);
    dt.store(tab, (uint32_t)wave, lane);
  }
  if constexpr (QL) __builtin_amdgcn_s_waitcnt(0);  // this wave's quad copies
  __syncthreads();
  if constexpr (QL) aload4(actq0, 0, A0);

  // HV: the heavy channels' blocks (ceil(2 nh / 64) of 64 positions) and
  // their descriptors, read once per workgroup
  const int nhb = HV ? (2 * __builtin_amdgcn_readfirstlane(*A.nheavy) + 63) / 64 : 0;
  const __amdgpu_buffer_rsrc_t rhw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(A.hw), 0, HV ? (int)((uint32_t)(kSplitPos / 8) * d_out * 4u) : 0,
      0x00020000);
  const uint32_t hrow = 2u * kSplitPos;  // bytes per token row of hv
  const __amdgpu_buffer_rsrc_t rhv = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(A.hv), 0, HV ? (int)((uint32_t)A.n * hrow) : 0, 0x00020000);

  for (int u = blockIdx.x; u < T; u += gridDim.x) {
    // this tile's scales, used in its epilogue: lane l holds the column
    // scales of columns 2l, 2l + 1 of the wave's tile and t_i of its tokens
    const uint32_t csp = (uint32_t)min(j0 + 2 * lane, A.d_out) * 4u;
    const uint32_t sw0 = __builtin_amdgcn_raw_buffer_load_b32(
        rsw, (int)csp, 0, 0);
    const uint32_t sw1 = __builtin_amdgcn_raw_buffer_load_b32(
        rsw, (int)(csp + 4u), 0, 0);
    float tsr[FT];
#pragma unroll
    for (int f = 0; f < FT; ++f)
      tsr[f] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(
                     rst, (int)((uint32_t)min(t0 + 32 * f + r32, A.n) * 4u), 0, 0));
#pragma unroll
    for (int c = 0; c < CW; ++c)
#pragma unroll
      for (int f = 0; f < FT; ++f)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[c][f][v] = 0.0f;

    // block b's codes are in c0 (b even) or c1; during its last step the
    // registers are refilled with the codes two blocks ahead (requested one
    // block before the step that expands them).  The loop body is
    // straight-line (an odd last block is peeled): with a conditional half in
    // it the compiler's wait analysis would assume the worst at the loop head
    // and wait for every load in flight.  Blocks past the end read zeros
    // (never used).
    if constexpr (QL) {
      // two quads per iteration, blocks b .. b + 7: quad m in actq0, m + 1
      // in actq1 (published before block b + 3), m + 2 copied into actq0
      // after that and published before block b + 7, m + 3 copied into
      // actq1 after that.  Block x's weights are in slot x mod 4, its
      // activation words in slot x mod 2.  In the last iteration the copies
      // are the next tile's quads 0 and 1, so it starts on them.
      const int nq = nblk >> 2;  // even
      qoperands(W0, A0, 0, a0, b0);
      for (int m = 0; m < nq; m += 2) {
        const int b = 4 * m;
        qblock(W0, A0, W1, A1, actq0, 1, W0, b + 4);
        qblock(W1, A1, W2, A0, actq0, 2, W1, b + 5);
        qblock(W2, A0, W3, A1, actq0, 3, W2, b + 6);
        publish();
        dma_quad(actq0, m + 2, nq);
        qblock(W3, A1, W0, A0, actq1, 0, W3, b + 7);
        qblock(W0, A0, W1, A1, actq1, 1, W0, b + 8);
        qblock(W1, A1, W2, A0, actq1, 2, W1, b + 9);
        qblock(W2, A0, W3, A1, actq1, 3, W2, b + 10);
        publish();
        dma_quad(actq1, m + 3, nq);
        qblock(W3, A1, W0, A0, actq0, 0, W3, b + 11);
      }
    } else {
      operands(c0, 0, a0, b0);
      int blk = 0;
      for (; blk + 1 < nblk; blk += 2) {
        block(c0, c1, c0, blk + 2);
        block(c1, c0, c1, blk + 3);
      }
      if (blk < nblk) block(c0, c1, c0, blk + 2);
    }

    if constexpr (HV) {
      // the heavy channels of the split compensation: value operand A.hv,
      // weight codes A.hw, nhb blocks
      if (nhb > 0) {
        uint32_t hoff[FT];
#pragma unroll
        for (int f = 0; f < FT; ++f)
          hoff[f] = (uint32_t)min(t0 + 32 * f + r32, A.n - 1) * hrow + 64u * (uint32_t)h;
        // blocks past the last heavy one (the tensors hold kSplitPos / 64)
        // read zeros: fetched, the two refills past it cost 2 / nhb more of
        // these reads per tile
        auto hload = [&](int b, auto& tc) { load_from(b, nhb - 1, tc, rhw, rhv, hoff); };
        if constexpr (CW * FT > 8) {
          TileCodes<CW, FT, true> h0, h1;
          hload(0, h0);
          hload(1, h1);
          operands(h0, 0, a0, b0);
          int hb = 0;
          for (; hb + 1 < nhb; hb += 2) {
            block_with(h0, h1, h0, hb + 2, hload);
            block_with(h1, h0, h1, hb + 3, hload);
          }
          if (hb < nhb) block_with(h0, h1, h0, hb + 2, hload);
        } else {
          // two workgroups per CU (256 registers a lane): a second whole value
          // block in flight spilled the main loop's registers, so a block is
          // taken one token group at a time (its weight words read again for
          // each): units (block, group) alternate between two buffers, the
          // next unit's words in flight while one is multiplied
          static_assert(FT == 2, "two token groups a wave");
          struct HUnit {
            uint32_t w[4][CW];  // weight word 4h + s of column group c
            uint4_t a[4];       // values 8 (4h + s) .. + 7 of the unit's group, step s
          };
          auto uload = [&](int b, int f, HUnit& hu) {
            const uint32_t bc = sblk(b, nhb - 1);
            const bool in = b < nhb;
            const __amdgpu_buffer_rsrc_t rvb = in ? rhv : rz, rwb = in ? rhw : rz;
#pragma unroll
            for (int st = 0; st < 4; ++st)
              hu.a[st] = __builtin_bit_cast(
                  uint4_t, __builtin_amdgcn_raw_buffer_load_b128(
                               rvb, (int)hoff[f], (int)(bc * 128u + 16u * (uint32_t)st), 0));
#pragma unroll
            for (int st = 0; st < 4; ++st)
#pragma unroll
              for (int c = 0; c < CW; ++c)
                hu.w[st][c] = __builtin_amdgcn_raw_buffer_load_b32(
                    rwb, (int)woff[c], (int)(bc * wblk + (uint32_t)st * wrow), 0);
          };
          auto umma = [&](const HUnit& hu, auto fc) {
            constexpr int f = decltype(fc)::value;
#pragma unroll
            for (int st = 0; st < 4; ++st) {
              half8_t a[CW];
#pragma unroll
              for (int c = 0; c < CW; ++c) a[c] = expand_dual(hu.w[st][c], tb, l4w);
              const half8_t bv = __builtin_bit_cast(half8_t, hu.a[st]);
#pragma unroll
              for (int c = 0; c < CW; ++c)
                acc[c][f] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[c], bv, acc[c][f], 0, 0, 0);
            }
          };
          // blocks past the last read zeros: never used
          HUnit x, y;
          uload(0, 0, x);
          uload(0, 1, y);
          for (int hb = 0; hb < nhb; ++hb) {
            umma(x, std::integral_constant<int, 0>{});
            uload(hb + 1, 0, x);
            umma(y, std::integral_constant<int, 1>{});
            uload(hb + 1, 1, y);
          }
        }
      }
    }

    const int jt = j0, tt = t0;

    // ---- epilogue: y (+)= t_i * s_j * acc, four consecutive columns per store
    if (2 * lane < 32 * CW)
      *reinterpret_cast<uint2*>(&wsc[wave][2 * lane]) = make_uint2(sw0, sw1);
    const bool vec = (A.d_out & 3) == 0 && (reinterpret_cast<uintptr_t>(A.y) & 15u) == 0;
#pragma unroll
    for (int f = 0; f < FT; ++f) {
      const int tok = tt + 32 * f + r32;
      if (tok >= A.n) continue;
      const float ts = tsr[f];
      float* yrow = A.y + (size_t)tok * A.d_out;
#pragma unroll
      for (int c = 0; c < CW; ++c)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int jl = 32 * c + 8 * g + 4 * h, j = jt + jl;
          if (vec) {
            if (j >= A.d_out) continue;  // d_out % 4 == 0: the four columns are all in or out
            const float4_t sw = *reinterpret_cast<const float4_t*>(&wsc[wave][jl]);
            float4_t v = {acc[c][f][4 * g], acc[c][f][4 * g + 1], acc[c][f][4 * g + 2],
                          acc[c][f][4 * g + 3]};
            v = ts * sw * v;
            // plain stores: non-temporal ones (cache policy nt) measured
            // slower at every shape, 1804 -> 1683 us at 4096 x 8192 x 28672
            // and 226 -> 184 us at 2048 x 4096 x 11008 when replaced by these
            float4_t* dst = reinterpret_cast<float4_t*>(yrow + j);
            *dst = A.accumulate ? *dst + v : v;
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (j + q >= A.d_out) continue;
              const float v = ts * wsc[wave][jl + q] * acc[c][f][4 * g + q];
              yrow[j + q] = A.accumulate ? yrow[j + q] + v : v;
            }
          }
        }
    }

    // ---- the next tile's first blocks, requested after this tile's stores
    if (u + (int)gridDim.x < T) {
      place(u + (int)gridDim.x);
      if constexpr (QL) {  // its quad 0 is in actq0 (published in the last iteration)
        wload4(0, W0);
        wload4(1, W1);
        wload4(2, W2);
        wload4(3, W3);
        aload4(actq0, 0, A0);
      } else {
        load(0, c0);
        load(1, c1);
      }
    }
  }
}

// Workgroups that fit on the device at once (persistent grids), per device.
static int resident_workgroups(int per_cu) {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256 * per_cu;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n * per_cu;
}

template <int CW, int FT, int WX, int WY, bool BV = false, bool HV = false>
static hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
  constexpr int TC = 32 * CW * WX, TT = 32 * FT * WY;
  constexpr int PER_CU = (CW * FT > 8 || BV || WX * WY > 4) ? 1 : 2;
  const int ncx = (a.d_out + TC - 1) / TC;
  const int nty = (a.n + TT - 1) / TT;
  const int grid = min(ncx * nty, resident_workgroups(PER_CU));
  if constexpr (!BV && WX == 2 && (FT == 4 || WY == 4)) {
    if (a.d_in % 512 == 0) {
      hipLaunchKernelGGL((k_gemm_mfma_tile<CW, FT, WX, WY, BV, HV, true>), dim3(grid),
                         dim3(WX * WY * 64), 0, s, a, ncx, nty);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((k_gemm_mfma_tile<CW, FT, WX, WY, BV, HV>), dim3(grid),
                     dim3(WX * WY * 64), 0, s, a, ncx, nty);
  return hipGetLastError();
}

// The dense part of the split compensation: B = fp16 values (a.idx_act, rows
// of a.a_row bytes), reduction length 2 * *a.kdyn positions, weight codes
// a.idx_w in the GEMM layout over those positions.
hipError_t launch_gemm_values(const GemmArgs& a, hipStream_t s) {
  return launch_tile<4, 2, 2, 2, true>(a, s);
}

// Workgroup tile 256 x 256 (2 x 2 waves of 128 x 128, 256 accumulator
// registers per lane: one wave per SIMD) when the grid fills at least three
// rounds of the 256 CUs, else 256 x 128 (waves of 128 x 64, two workgroups
// and two waves per SIMD on a CU).  Needs d_in % 64 == 0 (whole blocks of 64
// channels).
template <bool HV = false>
static hipError_t launch_gemm_tiles(const GemmArgs& a, hipStream_t s) {
  const long t44 = (long)((a.d_out + 255) / 256) * ((a.n + 255) / 256);
  if (t44 >= 3 * 256) return launch_tile<4, 4, 2, 2, false, HV>(a, s);
  return launch_tile<4, 2, 2, 2, false, HV>(a, s);
}

hipError_t launch_gemm_heavy(const GemmArgs& a, hipStream_t s) {
  return launch_gemm_tiles<true>(a, s);
}

template <int CW, int TF, int WX, int WY>
static void launch_prefill(const GemmArgs& a, hipStream_t s) {
  const int ncx = (a.d_out + WX * 16 * CW - 1) / (WX * 16 * CW);
  const int nty = (a.n + WY * 16 * TF - 1) / (WY * 16 * TF);
  if ((a.d_in / 8) % 16 == 0)
    hipLaunchKernelGGL((k_gemm_mfma_prefill<CW, TF, WX, WY, true>), dim3(ncx * nty),
                       dim3(WX * WY * 64), 0, s, a, ncx, nty);
  else
    hipLaunchKernelGGL((k_gemm_mfma_prefill<CW, TF, WX, WY, false>), dim3(ncx * nty),
                       dim3(WX * WY * 64), 0, s, a, ncx, nty);
}

template <int CW, int TF, int NW, int B, bool ROWS, bool PERCOL = false>
static void launch_gemv_b(const GemmArgs& a, hipStream_t s) {
  const int ntiles = (a.d_out + 16 * CW - 1) / (16 * CW);
  constexpr int PF = 2;  // blocks in flight per wave (four measured slower)
  if ((a.d_in / 8) % 16 == 0)
    hipLaunchKernelGGL((k_gemm_mfma_gemv<CW, TF, NW, PF, true, B, ROWS, PERCOL>), dim3(ntiles),
                       dim3(NW * 64), 0, s, a, ntiles);
  else
    hipLaunchKernelGGL((k_gemm_mfma_gemv<CW, TF, NW, PF, false, B, ROWS, PERCOL>), dim3(ntiles),
                       dim3(NW * 64), 0, s, a, ntiles);
}

// Per-output-channel codebooks: 16-column tiles, 16 waves, GEMM-layout rows
// for the fused compensation.
template <int TF>
static void launch_gemv_percol(const GemmArgs& a, hipStream_t s) {
  constexpr int NSLICES = (1024 / (16 * TF)) / 4;
  if (a.k == 0)
    launch_gemv_b<1, TF, 16, 0, false, true>(a, s);
  else if (2 * a.k <= 4 * NSLICES)
    launch_gemv_b<1, TF, 16, 4, false, true>(a, s);
  else
    launch_gemv_b<1, TF, 16, 8, false, true>(a, s);
}

// More than 32 tokens: one GEMV launch per 32-token chunk (token-major
// arguments offset to the chunk); every chunk re-reads the weight codes, from
// the last-level cache when they fit there.
hipError_t launch_gemm_percol(const GemmArgs& a, hipStream_t s) {
  constexpr int CHUNK = 32;
  for (int t0 = 0; t0 < a.n; t0 += CHUNK) {
    GemmArgs c = a;
    c.n = min(CHUNK, a.n - t0);
    c.idx_act = a.idx_act + (size_t)t0 * (size_t)(a.d_in / 2);
    c.act_scale = a.act_scale + t0;
    c.y = a.y + (size_t)t0 * (size_t)a.d_out;
    if (a.k > 0) {
      c.max_idx = a.max_idx + (size_t)t0 * a.k;
      c.min_idx = a.min_idx + (size_t)t0 * a.k;
      c.residual = a.residual + (size_t)t0 * 2 * a.k;
    }
    if (c.n <= 16)
      launch_gemv_percol<1>(c, s);
    else
      launch_gemv_percol<2>(c, s);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Outlier entries in flight per compensation thread: about a token's share of
// one slice, at most 8.
template <int CW, int TF, int NW, bool ROWS>
static void launch_gemv_r(const GemmArgs& a, hipStream_t s) {
  constexpr int NSLICES = (NW * 64 / (16 * TF)) / (16 * CW / (ROWS ? 8 : 4));
  if (2 * a.k <= 4 * NSLICES)
    launch_gemv_b<CW, TF, NW, 4, ROWS>(a, s);
  else
    launch_gemv_b<CW, TF, NW, 8, ROWS>(a, s);
}

// The fused compensation reads the row layout when the GEMM layout would cost
// at least twice the tile's own weight stream (n * 2k words of 4 B per
// column against d_in / 8): those row words are L2 hits while the tile
// streams them, the row layout's are separate (cold) reads of 0.5 B.
// No lists (k = 0): B = 0, a kernel without the outlier branch.
template <int CW, int TF, int NW>
static void launch_gemv(const GemmArgs& a, hipStream_t s) {
  if (a.k == 0)
    launch_gemv_b<CW, TF, NW, 0, false>(a, s);
  else if (a.idx_wr && 8ll * a.n * a.k >= (long long)a.d_in)
    launch_gemv_r<CW, TF, NW, true>(a, s);
  else
    launch_gemv_r<CW, TF, NW, false>(a, s);
}

// Two tile widths (k_gemm_mfma_gemv2): na = one workgroup per CU of 16*CWA
// columns, the rest in tiles of 16*CWB; the outlier lists as in launch_gemv
// (entries in flight chosen for the wider tiles).
// Whole K blocks only (d_in a multiple of 128): with a masked last block the
// wider body needs more than 128 VGPRs and two workgroups no longer fit a CU.
template <int CWA, int CWB, int NW, int B, bool ROWS>
static void launch_gemv2_b(const GemmArgs& a, int na, int nb, hipStream_t s) {
  constexpr int PF = 2;
  hipLaunchKernelGGL((k_gemm_mfma_gemv2<CWA, CWB, NW, PF, true, B, ROWS>), dim3(na + nb),
                     dim3(NW * 64), 0, s, a, na, nb);
}

template <int CWA, int CWB, int NW>
static void launch_gemv2(const GemmArgs& a, int na, hipStream_t s) {
  const int nb = (a.d_out - na * 16 * CWA + 16 * CWB - 1) / (16 * CWB);
  const bool rows = a.idx_wr && 8ll * a.n * a.k >= (long long)a.d_in;
  const int nsl = (NW * 4) / (16 * CWA / (rows ? 8 : 4));  // slices of the wider tiles
  if (a.k == 0)
    launch_gemv2_b<CWA, CWB, NW, 0, false>(a, na, nb, s);
  else if (rows && 2 * a.k <= 4 * nsl)
    launch_gemv2_b<CWA, CWB, NW, 4, true>(a, na, nb, s);
  else if (rows)
    launch_gemv2_b<CWA, CWB, NW, 8, true>(a, na, nb, s);
  else if (2 * a.k <= 4 * nsl)
    launch_gemv2_b<CWA, CWB, NW, 4, false>(a, na, nb, s);
  else
    launch_gemv2_b<CWA, CWB, NW, 8, false>(a, na, nb, s);
}

template <int TF>
static void launch_gemv_tf(const GemmArgs& a, hipStream_t s) {
  // The columns are dealt evenly over the CUs (per = 16-column tiles per CU):
  // the busiest CU sets the time.  Up to 64 columns per CU, one workgroup per
  // CU of 16 * per columns (16 waves at 16 or 32 columns, 8 at 48 or 64); a
  // 1024-thread workgroup fills a CU, so more of them than CUs would run in
  // two rounds.  Between 64 and 112 columns per CU (whole K blocks) two
  // workgroups per CU of about equal width, 48 + 32, 48 + 48 or 64 + 48
  // columns; beyond that, 64-column tiles.  LDS: reduction buffer
  // NW * CW * TF KiB <= 32 KiB; the fused compensation takes a token's
  // threads (NW * 64 / (16 * TF)) in slices of CW * 4 (row layout: CW * 2).
  const int ncu = resident_workgroups(1);
  const int per = ((a.d_out + 15) / 16 + ncu - 1) / ncu;
  if constexpr (TF == 1) {
    if (per <= 1) launch_gemv<1, 1, 16>(a, s);
    else if (per == 2) launch_gemv<2, 1, 16>(a, s);
    else if (per == 3) launch_gemv<3, 1, 8>(a, s);
    else if (per == 4) launch_gemv<4, 1, 8>(a, s);
    else if ((a.d_in / 8) % 16 == 0 && per == 5) launch_gemv2<3, 2, 8>(a, ncu, s);
    else if ((a.d_in / 8) % 16 == 0 && per == 6) launch_gemv<3, 1, 8>(a, s);
    else if ((a.d_in / 8) % 16 == 0 && per == 7) launch_gemv2<4, 3, 8>(a, ncu, s);
    else launch_gemv<4, 1, 8>(a, s);
  } else {
    if (per <= 1) launch_gemv<1, TF, 16>(a, s);
    else launch_gemv<2, TF, 8>(a, s);
  }
}

hipError_t launch_gemm_mfma(const GemmArgs& a, hipStream_t s) {
  if (a.n <= 16) {
    launch_gemv_tf<1>(a, s);
  } else if (a.n <= 32) {
    launch_gemv_tf<2>(a, s);
  } else if (a.d_in % 64 == 0) {
    return launch_gemm_tiles(a, s);
  } else {
    launch_prefill<4, 4, 2, 2>(a, s);
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
  __shared__ float lut1[256];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  lut1[tid] = A.lut->lut[tid];  // one coalesced load, then replicate from LDS
  __syncthreads();
  for (int e = tid; e < 256 * LUT_R; e += 256) lut_s[e] = lut1[e / LUT_R];
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
    if (t < ntok && j < A.d_out) {
      const int tok = tok0 + t;
      float* dst = A.y + (size_t)tok * A.d_out + j;
      const float val = A.act_scale[tok] * A.w_scale[j] * v;
      if (atomic)
        unsafeAtomicAdd(dst, val);
      else if (A.accumulate)
        *dst += val;
      else
        *dst = val;
    }
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
