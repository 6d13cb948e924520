// gemm_tile.hip -- the grouped FP8 GEMMs of stage (3) of the Fused MoE block
// (paper Section 3.1.1) for batches with many rows per expert (prefill-sized
// and skewed loads), on CDNA4 FP8 matrix cores.
//
// Work item = (M-tile of BM rows of one expert, 256-column block), the whole
// K range.  Items of one expert are ordered in groups of four column blocks:
// all M-tiles of a group, column block fastest, so the items an XCD runs side
// by side share four weight panels and a few A tiles in that XCD's L2
// (tile_item below maps workgroups to items).
//
// One workgroup of 4 x WM waves per item.  Wave (wm, wn) = (wave / 4,
// wave % 4) owns rows [16 MT wm, 16 MT (wm+1)) of the tile (BM = 16 MT WM)
// and 64 columns:
//   GEMM1: wn owns gate columns [32 wn, 32 wn + 32) of the 128-wide
//          intermediate block and the matching up columns (sub-tiles 0-1
//          gate, 2-3 up: SwiGLU pairs meet in the wave's registers; the
//          gate and up halves take their own weight-block scale);
//   GEMM2: wn owns output columns [64 wn, 64 wn + 64) of the 256-wide block.
// Every K-step's operands -- the A tile (rows gathered through perm_token
// for GEMM1), its row scales and the 256 weight rows -- go straight from
// global memory into an S-stage LDS ring (direct loads issued S-1 K-steps
// ahead, no registers), with one barrier per K-step.  In the eight-wave
// tiles the two waves of a SIMD take turns issuing a step's loads (see
// TileSrcPair), so one of them always has only math to issue.
//
// The weight fragment is the MFMA's first operand and the activation fragment
// its second, so lane l holds output columns 4*(l/16)+i (i = 0..3) of token
// row l%16 of each 16x16 sub-tile: one activation scale per lane and sub-tile
// row block.  Each 128-K step is one v_mfma_f32_16x16x128_f8f6f4 per
// sub-tile, started from zero and promoted into the fp32 accumulator with
// one FMA by (activation scale * weight-block scale), in K order -- the same
// arithmetic as the small-tile kernels that keep one K range per item (the
// matrix cores' block sum does not depend on which operand comes first).
#include "moe_device.h"

namespace moe {
namespace {

constexpr int kTileCols = 256;
constexpr int kGroupN = 4;  // column blocks per item group

// LDS stage: A tile (BM rows x 128 bytes), the 256 weight rows (4 blocks of
// 64, one per column wave), the row-scale slots (64 per wave).  Rows are
// 128 bytes; 16-byte chunk c of row r sits in slot c ^ f(r), f(r) =
// (r % 8) ^ ((r / 8) % 2): measured on gfx950, the fragment reads (16 rows,
// two 16-byte pieces per lane) then run without bank conflicts, while each
// direct load fetches whole 128-byte lines (8 rows per wave-wide load).
template <int MT, int WM, int S>
struct TileLayout {
  static constexpr int THREADS = 256 * WM;
  static constexpr int BM = 16 * MT * WM;
  static constexpr int A_BYTES = BM * 128;
  static constexpr int SCL = A_BYTES + 4 * 8192;
  static constexpr int STAGE = SCL + 4 * WM * 256;
  static constexpr int JUNK = 4 * WM * 256;  // landing area of the L2 prefetches
  // row-scale slots: row r16's MTW block scales at r16 * SS; rows 80 (or 48)
  // bytes apart put the 16 rows' float4 reads in distinct LDS banks (at 64
  // or 32 bytes they conflict four or two ways)
  static constexpr int SS = MT * WM >= 8 ? MT * WM + 4 : MT * WM;
  static_assert(16 * SS <= 64 * 4 * WM, "row-scale slots fit the workgroup's lanes");
  static constexpr int RING = S * STAGE + JUNK;
  // the ring, then the two weight-scale rows of an item (2 KB floats, filled
  // 64 at a time by direct loads)
  static size_t bytes(int KB) { return (size_t)RING + sizeof(float) * (size_t)((2 * KB + 63) / 64 * 64); }
};

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ int tile_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Direct global -> LDS loads.  The builtin sits in plain device functions:
// used inside the kernel template, it keeps the host compilation pass from
// emitting the kernel's launch stub.
__device__ __forceinline__ void lds_load16(const void *g, uint8_t *lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_void *)lds, 16, 0, 0);
}
__device__ __forceinline__ void lds_load4(const void *g, uint8_t *lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_void *)lds, 4, 0, 0);
}
// The same through a buffer resource: a per-lane 32-bit offset (VGPR) plus a
// uniform one (SGPR), so a K step's loads need no address arithmetic.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void lds_bload16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                            uint8_t *lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds, 16, voff, soff, 0, 0);
}
__device__ __forceinline__ void lds_bload4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                           uint8_t *lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds, 4, voff, soff, 0, 0);
}

// LDS reads of the K loop go through restrict-qualified pointers, so after
// inlining they carry alias-scope metadata.  Without it the compiler cannot
// tell them from the in-flight direct-to-LDS writes of later stages and waits
// for every outstanding load before each read; the K loop's explicit waits
// and barriers order the accesses instead.
__device__ __forceinline__ v8i tile_frag(const uint8_t *__restrict__ st, int lo, int hi) {
  const v4i a = *reinterpret_cast<const v4i *>(st + lo);
  const v4i b = *reinterpret_cast<const v4i *>(st + hi);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ __forceinline__ float4 tile_f4(const float *__restrict__ q) {
  return *reinterpret_cast<const float4 *>(q);
}
__device__ __forceinline__ float tile_f1(const float *__restrict__ q) { return *q; }

// Workgroup b -> work item.  Workgroups are dispatched round-robin over the
// 8 XCDs (b runs on XCD b % 8), and an XCD's 32 CUs each hold one workgroup.
// Items are taken in chunks of 32 -- in an expert's order, four column blocks
// of eight M-tiles -- and chunk c runs on XCD c % 8: an XCD's concurrent items
// share four weight panels and eight A tiles in its L2, and the eight XCDs
// work on neighbouring chunks (the same expert's panels) at the same time,
// so the panels one XCD re-reads are those its neighbours have just brought
// into the Infinity Cache.  The last n mod 256 items go contiguously to the
// XCDs.  Returns -1 for a workgroup without an item.
__device__ __forceinline__ int tile_item(int b, int n) {
  const int x = b & 7, j = b >> 3;
  const int full = n >> 8;  // complete rounds of 8 chunks
  if (j < 32 * full) return ((j >> 5) * 8 + x) * 32 + (j & 31);
  const int rest = n - 256 * full;
  const int per = (rest + 7) >> 3;
  const int k = j - 32 * full;
  const int it = 256 * full + x * per + k;
  return (k < per && it < n) ? it : -1;
}

// A work item's place: its expert, the expert's M-tile count, the M-tile and
// column block, the tile's rows, and the wave's first weight row and the two
// weight-scale blocks of its columns.
struct TileItem {
  int e, nt_e, mt_idx, nb, row0, nrows, wrow0, nblk0, nblk1;
};

template <bool G1, int BM>
__device__ __forceinline__ TileItem tile_decode(const GemmParams &p, int item, int wn) {
  TileItem t;
  const int NB = p.NB;
  // the item's M-tile entry: its expert, the expert's first M-tile, first
  // row and row count (one 16-byte load, uniform over the workgroup)
  const int4 te = reinterpret_cast<const int4 *>(p.tile_tab)[__builtin_amdgcn_readfirstlane(item / NB)];
  t.e = te.x;
  t.nt_e = (te.w + BM - 1) / BM;
  const int local = item - te.y * NB;
  const int G = (NB + kGroupN - 1) / kGroupN;
  const int grp = min(local / (kGroupN * t.nt_e), G - 1);
  const int wi = local - grp * kGroupN * t.nt_e;
  const int gsz = min(kGroupN, NB - kGroupN * grp);
  t.mt_idx = wi / gsz;
  t.nb = kGroupN * grp + wi % gsz;
  t.row0 = te.z + t.mt_idx * BM;
  t.nrows = min(BM, te.z + te.w - t.row0);
  const int half = wn >> 1;  // GEMM1: 0 gate, 1 up.  GEMM2: 128-column half
  if (G1) {
    // the wave's 64 weight rows: gate rows wrow0 .. wrow0+31 and the
    // matching up rows I + wrow0 .. (so SwiGLU pairs meet in the wave)
    (void)half;
    t.wrow0 = t.nb * 128 + 32 * wn;
    t.nblk0 = t.nb;
    t.nblk1 = p.I / 128 + t.nb;
  } else {
    t.wrow0 = t.nb * kTileCols + 64 * wn;
    t.nblk0 = min(2 * t.nb, p.N_total / 128 - 1);
    t.nblk1 = min(2 * t.nb + 1, p.N_total / 128 - 1);
  }
  // every field is uniform over the wave: keep them in scalar registers
  t.e = __builtin_amdgcn_readfirstlane(t.e);
  t.nt_e = __builtin_amdgcn_readfirstlane(t.nt_e);
  t.mt_idx = __builtin_amdgcn_readfirstlane(t.mt_idx);
  t.nb = __builtin_amdgcn_readfirstlane(t.nb);
  t.row0 = __builtin_amdgcn_readfirstlane(t.row0);
  t.nrows = __builtin_amdgcn_readfirstlane(t.nrows);
  t.wrow0 = __builtin_amdgcn_readfirstlane(t.wrow0);
  t.nblk0 = __builtin_amdgcn_readfirstlane(t.nblk0);
  t.nblk1 = __builtin_amdgcn_readfirstlane(t.nblk1);
  return t;
}

// This lane's source addresses of a work item's direct loads (K block 0).
template <int JA, int JB, int PF>
struct TileSrc {
  const uint8_t *a[JA];
  const uint8_t *b[JB];
  const uint8_t *pf[PF > 0 ? PF : 1];
  const float *s;
};

template <bool G1, int MT, int WM, int JA, int JB, int PF>
__device__ __forceinline__ void tile_sources(const GemmParams &p, const TileItem &t, int wave, int lane,
                                             TileSrc<JA, JB, PF> &src) {
  constexpr int BM = 16 * MT * WM;
  constexpr int MTW = MT * WM;
  const int wm = wave >> 2;
  const size_t K = (size_t)p.K;
  // A wave-wide 16-byte load fills 1 KB of a stage: lane L writes slot L,
  // i.e. row 8q + L/8, slot L % 8 of 8-row block q, and so fetches chunk
  // (L % 8) ^ f(row) of that row (f depends on the row's position in its
  // 16-row fragment only).
  const int sw_l = lane >> 3;
#pragma unroll
  for (int j = 0; j < JA; ++j) {
    const int r = 8 * (wave * JA + j) + sw_l;
    const int rr = min(r, t.nrows - 1);  // ragged tail: repeat the last row
    const int row = G1 ? p.perm_token[t.row0 + rr] : t.row0 + rr;
    src.a[j] = p.A + (size_t)row * K + 16 * ((lane & 7) ^ tile_swz(r));
  }
  // weight rows: the column wave wn's 64 rows are 8 blocks, loaded JB each by
  // the WM waves of that column
  const uint8_t *Bexp = p.B + (size_t)t.e * p.N_total * K;
#pragma unroll
  for (int j = 0; j < JB; ++j) {
    const int r = 8 * (wm * JB + j) + sw_l;
    const int rg = G1 ? (r < 32 ? t.wrow0 + r : p.I + t.wrow0 + r - 32)
                      : min(t.wrow0 + r, p.N_total - 1);  // ragged last GEMM2 block
    src.b[j] = Bexp + (size_t)rg * K + 16 * ((lane & 7) ^ tile_swz(r));
  }
  // L2 prefetch one K-step beyond the ring: one dword per 128-byte line,
  // landing in a junk LDS area that is never read.  Each line is prefetched
  // by one of the items that share it and run side by side on the XCD (the
  // others then hit in L2 instead of all waiting on the same miss): the A
  // rows of an M-tile are split over the kGroupN column blocks of its group,
  // the weight rows of a column block over MS consecutive M-tiles.  Lanes
  // past the item's share repeat its first line (one request per load).
  const int ms = t.nt_e >= 4 ? 4 : (t.nt_e >= 2 ? 2 : 1);
  const int a_share = BM / kGroupN;
  const int w_share = 256 / ms;
  const int a_first = (t.nb % kGroupN) * a_share;
  const int w_first = (t.mt_idx % ms) * w_share;
#pragma unroll
  for (int j = 0; j < PF; ++j) {
    int line = (wave * PF + j) * kWave + lane;
    if (line >= a_share + w_share) line = 0;
    if (line < a_share) {
      const int rr = min(a_first + line, t.nrows - 1);
      src.pf[j] = p.A + (size_t)(G1 ? p.perm_token[t.row0 + rr] : t.row0 + rr) * K;
    } else {
      const int c = w_first + line - a_share;  // weight row c % 64 of column wave c / 64
      const int w2 = c >> 6, rr = c & 63;
      const int row = G1 ? (rr < 32 ? t.nb * 128 + 32 * w2 + rr : p.I + t.nb * 128 + 32 * w2 + rr - 32)
                         : t.nb * kTileCols + 64 * w2 + rr;
      src.pf[j] = Bexp + (size_t)min(row, p.N_total - 1) * K;
    }
  }
  // row scales: row 16 j + r16 at slot r16 * SS + j (j < MTW; the other
  // slots are padding); lane L of wave w loads slot 64 w + L (padding and
  // slots past the tile are loaded but never read).  They come from the
  // K-block-major copy sa_tile (permuted rows): the 64 lanes' rows lie within
  // one tile, so a K step's scale load touches a few cache lines.
  constexpr int SS = TileLayout<MT, WM, 2>::SS;
  const int sl = 64 * wave + lane;
  const int sr = sl / SS, sj = sl % SS;
  const int r = (sr < 16 && sj < MTW) ? 16 * sj + sr : t.nrows - 1;
  src.s = p.sa_tile + (size_t)(t.row0 + min(r, t.nrows - 1)) * p.sa_row;
}

// The loads of the 8-wave tiles alternate between the two waves of each SIMD
// (waves wn and wn + 4): in a K step one of them issues the whole group of
// both -- their A blocks, the column wave's eight weight blocks, both waves'
// row scales -- and the other issues none, so that while the loading wave
// waits at issue for a free request slot its partner keeps the SIMD's matrix
// core busy.  These tiles issue no L2 prefetches: with the loads alternating,
// the prefetch requests only took request slots from the ring's loads
// (measured without them: prefill GEMM1 301 -> 274 us, GEMM2 166 -> 156,
// skewed GEMM1 1838 -> 1810).  The sources are 32-bit byte offsets from
// bases that are uniform over the wave (the activation rows from A, a weight
// row from its 8-row block's first row, the row scales from sa_tile), so the
// loads take the scalar-base address form and each K step only moves the
// bases.
template <int JA>
struct TileSrcPair {
  uint32_t a[2 * JA];  // A rows: wave wn's blocks, then wave wn + 4's
  uint32_t b[2];       // lane offset in an 8-row weight block, even / odd block
  uint32_t s[2];       // row-scale byte offsets of wave wn's slot, of wave wn + 4's
};

template <bool G1, int MT, int WM, int JA>
__device__ __forceinline__ void tile_sources_pair(const GemmParams &p, const TileItem &t, int wn, int lane,
                                                  TileSrcPair<JA> &src) {
  constexpr int MTW = MT * WM;
  constexpr int SS = TileLayout<MT, WM, 2>::SS;
  const uint32_t K = (uint32_t)p.K;
  const int sw_l = lane >> 3;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int w = wn + 4 * h;
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int r = 8 * (w * JA + j) + sw_l;
      const int rr = min(r, t.nrows - 1);
      const int row = G1 ? p.perm_token[t.row0 + rr] : t.row0 + rr;
      // (24-bit products: row < 2^24 and K < 2^24; a 32-bit multiply-add
      // would otherwise be formed as a 64-bit one and hold a register pair)
      src.a[h * JA + j] = __umul24((uint32_t)row, K) + 16 * ((lane & 7) ^ tile_swz(r));
    }
    const int sl = 64 * w + lane;
    const int sr = sl / SS, sj = sl % SS;
    const int r = (sr < 16 && sj < MTW) ? 16 * sj + sr : t.nrows - 1;
    src.s[h] = 4u * __umul24((uint32_t)(t.row0 + min(r, t.nrows - 1)), (uint32_t)p.sa_row);
  }
  // row 8 blk + sw_l of weight block blk: chunk (lane & 7) ^ sw_l ^ (blk & 1)
#pragma unroll
  for (int q = 0; q < 2; ++q) src.b[q] = __umul24((uint32_t)sw_l, K) + 16 * ((lane & 7) ^ sw_l ^ q);
}

// GEMM2's epilogue: the wave's accumulators (rows wrow + 16 m + r16 of the
// tile, columns wrow0 + 16 n + 4 g4 + i) as fp16 Y codes with one exponent
// per row and 16-column chunk; the chunk (sub-tile n) of row r16 is held by
// the lanes r16 + 16 g4, four columns each.
template <int MT>
__device__ __forceinline__ void tile_store_y(const GemmParams &p, const v4f (&acc)[MT][4], int row0,
                                             int nrows, int wrow0, int wrow, int r16, int g4) {
  const int HC = p.H / kYChunk;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int r = wrow + 16 * m + r16;
    int ex[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      float mx = fmaxf(fmaxf(fabsf(acc[m][n][0]), fabsf(acc[m][n][1])),
                       fmaxf(fabsf(acc[m][n][2]), fabsf(acc[m][n][3])));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      ex[n] = y16_exponent(mx);
    }
    if (r < nrows) {
      uint16_t *yrow = p.Y + (size_t)(row0 + r) * p.H + wrow0 + 4 * g4;
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        uint2 c;
        c.x = (uint32_t)y16_code(acc[m][n][0], ex[n]) | ((uint32_t)y16_code(acc[m][n][1], ex[n]) << 16);
        c.y = (uint32_t)y16_code(acc[m][n][2], ex[n]) | ((uint32_t)y16_code(acc[m][n][3], ex[n]) << 16);
        __builtin_nontemporal_store(u32x2{c.x, c.y}, reinterpret_cast<u32x2 *>(yrow + 16 * n));
      }
      // lane r16 + 16 g4 stores the exponent of chunk g4
      int eg = ex[0];
#pragma unroll
      for (int n = 1; n < 4; ++n) eg = g4 == n ? ex[n] : eg;
      __builtin_nontemporal_store((int8_t)eg, p.Ye + (size_t)(row0 + r) * HC + wrow0 / kYChunk + g4);
    }
  }
}

// GEMM1's epilogue: SwiGLU of the wave's 32 gate / 32 up column pairs (sub-
// tiles n and n + 2 of the accumulators), the row's amax over the 128-column
// block (four waves, through amax_l), scale amax / 448 (1 for an all-zero
// block), e4m3 codes (nearest even, saturating), written with the scales
// (row-major and, for the large-tile GEMM2, K-block-major).  The barrier
// waits for LDS only: loads in flight for a next item may stay in flight.
template <int MT, int BM>
__device__ __forceinline__ void tile_store_act(const GemmParams &p, const v4f (&acc)[MT][4],
                                               float (*amax_l)[BM], int row0, int nrows, int nb,
                                               int wn, int wrow, int r16, int g4) {
  float a[MT][2][4];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    float mx = 0.0f;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[m][h][i] = swiglu_fast(acc[m][h][i], acc[m][h + 2][i]);
        mx = fmaxf(mx, fabsf(a[m][h][i]));
      }
    // the row's 32 columns of this wave sit in lanes r16, r16+16, r16+32, r16+48
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (g4 == 0) amax_l[wn][wrow + 16 * m + r16] = mx;
  }
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  const int IB = p.I / 128;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int r = wrow + 16 * m + r16;
    const float amax = fmaxf(fmaxf(amax_l[0][r], amax_l[1][r]), fmaxf(amax_l[2][r], amax_l[3][r]));
    const float scale = (amax > 0.0f) ? amax / 448.0f : 1.0f;
    if (r < nrows) {
      uint8_t *arow = p.act + (size_t)(row0 + r) * p.I + nb * 128 + 32 * wn + 4 * g4;
      const DivBy ds(scale);  // the row's eight quotients share the divisor
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t q = 0u;
        if (amax > 0.0f)
          q = e4m3x2_rne_sat(ds(a[m][h][0]), ds(a[m][h][1])) |
              (e4m3x2_rne_sat(ds(a[m][h][2]), ds(a[m][h][3])) << 16);
        *reinterpret_cast<uint32_t *>(arow + 16 * h) = q;
      }
      if (wn == 0 && g4 == 0) {
        p.act_scale[(size_t)(row0 + r) * IB + nb] = scale;
        if (p.act_scale_k) p.act_scale_k[(size_t)nb * p.P_max + row0 + r] = scale;
      }
    }
  }
}

// GEMM2's epilogue through LDS (one-shot kernels, where the ring is free once
// every wave has drained its loads): the wave's fp16 codes go to its own LDS
// region as [16 MT rows][64 columns] (128-byte rows, 16-byte chunk c of row r
// in slot c ^ (r % 8) ^ (r / 8 % 2), so that rows r and r + 8 of a write
// fall in different banks), its exponents as [16 MT rows][4 chunks] (one
// dword per row), and are read
// back row-contiguously, so each global store instruction writes whole
// 128-byte lines (8 rows x 8 lanes x 16 bytes) instead of 32-byte pieces of
// four lines.  Same codes and exponents as tile_store_y.  Both write Y
// non-temporally: its 0.94 GB at the skewed load would otherwise fill the
// XCDs' L2 with lines no GEMM workgroup reads again, evicting the weight
// panels and activation tiles the concurrent items share (measured: skewed
// layer 3149 -> 3076 us over two alternating runs, the combine that reads Y
// back 227 -> 202 us, GEMM1 of the next call 1818 -> 1771)
template <int MT>
__device__ __forceinline__ void tile_store_y_lds(const GemmParams &p, const v4f (&acc)[MT][4], int row0,
                                                 int nrows, int wrow0, int wrow, int lane,
                                                 uint8_t *wl) {
  constexpr int R = 16 * MT;  // the wave's rows
  const int r16 = lane & 15, g4 = lane >> 4;
  uint8_t *el = wl + R * 128;  // exponents
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int lr = 16 * m + r16;
    int ex[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      float mx = fmaxf(fmaxf(fabsf(acc[m][n][0]), fabsf(acc[m][n][1])),
                       fmaxf(fabsf(acc[m][n][2]), fabsf(acc[m][n][3])));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      ex[n] = y16_exponent(mx);
    }
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      uint2 c;
      c.x = y16_code2(acc[m][n][0], acc[m][n][1], ex[n]);
      c.y = y16_code2(acc[m][n][2], acc[m][n][3], ex[n]);
      const int ch = (2 * n + (g4 >> 1)) ^ (lr & 7) ^ ((lr >> 3) & 1);  // chunk of columns 16n + 4g4
      *reinterpret_cast<uint2 *>(wl + lr * 128 + ch * 16 + 8 * (g4 & 1)) = c;
    }
    // every lane of the row holds its four exponents: one dword per row
    if (g4 == 0)
      *reinterpret_cast<uint32_t *>(el + lr * 4) =
          (uint32_t)(uint8_t)(int8_t)ex[0] | ((uint32_t)(uint8_t)(int8_t)ex[1] << 8) |
          ((uint32_t)(uint8_t)(int8_t)ex[2] << 16) | ((uint32_t)(uint8_t)(int8_t)ex[3] << 24);
  }
  // the wave reads back only its own region: its LDS operations are in order
  // (the empty asm keeps the compiler from moving reads above the writes)
  asm volatile("" ::: "memory");
  const int HC = p.H / kYChunk;
#pragma unroll
  for (int k = 0; k < R / 8; ++k) {
    const int lr = 8 * k + (lane >> 3), c = lane & 7;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(wl + lr * 128 + ((c ^ (lr & 7) ^ ((lr >> 3) & 1)) * 16));
    if (wrow + lr < nrows)
      __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p.Y + (size_t)(row0 + wrow + lr) * p.H + wrow0 + 8 * c));
  }
#pragma unroll
  for (int k = 0; k < R / 64; ++k) {
    const int lr = 64 * k + lane;
    const uint32_t v = *reinterpret_cast<const uint32_t *>(el + lr * 4);
    if (wrow + lr < nrows)
      __builtin_nontemporal_store(v, reinterpret_cast<uint32_t *>(p.Ye + (size_t)(row0 + wrow + lr) * HC + wrow0 / kYChunk));
  }
}

template <bool G1, int MT, int WM, int S>
__global__ __launch_bounds__(256 * WM) void gemm_tile_kernel(GemmParams p) {
  using L = TileLayout<MT, WM, S>;
  constexpr int NT = L::THREADS;
  static_assert(NT == 256 * WM, "launch bound");
  constexpr int BM = L::BM;
  static_assert(MT % 4 == 0, "row scales are read four at a time");

  __shared__ float amax_l[4][BM];
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: scalar LDS addresses
  const int wn = wave & 3;
  const int wm = wave >> 2;
  const int r16 = lane & 15;
  const int g4 = lane >> 4;

  const int item = tile_item(blockIdx.x, *p.n_items);
  if (item < 0) return;

  // ---- decode the work item
  const TileItem ti = tile_decode<G1, BM>(p, item, wn);
  const int e = ti.e, nb = ti.nb, row0 = ti.row0, nrows = ti.nrows, wrow0 = ti.wrow0;
  const int KB = p.KB;
  // (alternating loads) buffer resources of the A rows, the expert's weights
  // and the row scales; every offset into them fits 32 bits (the plan keeps
  // rows x row length of the 8-wave tiles' operands below 2^32 bytes)
  const __amdgpu_buffer_rsrc_t rs_a = tile_rsrc(p.A, 0xffffffffu);
  const __amdgpu_buffer_rsrc_t rs_b =
      tile_rsrc(p.B + (size_t)e * p.N_total * p.K, (uint32_t)p.N_total * (uint32_t)p.K);
  const __amdgpu_buffer_rsrc_t rs_s = tile_rsrc(p.sa_tile, 4u * (uint32_t)p.P_max * (uint32_t)p.KB);
  const int half = wn >> 1;

  // weight-block scales of the whole K range: sb_l[0][kb] (wn 0/1), sb_l[1][kb].
  // Wave 0 loads them straight into LDS before its first stage's loads, so
  // the prologue's wait and barrier cover them (no round trip through
  // registers and no barrier of their own in front of the A-row lookups:
  // skewed GEMM1 spends ~14 us per item outside its K loop)
  float *sb_l = reinterpret_cast<float *>(smem + L::RING);
  if (wave == 0) {
    const float *s0 = p.B_scale + ((size_t)e * (p.N_total / 128) + ti.nblk0) * KB;
    const float *s1 = p.B_scale + ((size_t)e * (p.N_total / 128) + ti.nblk1) * KB;
    for (int c = 0; c < 2 * KB; c += kWave) {
      const int i = c + lane;
      lds_load4(i < KB ? s0 + i : s1 + min(i - KB, KB - 1), reinterpret_cast<uint8_t *>(sb_l + c));
    }
  }
  // GEMM1: gate scales at sb_w[kb], up scales at sb_w[KB + kb]
  const float *sb_w = G1 ? sb_l : sb_l + half * KB;

  // ---- direct-load sources
  constexpr int JA = BM / 8 / (4 * WM);  // A blocks per wave
  constexpr int JB = 8 / WM;             // weight blocks per wave
  constexpr int kPfLoads = (BM / kGroupN + 256 + 4 * WM * kWave - 1) / (4 * WM * kWave);
  // the 8-wave tiles alternate a K step's loads between the waves of a SIMD
  constexpr bool kAlt = WM == 2;
  TileSrc<JA, JB, kPfLoads> src;
  TileSrcPair<JA> srcp;
  if constexpr (kAlt)
    tile_sources_pair<G1, MT, WM>(p, ti, wn, lane, srcp);
  else
    tile_sources<G1, MT, WM>(p, ti, wave, lane, src);
  const size_t sa_kb = (size_t)p.sa_kb;
  // this lane's two 16-byte pieces of a fragment (rows 16m + r16 of a block)
  const int fr = tile_swz(r16);
  const int rd_lo = r16 * 128 + 16 * ((2 * g4) ^ fr);
  const int rd_hi = r16 * 128 + 16 * ((2 * g4 + 1) ^ fr);

  v4f acc[MT][4];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[m][n] = v4f{0.f, 0.f, 0.f, 0.f};

  // Each K-step every wave issues one group of kGroup direct loads (stage
  // it+S-1), then kPfLoads prefetches (step it+S).  At the end of step `it`
  // stage it+1 must have landed: its group was issued S-2 steps earlier, so
  // the (S-2) later groups and this step's prefetches may be outstanding.
  // Inside a step the group is spread over the first kSpread of the MT row
  // blocks' MFMAs, the prefetches after it: issued in one burst, a wave
  // stalled at issue on the CU's full request queue before its first MFMA
  // (interleaved: prefill 643 -> 604 us, skewed 3698 -> 3622 us, measured on
  // one box; the last quarter of the blocks issues no loads, so the group
  // has the rest of the step to land even with a two-stage ring).
  constexpr int kGroup = JA + JB + 1;
  constexpr int kWait = (S - 2) * (kGroup + kPfLoads) + kPfLoads;
  // the 256-row GEMM1 tiles raise their waves' issue priority for a step's
  // math and drop it before the step's barrier (measured: skewed GEMM1
  // 1968 -> 1934 us over three alternating runs; the 128-row prefill tiles
  // lost 6 us with it, GEMM2 unchanged).  With alternating loads the loading
  // wave of a step runs above its partner for the whole step, so that its
  // loads and MFMAs issue first and the partner fills the gaps (skewed GEMM1
  // 1785 -> 1763 us, GEMM2 1065 -> 1057, prefill GEMM1 274 -> 271 over two
  // alternating runs)
  constexpr bool kPrio = G1 && L::BM == 256;
  constexpr int kSpread = MT / 2;
  static_assert(kWait < 64, "vmcnt holds 6 bits");
  static_assert(S >= 2, "LDS ring depth");
  // alternating loads: the loading wave's group; at a step's end it waits for
  // its group when the ring has two stages (that stage is read next) and for
  // nothing of its own with three (its partner loaded the next stage a step
  // earlier and waits for that group now)
  constexpr int kGroupP = 2 * JA + 8 + 2;
  constexpr int kWaitLd = S == 2 ? 0 : kGroupP;
  static_assert(!kAlt || (S <= 3 && JB * WM == 8 && kWaitLd < 64), "alternating loads");

#define TILE_STAGE(st) (smem + (st) * L::STAGE)
// load j of the group for stage st, K block kb: the wave's A blocks, then its
// weight blocks, then the row scales (j is a compile-time constant)
#define TILE_DMA_J(st, kb, j)                                                           \
  do {                                                                                  \
    uint8_t *d_ = TILE_STAGE(st);                                                       \
    const size_t ko_ = (size_t)(kb) * 128;                                              \
    if ((j) < JA)                                                                       \
      lds_load16(src.a[(j) < JA ? (j) : 0] + ko_, d_ + (wave * JA + (j)) * 1024);       \
    else if ((j) < JA + JB)                                                             \
      lds_load16(src.b[(j) >= JA && (j) < JA + JB ? (j) - JA : 0] + ko_,                \
                 d_ + L::A_BYTES + wn * 8192 + (wm * JB + (j) - JA) * 1024);            \
    else                                                                                \
      lds_load4(src.s + (kb) * sa_kb, d_ + L::SCL + wave * 256);                        \
  } while (0)
#define TILE_PREFETCH(kb)                                                               \
  do {                                                                                  \
    _Pragma("unroll") for (int j = 0; j < kPfLoads; ++j)                                \
        lds_load4(src.pf[j] + (size_t)(kb) * 128, smem + S * L::STAGE + wave * 256);    \
  } while (0)
// load j of a wave pair's group (alternating loads): the A blocks of wave wn
// and of wave wn + 4, the column wave's eight weight blocks, the two waves'
// row scales
#define TILE_DMA_P(st, kb, j)                                                           \
  do {                                                                                  \
    uint8_t *d_ = TILE_STAGE(st);                                                       \
    if ((j) < 2 * JA) {                                                                 \
      const int jj_ = (j) < 2 * JA ? (j) : 0;                                           \
      lds_bload16(rs_a, srcp.a[jj_], (uint32_t)(kb) * 128u,                             \
                  d_ + ((wn + 4 * (jj_ / JA)) * JA + jj_ % JA) * 1024);                 \
    } else if ((j) < 2 * JA + 8) {                                                      \
      const int blk_ = (j) - 2 * JA;                                                    \
      const int r0_ = G1 ? (blk_ < 4 ? wrow0 + 8 * blk_ : p.I + wrow0 + 8 * (blk_ - 4))  \
                         : min(wrow0 + 8 * blk_, p.N_total - 8);                        \
      lds_bload16(rs_b, srcp.b[blk_ & 1], (uint32_t)r0_ * (uint32_t)p.K + (uint32_t)(kb) * 128u, \
                  d_ + L::A_BYTES + wn * 8192 + blk_ * 1024);                           \
    } else {                                                                            \
      const int h_ = (j) - 2 * JA - 8 < 1 ? 0 : 1;                                      \
      lds_bload4(rs_s, srcp.s[h_], (uint32_t)(kb) * (uint32_t)sa_kb * 4u,               \
                 d_ + L::SCL + (wn + 4 * h_) * 256);                                    \
    }                                                                                   \
  } while (0)
#define TILE_NODMA(st, kb, j) \
  do {                        \
  } while (0)
#define TILE_NOPF(kb) \
  do {                \
  } while (0)
// One K-step of the wave's 16 MT x 64 block: per 16-row block m, four MFMAs
// (one per 16-column sub-tile), each started from zero and promoted with one
// FMA per accumulator; the next block's A fragment is read while this one
// is multiplied.  The compiler is left free to interleave the blocks: an
// FMA that reads the result of the MFMA issued just before it stalls for
// the whole matrix-core pass, so promotions are scheduled a few MFMAs late
// (a register-only probe on gfx950: 42 cycles per MFMA with one wave per
// SIMD, 62 when each block's promotions are pinned behind its MFMAs; 32 is
// the issue rate).  Two waves per SIMD (8-wave tiles) fill the rest.
// Blocks m < kSpread also issue their share of the next group (stage stl,
// K block kbl) and the last of them the prefetches (K block kbp); the
// scheduling barrier after them lets everything but vector-memory
// instructions move across (mask 0x78F), so the loads stay among that
// block's MFMAs while the math keeps its free order.  Only the first MV row
// blocks (a compile-time count) are multiplied: the others hold no pairs of
// the item, and their loads are still issued so that every wave's vmcnt
// bookkeeping is the same.
#define TILE_COMPUTE(st, kb, stl, kbl, kbp, MV, DMA, NG, PFM)                            \
  do {                                                                                  \
    const uint8_t *as_ = TILE_STAGE(st) + wm * MT * 2048;                               \
    const uint8_t *bs_ = TILE_STAGE(st) + L::A_BYTES + wn * 8192;                       \
    const float *sa_ =                                                                  \
        reinterpret_cast<const float *>(TILE_STAGE(st) + L::SCL) + r16 * L::SS + wm * MT; \
    const float sbv_ = tile_f1(sb_w + (kb));                                            \
    const float sbu_ = G1 ? tile_f1(sb_w + KB + (kb)) : sbv_;                           \
    float sav_[MT];                                                                     \
    _Pragma("unroll") for (int q_ = 0; q_ < MT / 4; ++q_) {                             \
      const float4 v_ = tile_f4(sa_ + 4 * q_);                                          \
      sav_[4 * q_ + 0] = v_.x;                                                          \
      sav_[4 * q_ + 1] = v_.y;                                                          \
      sav_[4 * q_ + 2] = v_.z;                                                          \
      sav_[4 * q_ + 3] = v_.w;                                                          \
    }                                                                                   \
    if (kAlt && (NG) > 0) __builtin_amdgcn_s_setprio(2);                                \
    else if (kPrio) __builtin_amdgcn_s_setprio(1);                                      \
    v8i bf_[4];                                                                         \
    _Pragma("unroll") for (int n = 0; n < 4; ++n) bf_[n] =                              \
        tile_frag(bs_ + n * 2048, rd_lo, rd_hi);                                        \
    v8i an_ = {};                                                                       \
    if ((MV) > 0) an_ = tile_frag(as_, rd_lo, rd_hi);                                   \
    _Pragma("unroll") for (int m = 0; m < MT; ++m) {                                    \
      if (m < kSpread) {                                                                \
        _Pragma("unroll") for (int j_ = (m * (NG)) / kSpread;                           \
                               j_ < ((m + 1) * (NG)) / kSpread; ++j_)                   \
            DMA(stl, kbl, j_);                                                          \
        if (m == kSpread - 1) PFM(kbp);                                                 \
        __builtin_amdgcn_sched_barrier(0x78F);                                          \
      }                                                                                 \
      if (m >= (MV)) continue;                                                          \
      const v8i af_ = an_;                                                              \
      if (m + 1 < (MV)) an_ = tile_frag(as_ + (m + 1) * 2048, rd_lo, rd_hi);            \
      const float c_ = sav_[m] * sbv_;                                                  \
      const float cu_ = G1 ? sav_[m] * sbu_ : c_;                                       \
      const v4f z_ = {0.f, 0.f, 0.f, 0.f};                                              \
      v4f t_[4];                                                                        \
      _Pragma("unroll") for (int n = 0; n < 4; ++n) t_[n] =                             \
          __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bf_[n], af_, z_, 0, 0, 0,    \
                                                           0, 0, 0);                    \
      _Pragma("unroll") for (int n = 0; n < 4; ++n)                                     \
          _Pragma("unroll") for (int i = 0; i < 4; ++i)                                 \
              acc[m][n][i] = __builtin_fmaf(t_[n][i], n < 2 ? c_ : cu_, acc[m][n][i]); \
    }                                                                                   \
  } while (0)

  // prologue: stages 0 .. S-2 in flight, wait for stage 0.  The barriers are
  // plain s_barrier after an explicit vmcnt wait: the generic workgroup
  // barrier would wait for every outstanding load.
  // (the prologue issues stages 0 .. S-2 each followed by its prefetch, so
  // it has the same shape as S-1 loop steps)
  // (alternating loads: stage st is loaded by the waves with wm = st % 2)
  const int wmu = __builtin_amdgcn_readfirstlane(wm);
  if constexpr (kAlt) {
#pragma unroll
    for (int st = 0; st < S - 1; ++st) {
      if (wmu == (st & 1)) {
#pragma unroll
        for (int j = 0; j < kGroupP; ++j) TILE_DMA_P(st, min(st, KB - 1), j);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  } else {
#pragma unroll
    for (int st = 0; st < S - 1; ++st) {
#pragma unroll
      for (int j = 0; j < kGroup; ++j) TILE_DMA_J(st, min(st, KB - 1), j);
      TILE_PREFETCH(min(st + 1, KB - 1));
      __builtin_amdgcn_sched_barrier(0);
    }
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kWait) : "memory");
  }

// the K loop with the first MV row blocks of the wave multiplied
// one K step it: the math of stage st_rd with loads of macro DMA (group size
// NG) and prefetch macro PFM, then this wave's wait (vmcnt W) and the barrier
#define TILE_STEP(MV, DMA, NG, PFM, W)                                                  \
  do {                                                                                  \
    TILE_COMPUTE(st_rd, it, st_ld, min(it + S - 1, KB - 1), min(it + S, KB - 1), MV,     \
                 DMA, NG, PFM);                                                         \
    __builtin_amdgcn_sched_barrier(0);                                                  \
    if (kPrio || kAlt) __builtin_amdgcn_s_setprio(0);                                   \
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W) : "memory");    \
    st_rd = st_rd + 1 == S ? 0 : st_rd + 1;                                             \
    st_ld = st_ld + 1 == S ? 0 : st_ld + 1;                                             \
    ++it;                                                                               \
  } while (0)
// The K loop with the first MV row blocks of the wave multiplied.  With
// alternating loads a wave loads in every other step (step it: the waves with
// wm = (it + S - 1) % 2); the loop body is one loading step and one step
// without loads, entered at the first loading step of this wave, so both
// roles stay in one straight-line body (a branch between two versions of a
// step would join their accumulators every step).
#define TILE_KLOOP(MV)                                                                  \
  do {                                                                                  \
    int st_rd = 0, st_ld = S - 1, it = 0;                                               \
    if constexpr (!kAlt) {                                                              \
      while (it < KB) TILE_STEP(MV, TILE_DMA_J, kGroup, TILE_PREFETCH, kWait);          \
    } else {                                                                            \
      if (wmu != ((S - 1) & 1)) TILE_STEP(MV, TILE_NODMA, 0, TILE_NOPF, 0);              \
      while (it + 1 < KB) {                                                             \
        TILE_STEP(MV, TILE_DMA_P, kGroupP, TILE_NOPF, kWaitLd);                          \
        TILE_STEP(MV, TILE_NODMA, 0, TILE_NOPF, 0);                                      \
      }                                                                                 \
      /* the last step's loads would only repeat the last K block */                    \
      if (it < KB) TILE_STEP(MV, TILE_NODMA, 0, TILE_NOPF, 0);                           \
    }                                                                                   \
  } while (0)
  // A ragged tile (an expert's last M-tile, or a tile taller than the
  // expert's rows) leaves whole 16-row blocks of a wave without pairs: the
  // wave then multiplies only its first MT/2 or MT/4 blocks, or none (their
  // accumulators stay zero and the epilogue stores no row past the tile's).
  const int mv = __builtin_amdgcn_readfirstlane(min(MT, max(0, (nrows - 16 * MT * wm + 15) >> 4)));
  if (mv > MT / 2) TILE_KLOOP(MT);
  else if (mv > MT / 4) TILE_KLOOP(MT / 2);
  else if (mv > 0) TILE_KLOOP(MT / 4);
  else TILE_KLOOP(0);
#undef TILE_KLOOP
#undef TILE_STEP
  // the last steps' (clamped) loads may still be landing in the ring
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");


  // accumulator element (m, n, i) of this lane: tile row 16 MT wm + 16m + r16,
  // column 16n + 4*g4 + i of the wave's 64 columns
  const int wrow = 16 * MT * wm;
  if (!G1) {
    // every wave's loads have drained: the ring is free for the staging
    asm volatile("s_barrier" ::: "memory");
    static_assert(L::RING >= 4 * WM * (16 * MT * 132), "Y staging fits the ring");
    if (wrow0 < p.N_total)
      tile_store_y_lds<MT>(p, acc, row0, nrows, wrow0, wrow, lane, smem + wave * (16 * MT * 132));
    return;
  }

  tile_store_act<MT, BM>(p, acc, amax_l, row0, nrows, nb, wn, wrow, r16, g4);
}

// The large-tile GEMMs as a persistent grid: one workgroup per CU walks the
// work items tile_item(b), tile_item(b + grid), ... (the grid a multiple of
// 8, so every item runs on the XCD the one-shot launch would give it, in the
// same rounds).  The LDS ring runs on across items: the last S-1 K steps of
// an item load the first stages of the next one, and its weight-block scales
// into the other half of a double buffer, so the next item's setup and first
// loads hide behind the current item's math, and the current item's Y
// stores go out while the next item's loads are in flight.  Needs KB >= S.
template <bool G1, int MT, int WM, int S>
__global__ __launch_bounds__(256 * WM) void tile_persist_kernel(GemmParams p) {
  using L = TileLayout<MT, WM, S>;
  constexpr int BM = L::BM;
  static_assert(MT % 4 == 0, "row scales are read four at a time");

  __shared__ float amax_l[4][BM];
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wn = wave & 3;
  const int wm = wave >> 2;
  const int r16 = lane & 15;
  const int g4 = lane >> 4;

  const int n_items = *p.n_items;
  int v = blockIdx.x;
  int item = tile_item(v, n_items);
  if (item < 0) return;

  const int KB = p.KB;
  const int half = wn >> 1;
  constexpr int JA = BM / 8 / (4 * WM);
  constexpr int JB = 8 / WM;
  constexpr int kPfLoads = (BM / kGroupN + 256 + 4 * WM * kWave - 1) / (4 * WM * kWave);
  constexpr int kGroup = JA + JB + 1;
  constexpr int kWait = (S - 2) * (kGroup + kPfLoads) + kPfLoads;
  constexpr bool kPrio = false;  // (see gemm_tile_kernel)
  constexpr bool kAlt = false;
  constexpr int kSpread = MT / 2;
  static_assert(kWait < 64, "vmcnt holds 6 bits");
  static_assert(S >= 2, "LDS ring depth");

  // weight-block scales, double-buffered: buffer q holds sb[0][kb] and
  // sb[1][kb] of one item at sbufs + q * SBP.  Wave 0 fills it with direct
  // loads issued before the item's first stage, so the wait for that stage
  // covers them.
  const int SBP = (2 * KB + kWave - 1) / kWave * kWave;
  float *sbufs = reinterpret_cast<float *>(smem + L::RING);
  auto load_sb = [&](const TileItem &t, int q) {
    if (wave != 0) return;
    const float *s0 = p.B_scale + ((size_t)t.e * (p.N_total / 128) + t.nblk0) * KB;
    const float *s1 = p.B_scale + ((size_t)t.e * (p.N_total / 128) + t.nblk1) * KB;
    for (int c = 0; c < SBP; c += kWave) {
      const int i = c + lane;
      const float *g = i < KB ? s0 + i : s1 + min(i - KB, KB - 1);
      lds_load4(g, reinterpret_cast<uint8_t *>(sbufs + q * SBP + c));
    }
  };

  TileItem ti = tile_decode<G1, BM>(p, item, wn);
  TileSrc<JA, JB, kPfLoads> src;
  tile_sources<G1, MT, WM>(p, ti, wave, lane, src);
  const size_t sa_kb = (size_t)p.sa_kb;
  const int fr = tile_swz(r16);
  const int rd_lo = r16 * 128 + 16 * ((2 * g4) ^ fr);
  const int rd_hi = r16 * 128 + 16 * ((2 * g4 + 1) ^ fr);

  v4f acc[MT][4];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[m][n] = v4f{0.f, 0.f, 0.f, 0.f};

  load_sb(ti, 0);
#pragma unroll
  for (int st = 0; st < S - 1; ++st) {
#pragma unroll
    for (int j = 0; j < kGroup; ++j) TILE_DMA_J(st, min(st, KB - 1), j);
    TILE_PREFETCH(min(st + 1, KB - 1));
    __builtin_amdgcn_sched_barrier(0);
  }
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kWait) : "memory");

  int st_rd = 0, st_ld = S - 1;
  int cur = 0;  // scale buffer of the item being computed
  int row0 = ti.row0, nrows = ti.nrows, wrow0 = ti.wrow0, nb = ti.nb;
  bool more = false;
  const int wrow = 16 * MT * wm;
  while (true) {
    // GEMM1: gate scales at sb_w[kb], up scales at sb_w[KB + kb]
    const float *sb_w = sbufs + cur * SBP + (G1 ? 0 : half * KB);
    for (int it = 0; it < KB; ++it) {
      const bool nxt = it >= KB - (S - 1);  // this step loads the next item
      if (it == KB - (S - 1)) {
        v += gridDim.x;
        const int ni = tile_item(v, n_items);
        more = ni >= 0;
        if (more) {
          ti = tile_decode<G1, BM>(p, ni, wn);
          tile_sources<G1, MT, WM>(p, ti, wave, lane, src);
          load_sb(ti, cur ^ 1);
        }
      }
      // K blocks of this step's loads and prefetches (with no next item the
      // loads repeat the current item's last block: in bounds, never read)
      const int kbl = !nxt ? it + S - 1 : (more ? it + S - 1 - KB : KB - 1);
      const int kbp = !nxt ? min(it + S, KB - 1) : (more ? min(it + S - KB, KB - 1) : KB - 1);
      TILE_COMPUTE(st_rd, it, st_ld, kbl, kbp, MT, TILE_DMA_J, kGroup, TILE_PREFETCH);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kWait) : "memory");
      st_rd = st_rd + 1 == S ? 0 : st_rd + 1;
      st_ld = st_ld + 1 == S ? 0 : st_ld + 1;
    }
    if (G1)
      tile_store_act<MT, BM>(p, acc, amax_l, row0, nrows, nb, wn, wrow, r16, g4);
    else if (wrow0 < p.N_total)
      tile_store_y<MT>(p, acc, row0, nrows, wrow0, wrow, r16, g4);
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < 4; ++n) acc[m][n] = v4f{0.f, 0.f, 0.f, 0.f};
    if (!more) break;
    row0 = ti.row0;
    nrows = ti.nrows;
    wrow0 = ti.wrow0;
    nb = ti.nb;
    cur ^= 1;
  }
  // the last steps' loads may still be landing in the ring
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

#undef TILE_COMPUTE
#undef TILE_PREFETCH
#undef TILE_DMA_J
#undef TILE_DMA_P
#undef TILE_NODMA
#undef TILE_NOPF
#undef TILE_STAGE

template <bool G1, int MT, int WM, int S>
hipError_t launch_tile(const GemmParams &p, int grid, hipStream_t st) {
  using L = TileLayout<MT, WM, S>;
  auto k = gemm_tile_kernel<G1, MT, WM, S>;
  // the dynamic LDS limit is a property of the code object: raise it once,
  // to the size at the largest supported K (512 blocks) or what the CU's
  // 160 KB leave beside the kernel's static arrays, whichever is smaller
  constexpr int kStatic = 4 * L::BM * (int)sizeof(float);
  const int cap = (int)L::bytes(512) < 160 * 1024 - kStatic ? (int)L::bytes(512) : 160 * 1024 - kStatic;
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, cap);
  if (attr != hipSuccess) return attr;
  if (L::bytes(p.KB) > (size_t)cap) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k, dim3(grid), dim3(L::THREADS), L::bytes(p.KB), st, p);
  return hipGetLastError();
}

// The persistent grid: as many workgroups as the device has CUs (a
// multiple of 8, at most the one-shot grid); one fits a CU (its LDS ring).
// (Its dynamic LDS, the ring and the scale double buffer, must leave room for
// the kernel's static row amax in the CU's 160 KB; larger K ranges use the
// one-shot kernel.)
constexpr int kPersistMaxLds = 160 * 1024 - 4 * 256 * (int)sizeof(float);

template <bool G1, int MT, int WM, int S>
hipError_t launch_persist(const GemmParams &p, int grid, hipStream_t st) {
  using L = TileLayout<MT, WM, S>;
  auto k = tile_persist_kernel<G1, MT, WM, S>;
  const size_t lds = (size_t)L::RING + sizeof(float) * 2 * (size_t)((2 * p.KB + kWave - 1) / kWave * kWave);
  if (lds > (size_t)kPersistMaxLds) return launch_tile<G1, MT, WM, S>(p, grid, st);
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, kPersistMaxLds);
  if (attr != hipSuccess) return attr;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return hipErrorInvalidValue;
  int g = cus / 8 * 8;
  if (g < 8) g = 8;
  if (g > grid) g = grid;
  hipLaunchKernelGGL(k, dim3(g), dim3(L::THREADS), lds, st, p);
  return hipGetLastError();
}

template <bool G1, int MT, int WM, int S>
hipError_t launch_any(const GemmParams &p, int grid, hipStream_t st) {
  // (GEMM2 only: GEMM1's 56-step items gained nothing from it, measured at
  // prefill; the eight-wave tiles keep the one-shot launch: with two waves per
  // SIMD the persistent loop's extra state spills registers, measured slower)
  if constexpr (!G1 && WM == 1) {
    if (p.KB >= S) return launch_persist<G1, MT, WM, S>(p, grid, st);
  }
  return launch_tile<G1, MT, WM, S>(p, grid, st);
}

}  // namespace

int gemm_tile_cols() { return kTileCols; }

hipError_t launch_gemm_tile(const GemmParams &p, bool g1, int BM, int grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  if (p.S != 1) return hipErrorInvalidValue;  // full-K items only
  switch (BM) {
    // 64 / 128 rows: three-stage ring (loads two K-steps ahead); the 128-row
    // tiles as 8 waves of 64 rows (two per SIMD, alternating loads: prefill
    // GEMM1 333 -> 324 us against 4 waves of 128 rows before the alternation,
    // GEMM2 179 -> 166 us against 4 waves of 128 rows on the persistent grid)
    case 64: return g1 ? launch_any<true, 4, 1, 3>(p, grid, st) : launch_any<false, 4, 1, 3>(p, grid, st);
    case 128: return g1 ? launch_any<true, 4, 2, 3>(p, grid, st) : launch_any<false, 4, 2, 3>(p, grid, st);
    // 256 rows: 8 waves (two per SIMD), two-stage ring
    case 256: return g1 ? launch_any<true, 8, 2, 2>(p, grid, st) : launch_any<false, 8, 2, 2>(p, grid, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace moe
