// gemm.hip -- stages (3) and (4) of the Fused MoE block (paper Section
// 3.1.1) for small and mid-sized batches, on CDNA4 FP8 matrix cores, and the
// combine of every batch size.
//
//  GEMM1: per resident expert e, rows = the tokens routed to e (gathered
//         through perm_token while the A tile is loaded: the paper's separate
//         gather kernel is folded into the GEMM's loads),
//         G = sum_kb (A_kb W13_kb^T) * sa[row,kb] * sw[n/128,kb]   (fp32)
//         then a = silu(gate) * up, per-row 1x128 amax, scale = amax/448,
//         FP8 re-quantisation -> act [P, I] e4m3 + act_scale.
//  GEMM2: Y = sum_kb (act_kb W2_kb^T) * sa2 * sw2 (fp32), stored as fp16
//         codes with a power-of-two exponent per row and 16 columns
//         (Y [P, H] + Ye [P, H/16]; the scaling is exact)
//  finalize: out[t] = bf16( sum over resident slots j (slot order) of
//            w_j * Y[pair_row[t,j]] ).
//
// Kernels here: the column-split GEMM1 (its K range optionally in two
// halves on separate waves; at most 16 tokens, the permutation rebuilt in
// each workgroup) and its re-quantisation launch, the streaming GEMM2
// (16-row tiles), GEMM2 with the combine in its epilogue (at most 16
// tokens), the LDS-staged GEMM1/GEMM2 for 32-row tiles, the finalize, and
// test hooks.  Larger tiles are in gemm_tile.hip.
//
// Work items of an expert are contiguous; workgroup b is mapped to item
// (b % 8) * ceil(n/8) + b / 8 so neighbouring items land on the same XCD
// (workgroups are dispatched round-robin over the 8 XCDs) and share weight
// panels and A tiles in that XCD's L2.  Each 128-K step is one
// v_mfma_f32_16x16x128_f8f6f4 per 16x16 sub-tile, started from zero and
// promoted into the fp32 accumulator with one FMA by the product of the
// row's activation scale and the block's weight scale.
//
// The LDS-staged kernel: BM rows x 256 columns x 128 K per step, 4 waves;
// in GEMM1 wave w owns gate columns [32w, 32w+32) and the matching up
// columns of the 128-wide intermediate block, so SwiGLU pairs live in the
// same lane.  A and B tiles are staged through LDS (double buffered, rows
// padded to 144 bytes).
#include "moe_device.h"
#include "scatter_device.h"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = 144;  // 128 data bytes + 16 pad
constexpr int kBN = 256;

template <int BM>
struct Layout {
  static constexpr int A = BM * kRowBytes;
  static constexpr int B = kBN * kRowBytes;
  static constexpr int SA = BM * 4;
  static constexpr int STAGE = A + B + SA + 16;
  static constexpr int AMAX = 4 * BM * 4;
  static constexpr int TB = 4 * 1028;  // tile_base copy (El <= 1024)
  static constexpr int TOTAL = 2 * STAGE + AMAX + TB;
};

__device__ __forceinline__ v8i lds_frag(const uint8_t *p) {
  const v4i lo = *reinterpret_cast<const v4i *>(p);
  const v4i hi = *reinterpret_cast<const v4i *>(p + 16);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

template <int BM, bool G1>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmParams p) {
  using L = Layout<BM>;
  constexpr int MT = BM / 16;
  constexpr int A_CHUNKS = BM * 8;
  constexpr int A_PER = (A_CHUNKS + kThreads - 1) / kThreads;
  constexpr int B_PER = kBN * 8 / kThreads;

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  float *amax_lds = reinterpret_cast<float *>(smem + 2 * L::STAGE);
  int *tb = reinterpret_cast<int *>(smem + 2 * L::STAGE + L::AMAX);

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;

  const int n_items = *p.n_items;
  const int per_xcd = (n_items + 7) / 8;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if ((int)(blockIdx.x >> 3) >= per_xcd || item >= n_items) return;

  for (int i = tid; i <= p.El; i += kThreads) tb[i] = p.tile_base[i];
  __syncthreads();

  // ---- decode the work item
  const int X = p.NB * p.S;
  const int qt = item / X;
  int lo = 0, hi = p.El;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tb[mid] <= qt) lo = mid; else hi = mid;
  }
  const int e = lo;
  const int nt_e = tb[e + 1] - tb[e];
  const int local = item - tb[e] * X;
  const int mt_idx = local % nt_e;
  const int rest = local / nt_e;
  const int s = rest % p.S;
  const int nb = rest / p.S;
  const int seg0 = p.expert_offsets[e];
  const int seg1 = p.expert_offsets[e + 1];
  const int row0 = seg0 + mt_idx * BM;
  const int nrows = min(BM, seg1 - row0);
  const int kb0 = (s * p.KB) / p.S;
  const int kb1 = ((s + 1) * p.KB) / p.S;
  const size_t K = (size_t)p.K;

  // ---- per-thread load assignments (fixed over the K loop)
  const uint8_t *a_src[A_PER];
  int a_dst[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    const int idx = tid + i * kThreads;
    const int r = idx >> 3, c = idx & 7;
    const int rr = min(r, nrows - 1);
    const int src = G1 ? p.perm_token[row0 + rr] : row0 + rr;
    a_src[i] = p.A + (size_t)src * K + c * 16;
    a_dst[i] = (idx < A_CHUNKS) ? r * kRowBytes + c * 16 : -1;
  }
  const float *sa_src = nullptr;
  if (tid < BM) {
    const int rr = min(tid, nrows - 1);
    const int src = G1 ? p.perm_token[row0 + rr] : row0 + rr;
    sa_src = p.A_scale + (size_t)src * p.KB;
  }
  const uint8_t *Bexp = p.B + (size_t)e * p.N_total * K;
  const uint8_t *b_src[B_PER];
#pragma unroll
  for (int i = 0; i < B_PER; ++i) {
    const int r = (tid >> 3) + 32 * i, c = tid & 7;
    int brow;
    if (G1)
      brow = (r < 128) ? nb * 128 + r : p.I + nb * 128 + (r - 128);
    else
      brow = min(nb * kBN + r, p.N_total - 1);  // ragged last block (H % 256 == 128)
    b_src[i] = Bexp + (size_t)brow * K + c * 16;
  }
  const float *sb_src = nullptr;
  if (tid < 2) {
    const int nblk = G1 ? (tid == 0 ? nb : p.I / 128 + nb) : min(2 * nb + tid, p.N_total / 128 - 1);
    sb_src = p.B_scale + ((size_t)e * (p.N_total / 128) + nblk) * p.KB;
  }

  u32x4 ra[A_PER], rb[B_PER];
  float rsa = 0.0f, rsb = 0.0f;
#define MOE_GLOAD(kb)                                                                   \
  do {                                                                                  \
    _Pragma("unroll") for (int i = 0; i < A_PER; ++i) if (a_dst[i] >= 0) ra[i] =        \
        *reinterpret_cast<const u32x4 *>(a_src[i] + (size_t)(kb) * 128);                \
    _Pragma("unroll") for (int i = 0; i < B_PER; ++i) rb[i] =                           \
        *reinterpret_cast<const u32x4 *>(b_src[i] + (size_t)(kb) * 128);                \
    if (tid < BM) rsa = sa_src[kb];                                                     \
    if (tid < 2) rsb = sb_src[kb];                                                      \
  } while (0)
#define MOE_LSTORE(buf)                                                                 \
  do {                                                                                  \
    uint8_t *st_ = smem + (buf) * L::STAGE;                                             \
    _Pragma("unroll") for (int i = 0; i < A_PER; ++i) if (a_dst[i] >= 0)                \
        *reinterpret_cast<u32x4 *>(st_ + a_dst[i]) = ra[i];                              \
    _Pragma("unroll") for (int i = 0; i < B_PER; ++i)                                   \
        *reinterpret_cast<u32x4 *>(st_ + L::A + ((tid >> 3) + 32 * i) * kRowBytes +     \
                                   (tid & 7) * 16) = rb[i];                              \
    float *sa_ = reinterpret_cast<float *>(st_ + L::A + L::B);                          \
    if (tid < BM) sa_[tid] = rsa;                                                       \
    if (tid < 2) sa_[BM + tid] = rsb;                                                   \
  } while (0)

  // LDS rows of this wave's four 16-column B sub-tiles
  int brow_lds[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
    brow_lds[nt] = G1 ? ((nt < 2 ? 0 : 128) + 32 * wave + 16 * (nt & 1)) : (64 * wave + 16 * nt);

  v4f acc[MT][4];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[m][nt] = v4f{0.f, 0.f, 0.f, 0.f};

  const int frag_off = (lane >> 4) * 32;
  const int r16 = lane & 15;

  MOE_GLOAD(kb0);
  MOE_LSTORE(0);
  __syncthreads();
  for (int kb = kb0; kb < kb1; ++kb) {
    const int cur = (kb - kb0) & 1;
    const bool more = kb + 1 < kb1;
    if (more) MOE_GLOAD(kb + 1);

    const uint8_t *st = smem + cur * L::STAGE;
    const uint8_t *As = st;
    const uint8_t *Bs = st + L::A;
    const float *sa = reinterpret_cast<const float *>(st + L::A + L::B);
    const float sb0 = sa[BM], sb1 = sa[BM + 1];
    v8i bf[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) bf[nt] = lds_frag(Bs + (brow_lds[nt] + r16) * kRowBytes + frag_off);
    float sbn[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
      sbn[nt] = G1 ? (nt < 2 ? sb0 : sb1) : (wave < 2 ? sb0 : sb1);
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const v8i af = lds_frag(As + (m * 16 + r16) * kRowBytes + frag_off);
      const float4 sav = *reinterpret_cast<const float4 *>(sa + m * 16 + 4 * (lane >> 4));
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const v4f z = {0.f, 0.f, 0.f, 0.f};
        const v4f t = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf[nt], z, 0, 0, 0, 0, 0, 0);
        acc[m][nt][0] = __builtin_fmaf(t[0], sav.x * sbn[nt], acc[m][nt][0]);
        acc[m][nt][1] = __builtin_fmaf(t[1], sav.y * sbn[nt], acc[m][nt][1]);
        acc[m][nt][2] = __builtin_fmaf(t[2], sav.z * sbn[nt], acc[m][nt][2]);
        acc[m][nt][3] = __builtin_fmaf(t[3], sav.w * sbn[nt], acc[m][nt][3]);
      }
    }
    if (more) MOE_LSTORE(cur ^ 1);
    __syncthreads();
  }

#undef MOE_GLOAD
#undef MOE_LSTORE

  // accumulator element (m, nt, i) of this lane is row m*16 + 4*(lane/16) + i,
  // column r16 of sub-tile nt
  if (!G1) {
    if (nb * kBN + 64 * wave >= p.H) return;  // this wave's columns are past H
    // Y as fp16 codes, one exponent per row and 16-column chunk (sub-tile
    // nt): the chunk's columns are the 16 lanes of the row's lane group
    const int HC = p.H / kYChunk;
    const int c0 = nb * kBN + 64 * wave;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = m * 16 + 4 * (lane >> 4) + i;
        int ex[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          float mx = fabsf(acc[m][nt][i]);
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
          ex[nt] = y16_exponent(mx);
        }
        if (r < nrows) {
          uint16_t *yrow = p.Y + (size_t)(row0 + r) * p.H + c0 + r16;
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) yrow[16 * nt] = y16_code(acc[m][nt][i], ex[nt]);
          if (r16 < 4) {
            int eg = ex[0];
#pragma unroll
            for (int nt = 1; nt < 4; ++nt) eg = r16 == nt ? ex[nt] : eg;
            p.Ye[(size_t)(row0 + r) * HC + c0 / kYChunk + r16] = (int8_t)eg;
          }
        }
      }
    return;
  }

  // SwiGLU in registers: sub-tiles 0/1 are gate, 2/3 the matching up columns
  float av[MT][4][2];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        av[m][i][h] = swiglu_spec(acc[m][h][i], acc[m][2 + h][i]);
      }
  // per-row amax over the 128-column block: 16 lanes x 2 columns x 4 waves
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = fmaxf(fabsf(av[m][i][0]), fabsf(av[m][i][1]));
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
      if (r16 == 0) amax_lds[wave * BM + m * 16 + 4 * (lane >> 4) + i] = mx;
    }
  __syncthreads();
  const int IB = p.I / 128;
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = m * 16 + 4 * (lane >> 4) + i;
      const float amax = fmaxf(fmaxf(amax_lds[r], amax_lds[BM + r]),
                               fmaxf(amax_lds[2 * BM + r], amax_lds[3 * BM + r]));
      const float scale = (amax > 0.0f) ? amax / 448.0f : 1.0f;
      if (r < nrows) {
        const uint32_t q2 = (amax > 0.0f)
                                ? e4m3x2_rne_sat(av[m][i][0] / scale, av[m][i][1] / scale)
                                : 0u;
        uint8_t *arow = p.act + (size_t)(row0 + r) * p.I + nb * 128 + 32 * wave + r16;
        arow[0] = (uint8_t)(q2 & 0xff);
        arow[16] = (uint8_t)(q2 >> 8);
        if (wave == 0 && r16 == 0) p.act_scale[(size_t)(row0 + r) * IB + nb] = scale;
      }
    }
}

// GEMM2 for small batches (BM = 16): the weight fragments are streamed from
// HBM straight into registers through a D-stage prefetch ring, with no LDS
// round trip and no barrier in the K loop.  Prefetches are issued
// unconditionally (past the end they re-read the last K block) so the
// compiler can keep D loads in flight instead of draining the queue at every
// branch.  8 waves; wave w owns output columns [16w, 16w+16) of a 128-wide
// block (one weight fragment per step: more waves stream at once, which is
// what the chip's streaming rate needs).  Activation and weight block scales
// of the whole K range are staged in LDS once.  The per-element arithmetic (MFMA block products, promotion
// order) is the same as the other GEMM kernels'.
constexpr int kStreamWaves = 8;

// ALDS: the item's whole A tile (16 rows x its K range) is staged in LDS once
// (rows padded by 16 bytes) instead of every wave loading it from L2 at each
// K step; used when the tile fits (GEMM2 at small batches).
template <int D, bool ALDS>
__global__ __launch_bounds__(kStreamWaves * kWave) void gemm2_stream_kernel(GemmParams p) {
  constexpr int NW = kStreamWaves;
  extern __shared__ __attribute__((aligned(16))) float scales[];  // sa[16][KB], sb[KB] (+1 row), A tile

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int r16 = lane & 15;
  const int frag_off = (lane >> 4) * 32;

  const int n_items = *p.n_items;
  const int per_xcd = (n_items + 7) / 8;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if ((int)(blockIdx.x >> 3) >= per_xcd || item >= n_items) return;

  // the item's M-tile entry: expert, its first M-tile, first row, rows
  const int X = p.NB * p.S;
  const int4 te = reinterpret_cast<const int4 *>(p.tile_tab)[__builtin_amdgcn_readfirstlane(item / X)];
  const int e = te.x;
  const int nt_e = (te.w + 15) / 16;
  const int local = item - te.y * X;
  const int mt_idx = local % nt_e;
  const int rest = local / nt_e;
  const int s = rest % p.S;
  const int nb = rest / p.S;
  const int seg0 = te.z;
  const int seg1 = te.z + te.w;
  const int row0 = seg0 + mt_idx * 16;
  const int nrows = min(16, seg1 - row0);
  const int kb0 = (s * p.KB) / p.S;
  const int kb1 = ((s + 1) * p.KB) / p.S;
  const int n = kb1 - kb0;
  const size_t K = (size_t)p.K;
  const int KB = p.KB;

  // B rows of the wave's sub-tile (inside one 128-row scale block).  They
  // depend on the expert and column block only: the first D weight loads go
  // out before the item's rows, scales and activation tile are looked up.
  const int brow0 = nb * 128 + 16 * wave + r16;
  const uint8_t *Bexp = p.B + (size_t)e * p.N_total * K;
  const uint8_t *b_ptr0 = Bexp + (size_t)brow0 * K + frag_off;
  v8i ra[D], rb0[D];
#pragma unroll
  for (int d = 0; d < D; ++d) rb0[d] = *reinterpret_cast<const v8i *>(b_ptr0 + (size_t)(kb0 + min(d, n - 1)) * 128);

  // stage the scales: sa[r][kb] of the tile's rows, sb[0/1][kb] of the blocks
  float *sa_l = scales;
  float *sb_l = scales + 16 * KB;
  for (int i = tid; i < 16 * KB; i += NW * kWave) {
    const int r = i / KB, kb = i % KB;
    const int rr = min(r, nrows - 1);
    const int src = row0 + rr;
    sa_l[i] = p.A_scale[(size_t)src * KB + kb];
  }
  {
    const float *sb0 = p.B_scale + ((size_t)e * (p.N_total / 128) + nb) * KB;
    for (int i = tid; i < KB; i += NW * kWave) sb_l[i] = sb0[i];
  }

  // A fragment source: the lane's row (ragged tails repeat the last row)
  const int arow = min(r16, nrows - 1);
  const int asrc = row0 + arow;
  const uint8_t *a_ptr = p.A + (size_t)asrc * K + frag_off;

  // A tile in LDS: row r, K step kb -> a_l + r * astride + (kb - kb0) * 128
  uint8_t *a_l = reinterpret_cast<uint8_t *>(scales) + ((18 * KB * 4 + 15) & ~15);
  const int astride = n * 128 + 16;
  if (ALDS) {
    const int chunks = 16 * n * 8;  // 16-byte chunks
    for (int c = tid; c < chunks; c += NW * kWave) {
      const int r = c / (n * 8), off = (c % (n * 8)) * 16;
      const int rr = min(r, nrows - 1);
      const int src = row0 + rr;
      *reinterpret_cast<u32x4 *>(a_l + r * astride + off) =
          *reinterpret_cast<const u32x4 *>(p.A + (size_t)src * K + (size_t)kb0 * 128 + off);
    }
  }
  const uint8_t *a_lds = a_l + r16 * astride + frag_off;

#define MOE_SLOAD(d, kb)                                                  \
  do {                                                                    \
    if (!ALDS) ra[d] = *reinterpret_cast<const v8i *>(a_ptr + (size_t)(kb) * 128); \
    rb0[d] = *reinterpret_cast<const v8i *>(b_ptr0 + (size_t)(kb) * 128); \
  } while (0)

  if (!ALDS) {
#pragma unroll
    for (int d = 0; d < D; ++d) ra[d] = *reinterpret_cast<const v8i *>(a_ptr + (size_t)(kb0 + min(d, n - 1)) * 128);
  }
  __syncthreads();  // scales staged

  v4f acc0 = {0.f, 0.f, 0.f, 0.f};
  const int srow = 4 * (lane >> 4);
  for (int base = 0; base < n; base += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int it = base + d;
      if (it < n) {
        const int kb = kb0 + it;
        const v4f z = {0.f, 0.f, 0.f, 0.f};
        const v8i af = ALDS ? lds_frag(a_lds + it * 128) : ra[d];
        const v4f t0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, rb0[d], z, 0, 0, 0, 0, 0, 0);
        const float s0 = sb_l[kb];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sa = sa_l[(srow + i) * KB + kb];
          acc0[i] = __builtin_fmaf(t0[i], sa * s0, acc0[i]);
        }
      }
      MOE_SLOAD(d, kb0 + min(it + D, n - 1));
    }
  }
#undef MOE_SLOAD

  // Y as fp16 codes: the wave's 16 columns of a row are one chunk, held by
  // the 16 lanes of the row's lane group
  const int c0 = nb * 128 + 16 * wave;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = srow + i;
    float mx = fabsf(acc0[i]);
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    const int ex = y16_exponent(mx);
    if (r < nrows) {
      p.Y[(size_t)(row0 + r) * p.H + c0 + r16] = y16_code(acc0[i], ex);
      if (r16 == 0) p.Ye[(size_t)(row0 + r) * (p.H / kYChunk) + c0 / kYChunk] = (int8_t)ex;
    }
  }
}

// GEMM1 for small batches, split over columns: a work item is one 16-row
// M-tile and 32 intermediate columns, so a handful of resident experts still
// yields several work items per CU (HBM streaming needs all 256 CUs busy;
// splitting K across workgroups would need a cross-workgroup reduction before
// the SwiGLU).  One wave streams the gate and up rows of both 16-column halves of
// the item against one A fragment (the tile's 16 gathered rows): four MFMAs
// per 128-K step with a D-stage register prefetch ring (unconditional, so
// loads stay in flight); SwiGLU pairs then sit in the same lane.  Four weight
// fragments per A fragment (fewer A loads per weight byte) measured faster
// than two waves of two fragments each.
// GU (the fewest rows per expert): items of 16 columns, wave 0 the gate rows
// and wave 1 the up rows, so twice as many waves stream (the chip's streaming
// rate needs many waves per CU); the up half meets the gate half in LDS.  The
// SwiGLU output goes to a_buf [P, I] fp32 and requant_kernel (the next launch)
// re-quantises it: no cross-workgroup synchronisation.  The re-quantisation
// applies the large-tile epilogue's operations (amax, scale, rounding) to the
// same fp32 values; with the K range in two halves (KS = 2) those sums differ
// from one pass over K by fp32 rounding order only.
// Stage (2) inside the narrow GEMM1 for batches of at most 16 tokens (T K <=
// 256 pairs): every workgroup rebuilds the permutation from the routing ids
// in LDS -- bits[e] marks the tokens holding local expert e, so a pair's row
// is offset[e] plus the count of its expert's tokens below it, the same
// stable (expert, token) order as the permutation kernel -- and workgroup 0
// writes the permuted-order arrays the later launches read.  Returns the
// GEMM1 work-item count.  Every thread of the 128-thread workgroup calls it.
constexpr int kNarrowPermPairs = 256;  // routed pairs the in-kernel permutation takes

template <int NT>
__device__ int narrow_permute(const GemmParams &p, int *tb, int *off, unsigned *bits,
                              int (*wsum)[2]) {
  constexpr int PPT = kNarrowPermPairs / NT;  // pairs per thread
  static_assert(PPT * NT == kNarrowPermPairs, "pairs split evenly over the threads");
  const PermuteParams &q = p.perm;
  const int tid = threadIdx.x;
  const int TK = q.T * q.K;
  int le[PPT], tk[PPT];
#pragma unroll
  for (int u = 0; u < PPT; ++u) {
    const int pr = tid + NT * u;
    const int x = q.topk_ids[min(pr, TK - 1)] - q.offset;
    le[u] = (pr < TK && x >= 0 && x < q.El) ? x : -1;
    tk[u] = pr / q.K;
  }
  for (int e = tid; e < q.El; e += NT) bits[e] = 0u;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < PPT; ++u)
    if (le[u] >= 0) atomicOr(&bits[le[u]], 1u << tk[u]);
  __syncthreads();
  // offsets and M-tile prefix: each thread a contiguous run of experts
  const int per = (q.El + NT - 1) / NT;
  const int e0 = tid * per;
  int tot_run = 0, tiles_run = 0;
  for (int e = e0; e < e0 + per && e < q.El; ++e) {
    const int n = __popc(bits[e]);
    tot_run += n;
    tiles_run += (n + q.BM - 1) / q.BM;
  }
  int run_start, tile_start, P, n_tiles;
  scatter_block_scan2<NT>(tot_run, tiles_run, wsum, run_start, tile_start, P, n_tiles);
  const bool writer = blockIdx.x == 0;
  int acc = run_start, tacc = tile_start;
  for (int e = e0; e < e0 + per && e < q.El; ++e) {
    const int n = __popc(bits[e]);
    off[e] = acc;
    tb[e] = tacc;
    if (writer) {
      q.expert_offsets[e] = acc;
      q.tile_base[e] = tacc;
      const int nt = (n + q.BM - 1) / q.BM;
      for (int t = 0; t < nt; ++t)
        reinterpret_cast<int4 *>(q.tile_tab)[tacc + t] = make_int4(e, tacc, acc, n);
    }
    acc += n;
    tacc += (n + q.BM - 1) / q.BM;
  }
  if (tid == 0) {
    off[q.El] = P;
    tb[q.El] = n_tiles;
    if (writer) {
      q.expert_offsets[q.El] = P;
      q.tile_base[q.El] = n_tiles;
      q.n_items[0] = n_tiles * q.items_per_tile1;
      q.n_items[1] = n_tiles * q.items_per_tile2;
    }
  }
  __syncthreads();
  if (writer) {
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
      const int pr = tid + NT * u;
      if (pr < TK) {
        int row = -1;
        if (le[u] >= 0) {
          row = off[le[u]] + __popc(bits[le[u]] & ((1u << tk[u]) - 1u));
          q.perm_token[row] = tk[u];
          q.perm_pair[row] = pr;
        }
        q.pair_row[pr] = row;
      }
    }
  }
  return n_tiles * q.items_per_tile1;
}

template <int D, bool GU, bool PERM, int KS>
__global__ __launch_bounds__((GU ? 2 : 1) * KS * kWave) void gemm1_narrow_kernel(GemmParams p) {
  constexpr int NR = GU ? 2 : 1;  // waves per K range (gate / up)
  constexpr int NT = NR * KS * kWave;
  constexpr int kCols = GU ? 16 : 32;  // intermediate columns per item
  static_assert(!PERM || GU, "in-kernel permutation: gate/up-split items");
  static_assert(KS == 1 || KS == 2, "K split in one or two ranges");
  __shared__ int tb[PERM ? 1028 : 1];            // M-tile prefix (PERM)
  __shared__ int pm_off[PERM ? 1028 : 1];        // expert offsets (PERM)
  __shared__ unsigned pm_bits[PERM ? 1024 : 1];  // tokens of each local expert (PERM)
  __shared__ int pm_tok[PERM ? 16 : 1];          // the item's rows' tokens (PERM)
  __shared__ int pm_wsum[PERM ? NT / kWave : 1][2];
  extern __shared__ __attribute__((aligned(16))) float scales[];  // sa[16][KB], sb[2][KB]

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int r16 = lane & 15;
  const int frag_off = (lane >> 4) * 32;

  const int n_items = PERM ? narrow_permute<NT>(p, tb, pm_off, pm_bits, pm_wsum) : *p.n_items;
  const int per_xcd = (n_items + 7) / 8;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if ((int)(blockIdx.x >> 3) >= per_xcd || item >= n_items) return;

  // the item's expert, its M-tile count and first M-tile, its rows: from the
  // workgroup's own permutation (PERM), else from the item's M-tile entry
  const int X = p.NB;  // column groups per M-tile
  const int qt = item / X;
  int e, nt_e, tb_e, seg0, seg1;
  if (PERM) {
    int lo = 0, hi = p.El;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (tb[mid] <= qt) lo = mid; else hi = mid;
    }
    e = lo;
    nt_e = tb[e + 1] - tb[e];
    tb_e = tb[e];
    seg0 = pm_off[e];
    seg1 = pm_off[e + 1];
  } else {
    const int4 te = reinterpret_cast<const int4 *>(p.tile_tab)[__builtin_amdgcn_readfirstlane(qt)];
    e = te.x;
    nt_e = (te.w + 15) / 16;
    tb_e = te.y;
    seg0 = te.z;
    seg1 = te.z + te.w;
  }
  const int local = item - tb_e * X;
  const int mt_idx = local % nt_e;
  const int j = local / nt_e;       // kCols-column group
  const int blk = j * kCols / 128;  // its 128-column block
  const int row0 = seg0 + mt_idx * 16;
  const int nrows = min(16, seg1 - row0);
  const int KB = p.KB;
  const size_t K = (size_t)p.K;
  // the wave's role (GU: 0 gate, 1 up) and its K blocks [kb0, kb1): with
  // KS > 1 the K ranges run on separate waves, their sums added in fixed
  // order (range 0, then 1, ...) before the SwiGLU
  const int role = GU ? (wave % NR) : 0;
  const int kh = wave / NR;
  const int KBh = (KB + KS - 1) / KS;
  const int kb0 = min(kh * KBh, KB), kb1 = min(kb0 + KBh, KB);
  if (PERM) {
    // the expert's rows in token order: row r is its r-th marked token (at
    // most 16 tokens, so one M-tile); ragged tails repeat the last row
    if (tid < 16) {
      unsigned m = pm_bits[e];
      const int r = min(tid, nrows - 1);
      for (int k = 0; k < r; ++k) m &= m - 1u;
      pm_tok[tid] = __builtin_ctz(m);
    }
    __syncthreads();
  }
  // token of row r of the tile (r < 16, clamped by the caller)
  auto row_token = [&](int r) { return PERM ? pm_tok[r] : p.perm_token[row0 + r]; };

  float *sa_l = scales;
  float *sb_l = scales + 16 * KB;
  const float *sg = p.B_scale + ((size_t)e * (p.N_total / 128) + blk) * KB;
  const float *su = p.B_scale + ((size_t)e * (p.N_total / 128) + p.I / 128 + blk) * KB;

  // Weight fragments: GU, wave 0 streams the 16 gate rows of its columns and
  // wave 1 the 16 up rows (rg0); otherwise one wave streams the gate and up
  // rows of two 16-column halves.  On the fast path their first D loads are
  // issued after the scale loads and before the scale stores: returns are in
  // order, so the stores wait for the scales only while the weight stream is
  // under way.
  const int col0 = j * kCols + r16, col1 = col0 + 16;
  const uint8_t *bexp = p.B + (size_t)e * p.N_total * K;
  const uint8_t *g0 = bexp + ((size_t)col0 + (GU && role ? p.I : 0)) * K + frag_off;
  const uint8_t *g1 = bexp + (size_t)col1 * K + frag_off;
  const uint8_t *u0 = g0 + (size_t)p.I * K;
  const uint8_t *u1 = g1 + (size_t)p.I * K;
  v8i rg0[D], rg1[D], ru0[D], ru1[D];
#define MOE_WPREFETCH()                                                     \
  do {                                                                      \
    _Pragma("unroll") for (int d = 0; d < D; ++d) {                         \
      const size_t o = (size_t)max(min(kb0 + d, kb1 - 1), 0) * 128;         \
      rg0[d] = *reinterpret_cast<const v8i *>(g0 + o);                      \
      if (!GU) {                                                            \
        rg1[d] = *reinterpret_cast<const v8i *>(g1 + o);                    \
        ru0[d] = *reinterpret_cast<const v8i *>(u0 + o);                    \
        ru1[d] = *reinterpret_cast<const v8i *>(u1 + o);                    \
      }                                                                     \
    }                                                                       \
  } while (0)
  // the lane's activation row (ragged tails repeat the last row) and its
  // first D fragments
  const int asrc = row_token(min(r16, nrows - 1));
  const uint8_t *a_ptr = p.A + (size_t)asrc * K + frag_off;
  v8i ra[D];
  constexpr int kSaPer = 16;  // scale registers per thread on the fast path
  if (!GU && 16 * KB <= kSaPer * NT && KB <= NT) {
    // branch-free (clamped indices) so that each group of loads goes out
    // back to back: the tile's token ids, then the activation fragments and
    // the activation and weight scales, then the weights; one wait per
    // dependent step.  (Measured at 32-column items: 193 -> 188 us at
    // T = 256; the two-wave 16-column items are faster with the loop below.)
    const int last = 16 * KB - 1;
    int srcv[kSaPer];
#pragma unroll
    for (int q = 0; q < kSaPer; ++q) {
      const int r = min(tid + q * NT, last) / KB;
      srcv[q] = row_token(min(r, nrows - 1));
    }
#pragma unroll
    for (int d = 0; d < D; ++d)
      ra[d] = *reinterpret_cast<const v8i *>(a_ptr + (size_t)max(min(kb0 + d, kb1 - 1), 0) * 128);
    float sav[kSaPer];
#pragma unroll
    for (int q = 0; q < kSaPer; ++q) {
      const int kb = min(tid + q * NT, last) % KB;
      sav[q] = p.A_scale[(size_t)srcv[q] * KB + kb];
    }
    const float sgv = sg[min(tid, KB - 1)];
    const float suv = su[min(tid, KB - 1)];
    MOE_WPREFETCH();
#pragma unroll
    for (int q = 0; q < kSaPer; ++q) {
      const int i = tid + q * NT;
      if (i < 16 * KB) sa_l[i] = sav[q];
    }
    if (tid < KB) {
      sb_l[tid] = sgv;
      sb_l[KB + tid] = suv;
    }
  } else {
    for (int i = tid; i < 16 * KB; i += NT) {
      const int r = i / KB, kb = i % KB;
      const int src = row_token(min(r, nrows - 1));
      sa_l[i] = p.A_scale[(size_t)src * KB + kb];
    }
    for (int i = tid; i < KB; i += NT) {
      sb_l[i] = sg[i];
      sb_l[KB + i] = su[i];
    }
#pragma unroll
    for (int d = 0; d < D; ++d)
      ra[d] = *reinterpret_cast<const v8i *>(a_ptr + (size_t)max(min(kb0 + d, kb1 - 1), 0) * 128);
    MOE_WPREFETCH();
  }
#undef MOE_WPREFETCH

  if (GU) {
    // wave 0 streams the 16 gate rows, wave 1 the matching 16 up rows; the up
    // accumulators meet the gate ones in LDS for the SwiGLU
    __shared__ float up_l[4][kWave];
    __shared__ float half_l[KS > 1 ? KS - 1 : 1][NR][4][kWave];
    const int col = col0;
    const float *sbw = sb_l + (role ? KB : 0);
    __syncthreads();  // scales staged

    v4f acc = {0.f, 0.f, 0.f, 0.f};
    const int srow = 4 * (lane >> 4);
    for (int base = kb0; base < kb1; base += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int kb = base + d;
        if (kb < kb1) {
          const v4f z = {0.f, 0.f, 0.f, 0.f};
          const v4f t = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ra[d], rg0[d], z, 0, 0, 0, 0, 0, 0);
          const float sw = sbw[kb];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float sa = sa_l[(srow + i) * KB + kb];
            acc[i] = __builtin_fmaf(t[i], sa * sw, acc[i]);
          }
        }
        const size_t o = (size_t)min(kb + D, kb1 - 1) * 128;
        ra[d] = *reinterpret_cast<const v8i *>(a_ptr + o);
        rg0[d] = *reinterpret_cast<const v8i *>(g0 + o);
      }
    }
    if (KS > 1) {
      if (kh > 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) half_l[kh - 1][role][i][lane] = acc[i];
      }
      __syncthreads();
      if (kh == 0) {
#pragma unroll
        for (int h = 0; h < KS - 1; ++h)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] += half_l[h][role][i][lane];
      }
    }
    if (kh == 0 && role == 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) up_l[i][lane] = acc[i];
    }
    __syncthreads();
    if (kh == 0 && role == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = srow + i;
        if (r < nrows) p.abuf[(size_t)(row0 + r) * p.I + col] = swiglu_spec(acc[i], up_l[i][lane]);
      }
    }
    return;
  }

  // one wave, the item's two 16-column sub-tiles: four weight fragments (gate
  // and up of each) against one A fragment per K step
  __syncthreads();  // scales staged

  v4f ag0 = {0.f, 0.f, 0.f, 0.f}, ag1 = ag0, au0 = ag0, au1 = ag0;
  const int srow = 4 * (lane >> 4);
  for (int base = kb0; base < kb1; base += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int kb = base + d;
      if (kb < kb1) {
        const v4f z = {0.f, 0.f, 0.f, 0.f};
        const v4f tg0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ra[d], rg0[d], z, 0, 0, 0, 0, 0, 0);
        const v4f tg1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ra[d], rg1[d], z, 0, 0, 0, 0, 0, 0);
        const v4f tu0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ra[d], ru0[d], z, 0, 0, 0, 0, 0, 0);
        const v4f tu1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(ra[d], ru1[d], z, 0, 0, 0, 0, 0, 0);
        const float sg = sb_l[kb], su = sb_l[KB + kb];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sa = sa_l[(srow + i) * KB + kb];
          ag0[i] = __builtin_fmaf(tg0[i], sa * sg, ag0[i]);
          ag1[i] = __builtin_fmaf(tg1[i], sa * sg, ag1[i]);
          au0[i] = __builtin_fmaf(tu0[i], sa * su, au0[i]);
          au1[i] = __builtin_fmaf(tu1[i], sa * su, au1[i]);
        }
      }
      const size_t o = (size_t)min(kb + D, kb1 - 1) * 128;
      ra[d] = *reinterpret_cast<const v8i *>(a_ptr + o);
      rg0[d] = *reinterpret_cast<const v8i *>(g0 + o);
      rg1[d] = *reinterpret_cast<const v8i *>(g1 + o);
      ru0[d] = *reinterpret_cast<const v8i *>(u0 + o);
      ru1[d] = *reinterpret_cast<const v8i *>(u1 + o);
    }
  }
  if (KS > 1) {
    // the other K ranges' sums join the first's through LDS, in range order
    __shared__ float half_l[KS > 1 ? KS - 1 : 1][4][4][kWave];
    if (kh > 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        half_l[kh - 1][0][i][lane] = ag0[i];
        half_l[kh - 1][1][i][lane] = ag1[i];
        half_l[kh - 1][2][i][lane] = au0[i];
        half_l[kh - 1][3][i][lane] = au1[i];
      }
    }
    __syncthreads();
    if (kh > 0) return;
#pragma unroll
    for (int h = 0; h < KS - 1; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ag0[i] += half_l[h][0][i][lane];
        ag1[i] += half_l[h][1][i][lane];
        au0[i] += half_l[h][2][i][lane];
        au1[i] += half_l[h][3][i][lane];
      }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = srow + i;
    if (r < nrows) {
      p.abuf[(size_t)(row0 + r) * p.I + col0] = swiglu_spec(ag0[i], au0[i]);
      p.abuf[(size_t)(row0 + r) * p.I + col1] = swiglu_spec(ag1[i], au1[i]);
    }
  }
}

// Re-quantisation of the column-split GEMM1 output: rows [0, P) of a_buf
// (P = expert_offsets[El], on the device), one 128-column block per 16
// threads: amax, scale = amax / 448, e4m3 codes -- the same operations on the
// same fp32 values as the single-item GEMM1 epilogue.
__global__ __launch_bounds__(256) void requant_kernel(GemmParams p) {
  const int P = p.expert_offsets[p.El];
  const int IB = p.I / 128;
  const int g = blockIdx.x * 16 + (threadIdx.x >> 4);  // (row, block) pair
  if (g >= P * IB) return;
  const int row = g / IB, blk = g % IB;
  const int c0 = (threadIdx.x & 15) * 8;
  const float *src = p.abuf + (size_t)row * p.I + blk * 128 + c0;
  const float4 x0 = *reinterpret_cast<const float4 *>(src);
  const float4 x1 = *reinterpret_cast<const float4 *>(src + 4);
  const float v[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
  float mx = 0.0f;
#pragma unroll
  for (int c = 0; c < 8; ++c) mx = fmaxf(mx, fabsf(v[c]));
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  const float scale = (mx > 0.0f) ? mx / 448.0f : 1.0f;
  uint2 w2 = {0u, 0u};
  if (mx > 0.0f) {
    w2.x = e4m3x2_rne_sat(v[0] / scale, v[1] / scale) | (e4m3x2_rne_sat(v[2] / scale, v[3] / scale) << 16);
    w2.y = e4m3x2_rne_sat(v[4] / scale, v[5] / scale) | (e4m3x2_rne_sat(v[6] / scale, v[7] / scale) << 16);
  }
  *reinterpret_cast<uint2 *>(p.act + (size_t)row * p.I + blk * 128 + c0) = w2;
  if (c0 == 0) p.act_scale[(size_t)row * IB + blk] = scale;
}

// The combine: out[t] = bf16(sum over the token's resident slots, in slot
// order, of w_j * Y[pair_row[t, j]]), Y read back from its fp16 codes and
// chunk exponents (exact).  All K pair rows and weights are loaded first,
// then the Y codes and exponents of the resident slots, so a token costs two
// dependent round trips, not 2K.  Workgroup (t, y) holds token t, and its
// thread i the CW consecutive columns starting at CW (y * blockDim + i)
// (CW = 16: one exponent byte and 32 bytes of codes per slot; CW = 8: half a
// chunk): the token's slots are uniform over the workgroup (absent slots
// branch around their loads without splitting a wave) and a wave's loads of
// one slot are contiguous.  KM >= K slots (4, 8 or 16).
constexpr int kFinalizeMaxThreads = 512;
template <int KM, int CW>
__global__ __launch_bounds__(kFinalizeMaxThreads) void finalize_kernel(FinalizeParams p) {
  constexpr int NV = CW / 8;  // 16-byte pieces per slot
  const int HC = p.H / kYChunk;
  const int t = blockIdx.x;
  const int c0 = (blockIdx.y * blockDim.x + threadIdx.x) * CW;
  if (c0 >= p.H) return;
  int pr[KM];
  float w[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    const int jj = min(j, p.K - 1);
    pr[j] = j < p.K ? p.pair_row[(size_t)t * p.K + jj] : -1;
    w[j] = p.topk_w[(size_t)t * p.K + jj];
  }
  uint4 yc[KM][NV];
  int ye[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
#pragma unroll
    for (int v = 0; v < NV; ++v) yc[j][v] = uint4{0u, 0u, 0u, 0u};
    ye[j] = 0;
    if (pr[j] >= 0) {
      const uint4 *yr = reinterpret_cast<const uint4 *>(p.Y + (size_t)pr[j] * p.H + c0);
#pragma unroll
      for (int v = 0; v < NV; ++v) yc[j][v] = yr[v];
      ye[j] = p.Ye[(size_t)pr[j] * HC + c0 / kYChunk];
    }
  }
  float acc[CW];
#pragma unroll
  for (int c = 0; c < CW; ++c) acc[c] = 0.0f;
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (pr[j] >= 0) {
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        const uint4 q = yc[j][c >> 3];
        const uint32_t u = (c & 7) < 2 ? q.x : ((c & 7) < 4 ? q.y : ((c & 7) < 6 ? q.z : q.w));
        const float y = y16_value((uint16_t)(u >> (16 * (c & 1))), ye[j]);
        acc[c] = __builtin_fmaf(w[j], y, acc[c]);
      }
    }
  }
  uint4 *orow = reinterpret_cast<uint4 *>(p.out + (size_t)t * p.H + c0);
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const float *a = acc + 8 * v;
    orow[v] = uint4{(uint32_t)f32_to_bf16_rne(a[0]) | ((uint32_t)f32_to_bf16_rne(a[1]) << 16),
                    (uint32_t)f32_to_bf16_rne(a[2]) | ((uint32_t)f32_to_bf16_rne(a[3]) << 16),
                    (uint32_t)f32_to_bf16_rne(a[4]) | ((uint32_t)f32_to_bf16_rne(a[5]) << 16),
                    (uint32_t)f32_to_bf16_rne(a[6]) | ((uint32_t)f32_to_bf16_rne(a[7]) << 16)};
  }
}

// GEMM2 and the weighted combine of stage (4) in one kernel, for batches of at
// most 16 tokens (every resident expert then has a single 16-row tile).  A
// workgroup owns 16 output columns of every token.  Each tile's K range is cut
// into C chunks, and chunk u of the batch goes to wave u % NW: the wave
// streams the 16 weight rows of its columns against the chunk's activation
// rows (one MFMA per 128-K block, promoted by the row and block scales, as in
// the other GEMM kernels) and at the chunk's end adds w_pair * partial into
// its own LDS accumulator at the pair's token.  The waves' accumulators are
// then summed in wave order and every output element is rounded to bf16
// once.  No fp32 Y goes to memory and no combine launch follows; the
// summation order is fixed, so the output is deterministic.  The chunks keep
// the waves evenly loaded whatever the number of resident experts.  The
// activation rows (when all P fit), their scales and the tiles' weight-block
// scales are staged in LDS once, so the K loop's only global loads are the
// weight fragments.
constexpr int kCombineWaves = 8;
constexpr int kCombineTokens = 16;
constexpr int kCombineStageBytes = 48 * 1024;  // LDS for the activation rows

struct CombineLayout {
  int P_max, KB, stage_rows, astride;
  __host__ __device__ CombineLayout(int P_max_, int I) : P_max(P_max_), KB(I / 128) {
    astride = I + 16;
    stage_rows = kCombineStageBytes / astride;
  }
  __host__ __device__ int sa() const { return 5 * P_max; }                 // [P_max, KB] f32
  __host__ __device__ int sw() const { return sa() + P_max * KB; }         // [tiles, KB] f32
  __host__ __device__ int act() const { return sw() + P_max * KB; }        // rows, in ints
  __host__ __device__ size_t bytes() const {
    return sizeof(int) * (size_t)act() + (size_t)stage_rows * astride;
  }
};

template <int D>
__global__ __launch_bounds__(kCombineWaves * kWave) void gemm2_combine_kernel(GemmParams p,
                                                                             CombineParams c) {
  constexpr int NW = kCombineWaves;
  constexpr int NT = NW * kWave;
  __shared__ float acc_l[NW][kCombineTokens][16];
  extern __shared__ __attribute__((aligned(16))) int dyn[];
  const CombineLayout Ly(p.P_max, p.K);
  int *t_e = dyn;                    // per tile: expert, first row, rows
  int *t_row0 = dyn + p.P_max;
  int *t_n = dyn + 2 * p.P_max;
  int *r_tok = dyn + 3 * p.P_max;    // per permuted row: token, weight
  float *r_w = reinterpret_cast<float *>(dyn + 4 * p.P_max);
  float *sa_l = reinterpret_cast<float *>(dyn + Ly.sa());
  float *sw_l = reinterpret_cast<float *>(dyn + Ly.sw());
  uint8_t *a_l = reinterpret_cast<uint8_t *>(dyn + Ly.act());

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int r16 = lane & 15;
  const int srow = 4 * (lane >> 4);
  const int frag_off = (lane >> 4) * 32;
  const int col0 = blockIdx.x * 16;
  const int KB = p.KB;
  const size_t K = (size_t)p.K;

  // the tiles' entries (expert, first row, rows), loaded for every possible
  // tile together with the tile count (at most 16 tokens: one tile per
  // resident expert, so at most min(P_max, El); entries past the count are
  // left over from other batches and never used)
  for (int i = tid; i < NW * kCombineTokens * 16; i += NT) (&acc_l[0][0][0])[i] = 0.0f;
  const int n_tiles = p.tile_base[p.El];
  const int P = p.expert_offsets[p.El];
  for (int q = tid; q < min(p.P_max, p.El); q += NT) {
    const int4 te = reinterpret_cast<const int4 *>(p.tile_tab)[q];
    const int row0 = te.z + 16 * (q - te.y);
    t_e[q] = te.x;
    t_row0[q] = row0;
    t_n[q] = min(16, te.z + te.w - row0);
  }
  __syncthreads();

  // this wave's steps: unit j of the wave is chunk u = wave + NW j of the
  // batch, i.e. tile u / C, K blocks [(u % C) L, (u % C) L + L)
  const int L = KB / c.C;
  const int n_units = n_tiles * c.C;
  const int my_units = n_units > wave ? (n_units - wave + NW - 1) / NW : 0;
  const int steps = my_units * L;
  const bool alds = P <= Ly.stage_rows;
  const uint8_t *wcol = p.B + ((size_t)col0 + r16) * K + frag_off;
  const size_t w_exp = (size_t)p.N_total * K;

  v8i ra[D], rb[D];
  // loads of step s (clamped to the last step, so every load is in bounds)
  auto issue = [&](int d, int s) {
    s = min(s, steps - 1);
    const int u = wave + NW * (s / L);
    const int q = u / c.C;
    const int kb = (u % c.C) * L + s % L;
    rb[d] = *reinterpret_cast<const v8i *>(wcol + t_e[q] * w_exp + (size_t)kb * 128);
    if (!alds) {
      const int arow = t_row0[q] + min(r16, t_n[q] - 1);
      ra[d] = *reinterpret_cast<const v8i *>(p.A + (size_t)arow * K + (size_t)kb * 128 + frag_off);
    }
  };
  if (steps > 0) {
#pragma unroll
    for (int d = 0; d < D; ++d) issue(d, d);
  }

  // stage the rows' tokens and weights, the activation scales, the tiles'
  // weight-block scales and (when they fit) the activation rows
  for (int r = tid; r < P; r += NT) {
    const int pp = c.perm_pair[r];
    r_tok[r] = pp / c.K;
    r_w[r] = c.topk_w[pp];
  }
  for (int i = tid; i < P * KB; i += NT) sa_l[i] = p.A_scale[i];
  for (int i = tid; i < n_tiles * KB; i += NT) {
    const int q = i / KB, kb = i % KB;
    sw_l[i] = p.B_scale[((size_t)t_e[q] * (p.N_total / 128) + col0 / 128) * KB + kb];
  }
  if (alds) {
    const int cpr = p.K / 16;  // 16-byte chunks per row
    for (int i = tid; i < P * cpr; i += NT) {
      const int r = i / cpr, off = (i % cpr) * 16;
      *reinterpret_cast<u32x4 *>(a_l + r * Ly.astride + off) =
          *reinterpret_cast<const u32x4 *>(p.A + (size_t)r * K + off);
    }
  }
  __syncthreads();

  if (steps > 0) {
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    for (int base = 0; base < steps; base += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int s = base + d;
        if (s < steps) {
          const int u = wave + NW * (s / L);
          const int q = u / c.C;
          const int kb = (u % c.C) * L + s % L;
          const int row0 = t_row0[q], n = t_n[q];
          const v8i af = alds ? lds_frag(a_l + (row0 + min(r16, n - 1)) * Ly.astride + kb * 128 + frag_off)
                              : ra[d];
          const v4f z = {0.f, 0.f, 0.f, 0.f};
          const v4f t = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, rb[d], z, 0, 0, 0, 0, 0, 0);
          const float sw = sw_l[q * KB + kb];
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc[i] = __builtin_fmaf(t[i], sa_l[(row0 + min(srow + i, n - 1)) * KB + kb] * sw, acc[i]);
          if (s % L == L - 1) {
            // the chunk is complete: weight its rows into their tokens
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int r = srow + i;
              if (r < n) {
                float *a = &acc_l[wave][r_tok[row0 + r]][r16];
                *a = __builtin_fmaf(r_w[row0 + r], acc[i], *a);
              }
              acc[i] = 0.0f;
            }
          }
          issue(d, s + D);
        }
      }
    }
  }
  __syncthreads();
  if (tid < kCombineTokens * 16) {
    const int t = tid >> 4, col = tid & 15;
    if (t < c.T) {
      float sum = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) sum += acc_l[w][t][col];
      c.out[(size_t)t * p.H + col0 + col] = f32_to_bf16_rne(sum);
    }
  }
}

template <int BM, bool G1>
hipError_t launch_gemm_bm(const GemmParams &p, int grid, hipStream_t st) {
  auto k = gemm_kernel<BM, G1>;
  const int lds = Layout<BM>::TOTAL;
  // raise the dynamic LDS limit once per kernel instantiation (per process;
  // the attribute is a property of the code object, not of the device)
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), lds, st, p);
  return hipGetLastError();
}

constexpr int kStreamDepth = 4;

// GEMM2 for 16-row tiles: the streaming kernel (its item's A tile in LDS
// when it is at most 32 KB)
hipError_t launch_gemm2_stream(const GemmParams &p, int grid, hipStream_t st) {
  const int n_max = (p.KB + p.S - 1) / p.S;
  const size_t a_bytes = 16 * ((size_t)n_max * 128 + 16);
  const bool alds = a_bytes <= 32768 + 256;
  const size_t lds = ((sizeof(float) * 18 * (size_t)p.KB + 15) & ~(size_t)15) + (alds ? a_bytes : 0);
  if (alds)
    hipLaunchKernelGGL((gemm2_stream_kernel<kStreamDepth, true>), dim3(grid), dim3(kStreamWaves * kWave),
                       lds, st, p);
  else
    hipLaunchKernelGGL((gemm2_stream_kernel<kStreamDepth, false>), dim3(grid), dim3(kStreamWaves * kWave),
                       lds, st, p);
  return hipGetLastError();
}

// Test hook: the FP8 encoder of the re-quantisation epilogue, elementwise.
__global__ void e4m3_encode_kernel(const float *x, uint8_t *q, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 2;
  if (i >= n) return;
  const float b = (i + 1 < n) ? x[i + 1] : 0.0f;
  const uint32_t c = e4m3x2_rne_sat(x[i], b);
  q[i] = (uint8_t)(c & 0xff);
  if (i + 1 < n) q[i + 1] = (uint8_t)(c >> 8);
}

// Test hook: one v_mfma_f32_16x16x128_f8f6f4 per case with the operand and
// result lane layouts the GEMM kernels use.  a, b: [n, 16, 128] e4m3 (rows of
// A and of W); d: [n, 16, 16] fp32 with d[i][j] = sum_k a[i][k] * b[j][k].
__global__ __launch_bounds__(64) void mfma_block_kernel(const uint8_t *a, const uint8_t *b,
                                                        float *d) {
  const int lane = threadIdx.x;
  const size_t c = blockIdx.x;
  const int r16 = lane & 15, off = (lane >> 4) * 32;
  const v8i af = *reinterpret_cast<const v8i *>(a + c * 2048 + r16 * 128 + off);
  const v8i bf = *reinterpret_cast<const v8i *>(b + c * 2048 + r16 * 128 + off);
  const v4f z = {0.f, 0.f, 0.f, 0.f};
  const v4f t = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf, z, 0, 0, 0, 0, 0, 0);
#pragma unroll
  for (int i = 0; i < 4; ++i) d[c * 256 + (4 * (lane >> 4) + i) * 16 + r16] = t[i];
}

}  // namespace

hipError_t launch_debug_mfma_block(const uint8_t *a, const uint8_t *b, float *d, int64_t n,
                                   hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(mfma_block_kernel, dim3((unsigned)n), dim3(64), 0, st, a, b, d);
  return hipGetLastError();
}

// GEMM1 with the LDS-staged kernel: 32-row tiles (16-row batches use the
// column-split kernel, 64 rows and more the large-tile kernels)
hipError_t launch_gemm1(const GemmParams &p, int BM, int grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  return BM == 32 ? launch_gemm_bm<32, true>(p, grid, st) : hipErrorInvalidValue;
}
template <int KS>
hipError_t launch_gemm1_narrow_ks(const GemmParams &p, int grid, bool gate_up_split, bool permute,
                                  hipStream_t st) {
  const size_t lds = sizeof(float) * 18 * (size_t)p.KB;
  if (permute) {
    if (!gate_up_split || p.perm.T * p.perm.K > kNarrowPermPairs || p.perm.T > 16 ||
        p.perm.El > 1024 || p.perm.BM != 16)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm1_narrow_kernel<kStreamDepth, true, true, KS>), dim3(grid), dim3(2 * KS * kWave),
                       lds, st, p);
    return hipGetLastError();
  } else if (gate_up_split) {
    hipLaunchKernelGGL((gemm1_narrow_kernel<kStreamDepth, true, false, KS>), dim3(grid), dim3(2 * KS * kWave),
                       lds, st, p);
    return hipGetLastError();
  }
  {
    hipLaunchKernelGGL((gemm1_narrow_kernel<kStreamDepth, false, false, KS>), dim3(grid), dim3(KS * kWave),
                       lds, st, p);
  }
  return hipGetLastError();
}
hipError_t launch_gemm1_narrow(const GemmParams &p, int grid, bool gate_up_split, bool permute,
                               int k_split, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  if (k_split == 1) return launch_gemm1_narrow_ks<1>(p, grid, gate_up_split, permute, st);
  if (k_split == 2) return launch_gemm1_narrow_ks<2>(p, grid, gate_up_split, permute, st);
  return hipErrorInvalidValue;
}
int gemm1_narrow_cols(bool gate_up_split) { return gate_up_split ? 16 : 32; }
hipError_t launch_requant(const GemmParams &p, int P_max, hipStream_t st) {
  const int pairs = P_max * (p.I / 128);
  if (pairs <= 0) return hipSuccess;
  hipLaunchKernelGGL(requant_kernel, dim3((pairs + 15) / 16), dim3(256), 0, st, p);
  return hipGetLastError();
}
// GEMM2 for 16- and 32-row tiles (64 rows and more: the large-tile kernels)
hipError_t launch_gemm2(const GemmParams &p, int BM, int grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  if (p.S != 1) return hipErrorInvalidValue;  // Y holds one K plane
  switch (BM) {
    case 16: return launch_gemm2_stream(p, grid, st);
    case 32: return launch_gemm_bm<32, false>(p, grid, st);
    default: return hipErrorInvalidValue;
  }
}

template <int CW>
hipError_t launch_finalize_cw(const FinalizeParams &p, hipStream_t st) {
  // 16 columns per thread: one workgroup per token where the row fits
  // (H = 7168: 448 threads).  8 columns: column blocks of 256 threads (when
  // most slots are absent, more and shorter workgroups per token measured
  // faster: prefill 28.2 -> 25.8 us against 512-thread blocks)
  const int cap = CW == 16 ? kFinalizeMaxThreads : 256;
  const int per_token = p.H / CW;
  const int nt = per_token < cap ? (per_token + kWave - 1) / kWave * kWave : cap;
  const dim3 grid(p.T, (per_token + nt - 1) / nt);
  if (p.K <= 4)
    hipLaunchKernelGGL((finalize_kernel<4, CW>), grid, dim3(nt), 0, st, p);
  else if (p.K <= 8)
    hipLaunchKernelGGL((finalize_kernel<8, CW>), grid, dim3(nt), 0, st, p);
  else
    hipLaunchKernelGGL((finalize_kernel<16, CW>), grid, dim3(nt), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeParams &p, hipStream_t st) {
  if (p.T == 0) return hipSuccess;
  return p.cw == 16 ? launch_finalize_cw<16>(p, st) : launch_finalize_cw<8>(p, st);
}

int combine_max_tokens() { return kCombineTokens; }
bool combine_fits(int P_max, int I) { return CombineLayout(P_max, I).bytes() <= 96 * 1024; }

hipError_t launch_gemm2_combine(const GemmParams &p, const CombineParams &c, hipStream_t st) {
  if (c.T <= 0) return hipSuccess;
  if (c.T > kCombineTokens || p.KB % c.C || p.H % 16) return hipErrorInvalidValue;
  auto k = gemm2_combine_kernel<kStreamDepth>;
  const size_t lds = CombineLayout(p.P_max, p.K).bytes();
  if (lds > 96 * 1024) return hipErrorInvalidValue;
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(k, dim3(p.H / 16), dim3(kCombineWaves * kWave), lds, st, p, c);
  return hipGetLastError();
}

hipError_t launch_debug_e4m3_encode(const float *x, uint8_t *q, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t threads = (n + 1) / 2;
  hipLaunchKernelGGL(e4m3_encode_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st,
                     x, q, n);
  return hipGetLastError();
}

}  // namespace moe
