// indexer.hip -- the DSA TopK Indexer (paper Section 3.1.3): for each
// sequence, score every cached token against the query's 64 heads,
//   score(j) = sum over heads h of ReLU(q_h . k_j) * w_h,
// and return the TopK best tokens.  The key cache is paged (PS tokens per
// page) in FP8 e4m3 with one fp32 scale per token; q is FP8 e4m3.
//
// The returned indices must be exactly the reference's, so the scores follow
// one fixed fp32 sequence (scalar fused multiply-adds, as the paper's kernel
// keeps a scalar fp32 dot product for the same reason):
//   kd[d]  = decode(k[d]) * scale                       (one rounding)
//   dot_h  = fmaf chain over d ascending from 0 of decode(q[h][d]) * kd[d]
//   score  = fmaf chain over h ascending from 0 of (dot_h > 0 ? dot_h : 0) * w_h
// Selection: larger score first, equal scores to the lower position; the
// selected tokens come back in ascending position order as physical cache
// indices page * PS + slot, the row padded with -1.  A sequence of at most
// TopK tokens returns all of them without scoring (the device reads
// seq_lens and takes that path itself, no host round trip).
//
// Two kernels: dsa_scores_kernel (4 or 16 threads per token, 16 or 4 heads each; the
// token's 128 key values live in registers, the 64 query rows in LDS, read as
// broadcasts) and
// dsa_select_kernel (one 1024-thread workgroup per sequence: a four-pass
// 8-bit radix select of the TopK-th key, then an ordered compaction).  For
// batches that may hold long sequences, the four histogram passes are spread
// over many workgroups per sequence (dsa_hist_kernel, global histograms
// cleared by the score kernel) and the select kernel only replays them.
//
// Built with -ffp-contract=off: only the explicit fmaf calls fuse.
#include "moe_device.h"

namespace moe {
namespace {

constexpr int kNH = 64;    // query heads
constexpr int kD = 128;    // head dimension
constexpr int kScoreThreads = 256;
constexpr int kSelThreads = 1024;
constexpr int kSelPer = 16;  // positions per select thread per chunk
constexpr int kSmallSelThreads = 256;  // select workgroup for block tables of at most 4,096 tokens

// Device-side inputs are clamped into range (a sequence length into
// [0, max_pages * PS], a page id into [0, num_pages)), so bad values give
// wrong indices, never an out-of-bounds access.
__device__ __forceinline__ int seq_len_of(const DsaParams &p, int b) {
  return min(max(p.seq_lens[b], 0), p.max_len);
}
__device__ __forceinline__ int page_of(const DsaParams &p, int page) {
  return min(max(page, 0), p.num_pages - 1);
}

// TPW tokens per workgroup, 256 / TPW threads per token, each the dot
// products of its share of the heads (independent chains, interleaved four at
// a time); the ReLU'd dots go through LDS and the token's first thread runs
// the head chain in order.  64 tokens per workgroup for batches with long
// sequences; 16 when the batch is short, so that a sequence of a few
// thousand tokens still spreads over a hundred CUs and more.  The arithmetic
// per token is the same either way.
typedef float v2f __attribute__((ext_vector_type(2)));

template <int TPW>
__global__ __launch_bounds__(kScoreThreads) void dsa_scores_kernel(DsaParams p, int force) {
  constexpr int kTokPerWG = TPW;
  constexpr int kHeadsPerThread = kNH / (kScoreThreads / TPW);
  static_assert(kHeadsPerThread % 4 == 0, "heads in groups of four");
  // 16-token workgroups: a wave spans 16 head groups, so its query reads are
  // not broadcasts and LDS bandwidth bounds the loop: the query stays in e4m3
  // codes there (a quarter of the bytes), decoded exactly where it is used.
  // 64-token workgroups: a wave is one head group (broadcast reads) and the
  // loop is bound by the fused multiply-adds: the query is decoded once.
  constexpr bool kCodes = TPW < kWave;
  __shared__ __attribute__((aligned(16))) uint8_t q_c[kCodes ? kNH * kD : 16];
  __shared__ __attribute__((aligned(16))) float q_l[kCodes ? 4 : kNH * kD];
  __shared__ float w_l[kNH];
  __shared__ float r_l[kTokPerWG][kNH + 1];
  const int b = blockIdx.y;
  const int L = seq_len_of(p, b);
  const int j0 = blockIdx.x * kTokPerWG;
  if (blockIdx.x == 0 && p.hist) {  // the radix histograms of this sequence start at zero
    for (int i = threadIdx.x; i < 4 * 256; i += kScoreThreads)
      p.hist[((size_t)(i / 256) * p.B + b) * 256 + (i % 256)] = 0;
  }
  if (j0 >= L || (!force && L <= p.topk)) return;  // whole workgroup
  const int tid = threadIdx.x;
  const int tl = tid & (kTokPerWG - 1);  // token of the workgroup
  const int qq = tid / kTokPerWG;        // head quarter

  // the query's 64 x 128 codes (32 per thread), as codes or decoded exactly
  // to fp32
  {
    const uint8_t *qb = p.q + (size_t)b * kNH * kD;
    const u32x4 a = *reinterpret_cast<const u32x4 *>(qb + tid * 32);
    const u32x4 c = *reinterpret_cast<const u32x4 *>(qb + tid * 32 + 16);
    if (kCodes) {
      *reinterpret_cast<u32x4 *>(&q_c[tid * 32]) = a;
      *reinterpret_cast<u32x4 *>(&q_c[tid * 32 + 16]) = c;
    } else {
      float *dst = &q_l[tid * 32];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int wa = (int)a[i], wc = (int)c[i];
        dst[4 * i + 0] = __builtin_amdgcn_cvt_f32_fp8(wa, 0);
        dst[4 * i + 1] = __builtin_amdgcn_cvt_f32_fp8(wa, 1);
        dst[4 * i + 2] = __builtin_amdgcn_cvt_f32_fp8(wa, 2);
        dst[4 * i + 3] = __builtin_amdgcn_cvt_f32_fp8(wa, 3);
        dst[16 + 4 * i + 0] = __builtin_amdgcn_cvt_f32_fp8(wc, 0);
        dst[16 + 4 * i + 1] = __builtin_amdgcn_cvt_f32_fp8(wc, 1);
        dst[16 + 4 * i + 2] = __builtin_amdgcn_cvt_f32_fp8(wc, 2);
        dst[16 + 4 * i + 3] = __builtin_amdgcn_cvt_f32_fp8(wc, 3);
      }
    }
    if (tid < kNH) w_l[tid] = p.weights[(size_t)b * kNH + tid];
  }

  // this thread's token: its 128 dequantised key values in registers
  const int j = min(j0 + tl, L - 1);  // past the end: a repeat, not stored
  const int page = page_of(p, p.block_table[(size_t)b * p.max_pages + j / p.PS]);
  const size_t tok = (size_t)page * p.PS + (j % p.PS);
  const uint8_t *krow = p.k_cache + tok * kD;
  const float scale = p.k_scale[tok];
  float kd[kD];
#pragma unroll
  for (int c = 0; c < kD / 16; ++c) {
    const u32x4 v = *reinterpret_cast<const u32x4 *>(krow + 16 * c);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int wv = (int)v[i];
      kd[16 * c + 4 * i + 0] = __builtin_amdgcn_cvt_f32_fp8(wv, 0) * scale;
      kd[16 * c + 4 * i + 1] = __builtin_amdgcn_cvt_f32_fp8(wv, 1) * scale;
      kd[16 * c + 4 * i + 2] = __builtin_amdgcn_cvt_f32_fp8(wv, 2) * scale;
      kd[16 * c + 4 * i + 3] = __builtin_amdgcn_cvt_f32_fp8(wv, 3) * scale;
    }
  }
  __syncthreads();

  // each head's dot: its own fused multiply-add chain over d ascending
  constexpr int kHG = 4;
  for (int h0 = qq * kHeadsPerThread; h0 < (qq + 1) * kHeadsPerThread; h0 += kHG) {
    float dot[kHG];
#pragma unroll
    for (int g = 0; g < kHG; ++g) dot[g] = 0.0f;
#pragma unroll
    for (int d = 0; d < kD; d += 4) {
#pragma unroll
      for (int g = 0; g < kHG; ++g) {
        float4 q4;
        if (kCodes) {
          const int c4 = *reinterpret_cast<const int *>(&q_c[(h0 + g) * kD + d]);
          const v2f lo = __builtin_amdgcn_cvt_pk_f32_fp8(c4, false);  // codes d, d+1
          const v2f hi = __builtin_amdgcn_cvt_pk_f32_fp8(c4, true);   // codes d+2, d+3
          q4 = float4{lo[0], lo[1], hi[0], hi[1]};
        } else {
          q4 = *reinterpret_cast<const float4 *>(&q_l[(h0 + g) * kD + d]);
        }
        dot[g] = __builtin_fmaf(q4.x, kd[d + 0], dot[g]);
        dot[g] = __builtin_fmaf(q4.y, kd[d + 1], dot[g]);
        dot[g] = __builtin_fmaf(q4.z, kd[d + 2], dot[g]);
        dot[g] = __builtin_fmaf(q4.w, kd[d + 3], dot[g]);
      }
    }
#pragma unroll
    for (int g = 0; g < kHG; ++g) r_l[tl][h0 + g] = dot[g] > 0.0f ? dot[g] : 0.0f;
  }
  __syncthreads();
  // the head chain, in order
  if (qq == 0 && j0 + tl < L) {
    float acc = 0.0f;
#pragma unroll 8
    for (int h = 0; h < kNH; ++h) acc = __builtin_fmaf(r_l[tl][h], w_l[h], acc);
    p.scores[(size_t)b * p.max_len + j0 + tl] = acc;
  }
}

// fp32 -> an unsigned key with the same order (-0 taken as +0, so equal
// scores get equal keys)
__device__ __forceinline__ uint32_t score_key(float v) {
  uint32_t u = __float_as_uint(v);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive scan over the wave with DPP: a window of four lanes (row_shr 1,
// 2, 3 of the original values), row_shr 4 and 8 into the upper lanes of each
// 16-lane row, then row_bcast 15 and 31 across rows.
template <int kCtrl, int kRows, int kBanks>
__device__ __forceinline__ int sel_dpp(int v) {
  return __builtin_amdgcn_update_dpp(0, v, kCtrl, kRows, kBanks, false);
}
__device__ __forceinline__ int wave_scan_incl(int v) {
  int x = v + sel_dpp<0x111, 0xf, 0xf>(v);
  x += sel_dpp<0x112, 0xf, 0xf>(v);
  x += sel_dpp<0x113, 0xf, 0xf>(v);
  x += sel_dpp<0x114, 0xf, 0xe>(x);
  x += sel_dpp<0x118, 0xf, 0xc>(x);
  x += sel_dpp<0x142, 0xa, 0xf>(x);
  x += sel_dpp<0x143, 0xc, 0xf>(x);
  return x;
}

// Block-wide exclusive prefix sums of two values over the workgroup's
// threads in order: the prefixes and the totals.  Every thread must call it.
template <int NW>
__device__ __forceinline__ void block_excl_sum2(int a, int b, int (*wave_sum)[2], int &pa, int &pb,
                                                int &ta, int &tb) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int xa = wave_scan_incl(a), xb = wave_scan_incl(b);
  __syncthreads();  // previous users of wave_sum are done
  if (lane == kWave - 1) {
    wave_sum[wave][0] = xa;
    wave_sum[wave][1] = xb;
  }
  __syncthreads();
  int ba = 0, bb = 0, aa = 0, ab = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int ca = wave_sum[w][0], cb = wave_sum[w][1];
    ba += (w < wave) ? ca : 0;
    bb += (w < wave) ? cb : 0;
    aa += ca;
    ab += cb;
  }
  pa = ba + xa - a;
  pb = bb + xb - b;
  ta = aa;
  tb = ab;
}

// One radix-select step, run by one wave: given the 256 bin counts of the
// keys matching `prefix` under `mask` (summed over `nsub` sub-histograms
// `stride` ints apart) and the `left`-th largest of them sought, fix the
// next 8 bits (at `shift`) and the count still sought inside that bin.  Lane
// l holds bins 4l .. 4l+3; suffix sums over the lanes pick the bin.
struct SelState {
  uint32_t prefix, mask;
  int left;
};

__device__ __forceinline__ void resolve_bin(const int *bins, int nsub, int stride, int shift,
                                            SelState *st) {
  const int lane = threadIdx.x & (kWave - 1);
  int c[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int s = 0;
    for (int w = 0; w < nsub; ++w) s += bins[w * stride + 4 * lane + i];
    c[i] = s;
  }
  const int mine = c[0] + c[1] + c[2] + c[3];
  const int incl = wave_scan_incl(mine);
  const int suffix = __builtin_amdgcn_readlane(incl, kWave - 1) - incl + mine;  // lanes >= lane
  const int above = suffix - mine;  // keys in bins of higher lanes
  const int left = st->left;
  const uint32_t prefix = st->prefix, mask = st->mask;
  __builtin_amdgcn_wave_barrier();
  if (above < left && suffix >= left) {  // exactly one lane
    int acc = above, bin = 4 * lane;
    for (int i = 3; i >= 0; --i) {
      if (acc + c[i] >= left) {
        bin = 4 * lane + i;
        break;
      }
      acc += c[i];
    }
    st->prefix = prefix | ((uint32_t)bin << shift);
    st->mask = mask | (255u << shift);
    st->left = left - acc;
  }
}

// Keys of positions [j_begin, j_end) matching the state, counted into the
// per-wave LDS histograms by byte `shift`.
__device__ __forceinline__ void count_keys(const float *sc, int j_begin, int j_end, int nthreads,
                                           const SelState &st, int shift, int *my_hist) {
  for (int j4 = j_begin + (int)threadIdx.x; j4 < j_end; j4 += 4 * nthreads) {
    uint32_t k[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = j4 + i * nthreads;
      k[i] = j < j_end ? score_key(sc[j]) : 0u;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (j4 + i * nthreads < j_end && (k[i] & st.mask) == st.prefix)
        atomicAdd(&my_hist[(k[i] >> shift) & 255u], 1);
  }
}

// Long sequences, pass `pass` of the radix select spread over the grid's x
// dimension: each workgroup first replays the earlier passes from their
// global histograms (every workgroup reaches the same state), then counts
// its slice of positions and adds its bins to the pass's global histogram.
// Sequences of at most topk tokens return at once.
constexpr int kHistThreads = 256;

__global__ __launch_bounds__(kHistThreads) void dsa_hist_kernel(DsaParams p, int pass) {
  __shared__ int hist[kHistThreads / kWave][256];
  __shared__ SelState st;
  const int b = blockIdx.y;
  const int L = seq_len_of(p, b);
  if (L <= p.topk) return;
  const int tid = threadIdx.x, wave = tid / kWave;
  const int per = (L + gridDim.x - 1) / gridDim.x;
  const int j_begin = blockIdx.x * per;
  const int j_end = min(L, j_begin + per);
  if (j_begin >= j_end) return;
  if (tid == 0) st = SelState{0u, 0u, p.topk};
  for (int i = tid; i < (kHistThreads / kWave) * 256; i += kHistThreads) (&hist[0][0])[i] = 0;
  __syncthreads();
  for (int q = 0; q < pass; ++q) {
    if (wave == 0) resolve_bin(p.hist + ((size_t)q * p.B + b) * 256, 1, 0, 24 - 8 * q, &st);
    __syncthreads();
  }
  const SelState s0 = st;
  count_keys(p.scores + (size_t)b * p.max_len, j_begin, j_end, kHistThreads, s0, 24 - 8 * pass,
             hist[wave]);
  __syncthreads();
  int *g = p.hist + ((size_t)pass * p.B + b) * 256;
  for (int i = tid; i < 256; i += kHistThreads) {
    int c = 0;
    for (int w = 0; w < kHistThreads / kWave; ++w) c += hist[w][i];
    if (c) atomicAdd(&g[i], c);
  }
}

// Ordered compaction of a run of kPer consecutive positions per thread
// (thread t: j0 .. j0 + kPer - 1): position j is taken if its key beats the
// threshold, or equals it and fewer than `need` equal keys come before it; its
// output slot is (keys above the threshold before j) + min(equal keys before
// j, need), from one block scan of the two counts, plus the counts of the
// positions before the workgroup's run (gt_before, eq_before).  Every thread
// of the workgroup must call it (it contains barriers).
template <int NW, int kPer>
__device__ __forceinline__ void compact_slice(const DsaParams &p, int L, int j0, uint32_t thr, int need,
                                              int gt_before, int eq_before, const uint32_t (&kr)[kPer],
                                              int (*wave_cnt)[2], int32_t *out, const int32_t *bt) {
  int ngt = 0, neq = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const bool in = j0 + i < L;
    ngt += (in && kr[i] > thr) ? 1 : 0;
    neq += (in && kr[i] == thr) ? 1 : 0;
  }
  // the cache index of each position: the positions are consecutive, so one
  // division gives the first (page, slot); with pages of at least kPer tokens
  // they span at most two pages, whose block-table entries are loaded ahead of
  // the scan
  const int q0 = j0 / p.PS, r0 = j0 - q0 * p.PS;
  const bool two_pages = p.PS >= kPer;
  int pg0 = 0, pg1 = 0;
  if (two_pages) {
    pg0 = page_of(p, bt[min(q0, p.max_pages - 1)]);
    pg1 = page_of(p, bt[min(q0 + 1, p.max_pages - 1)]);
  }
  int gtb, eqb, gt_total, eq_total;
  block_excl_sum2<NW>(ngt, neq, wave_cnt, gtb, eqb, gt_total, eq_total);
  gtb += gt_before;
  eqb += eq_before;
  int q = q0, r = r0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const bool in = j0 + i < L;
    const bool gt = in && kr[i] > thr;
    const bool eq = in && kr[i] == thr;
    if (gt || (eq && eqb < need)) {
      const int page = two_pages ? (q == q0 ? pg0 : pg1) : page_of(p, bt[min(q, p.max_pages - 1)]);
      out[gtb + min(eqb, need)] = page * p.PS + r;
    }
    gtb += gt ? 1 : 0;
    eqb += eq ? 1 : 0;
    if (++r == p.PS) {
      r = 0;
      ++q;
    }
  }
}

// One workgroup per sequence of a batch whose block table holds fewer than
// kWideSelectLen tokens: the four radix passes over keys held in registers,
// then the ordered compaction.
template <int NT>
__global__ __launch_bounds__(NT) void dsa_select_kernel(DsaParams p) {
  constexpr int kPer = kSelPer;
  constexpr int NW = NT / kWave;
  __shared__ int hist[2][NW][256];
  __shared__ int wave_cnt[NW][2];
  __shared__ SelState st;
  const int b = blockIdx.x;
  const int L = seq_len_of(p, b);
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  int32_t *out = p.out + (size_t)b * p.topk;
  const int32_t *bt = p.block_table + (size_t)b * p.max_pages;

  if (L <= p.topk) {  // every token, in position order, then -1
    for (int i = tid; i < p.topk; i += NT)
      out[i] = i < L ? page_of(p, bt[i / p.PS]) * p.PS + i % p.PS : -1;
    return;
  }
  const float *sc = p.scores + (size_t)b * p.max_len;

  // keys of positions tid * kPer + i (one chunk: such batches hold fewer than
  // NT * kPer tokens); positions past L get key 0 and are never counted
  uint32_t kr[kPer];
  auto load_keys = [&](int j0) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int j = j0 + i;
      kr[i] = j < L ? score_key(sc[j]) : 0u;
    }
  };
  load_keys(tid * kPer);
  for (int i = tid; i < NW * 256; i += NT) (&hist[0][0][0])[i] = 0;

  // radix select of the topk-th largest key, 8 bits per pass from the top:
  // `prefix` holds the bits fixed so far (under `mask`), `left` how many of
  // the keys matching them are still to be taken.  Local histograms are
  // double-buffered: the next pass's buffer is cleared while this one counts.
  if (tid == 0) st = SelState{0u, 0u, p.topk};
  __syncthreads();
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const SelState s0 = st;
    int *h = &hist[pass & 1][wave][0];
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (tid * kPer + i < L && (kr[i] & s0.mask) == s0.prefix) atomicAdd(&h[(kr[i] >> shift) & 255u], 1);
    if (pass < 3)
      for (int i = tid; i < NW * 256; i += NT) (&hist[(pass + 1) & 1][0][0])[i] = 0;
    __syncthreads();
    if (wave == 0) resolve_bin(&hist[pass & 1][0][0], NW, 256, shift, &st);
    __syncthreads();
  }
  const uint32_t thr = st.prefix;   // the topk-th largest key
  const int need = st.left;         // keys equal to it that are taken

  // ordered compaction: position j is taken if its key beats the threshold,
  // or equals it and fewer than `need` equal keys come before it; its output
  // slot is (keys above the threshold before j) + min(equal keys before j,
  // need), from one block scan of the two counts
  compact_slice<NW, kPer>(p, L, tid * kPer, thr, need, 0, 0, kr, wave_cnt, out, bt);
}

// Long sequences after the four histogram passes: the radix state replayed
// from the global histograms, then the positions in slices of kSlice, one
// workgroup each.  dsa_count_kernel counts each slice's keys above and equal
// to the threshold (slice 0 also stores the final state); dsa_compact_kernel
// sums the counts of the slices before its own and compacts its slice.  The
// counts [B, slices, 2] and the states [B, 2] follow the histograms in the
// workspace.
constexpr int kSlice = 2048;
constexpr int kSliceThreads = 256;
constexpr int kSlicePer = kSlice / kSliceThreads;
constexpr int kSliceWaves = kSliceThreads / kWave;

__device__ __forceinline__ int *slice_counts(const DsaParams &p, int b) {
  const int ns = (p.max_len + kSlice - 1) / kSlice;
  return p.hist + (size_t)4 * p.B * 256 + (size_t)b * ns * 2;
}
__device__ __forceinline__ int *slice_state(const DsaParams &p, int b) {
  const int ns = (p.max_len + kSlice - 1) / kSlice;
  return p.hist + (size_t)4 * p.B * 256 + (size_t)p.B * ns * 2 + (size_t)b * 2;
}

__global__ __launch_bounds__(kSliceThreads) void dsa_count_kernel(DsaParams p) {
  __shared__ SelState st;
  __shared__ int wave_cnt[kSliceWaves][2];
  const int b = blockIdx.y, s = blockIdx.x, tid = threadIdx.x;
  const int L = seq_len_of(p, b);
  const int j_begin = s * kSlice;
  if (L <= p.topk || j_begin >= L) return;  // whole workgroup
  if (tid == 0) st = SelState{0u, 0u, p.topk};
  __syncthreads();
  for (int q = 0; q < 4; ++q) {
    if (tid < kWave) resolve_bin(p.hist + ((size_t)q * p.B + b) * 256, 1, 0, 24 - 8 * q, &st);
    __syncthreads();
  }
  const uint32_t thr = st.prefix;
  const float *sc = p.scores + (size_t)b * p.max_len;
  const int j0 = j_begin + tid * kSlicePer;
  int ngt = 0, neq = 0;
#pragma unroll
  for (int i = 0; i < kSlicePer; ++i) {
    const int j = j0 + i;
    const uint32_t k = j < L ? score_key(sc[j]) : 0u;
    ngt += (j < L && k > thr) ? 1 : 0;
    neq += (j < L && k == thr) ? 1 : 0;
  }
  int pa, pb, tg, te;
  block_excl_sum2<kSliceWaves>(ngt, neq, wave_cnt, pa, pb, tg, te);
  if (tid == 0) {
    int *cnt = slice_counts(p, b) + (size_t)s * 2;
    cnt[0] = tg;
    cnt[1] = te;
    if (s == 0) {
      int *state = slice_state(p, b);
      state[0] = (int)thr;
      state[1] = st.left;
    }
  }
}

__global__ __launch_bounds__(kSliceThreads) void dsa_compact_kernel(DsaParams p) {
  __shared__ int wave_cnt[kSliceWaves][2];
  const int b = blockIdx.y, s = blockIdx.x, tid = threadIdx.x;
  const int L = seq_len_of(p, b);
  int32_t *out = p.out + (size_t)b * p.topk;
  const int32_t *bt = p.block_table + (size_t)b * p.max_pages;
  if (L <= p.topk) {  // every token, in position order, then -1
    for (int i = tid; i < kSlice; i += kSliceThreads) {
      const int pos = s * kSlice + i;
      if (pos < p.topk) out[pos] = pos < L ? page_of(p, bt[pos / p.PS]) * p.PS + pos % p.PS : -1;
    }
    return;
  }
  const int j_begin = s * kSlice;
  if (j_begin >= L) return;  // whole workgroup
  const int *state = slice_state(p, b);
  const uint32_t thr = (uint32_t)state[0];
  const int need = state[1];
  // the keys above and equal to the threshold in the slices before this one
  const int *cnt = slice_counts(p, b);
  int g = 0, e = 0;
  for (int t = tid; t < s; t += kSliceThreads) {
    g += cnt[(size_t)t * 2];
    e += cnt[(size_t)t * 2 + 1];
  }
  int pa, pb, gt_before, eq_before;
  block_excl_sum2<kSliceWaves>(g, e, wave_cnt, pa, pb, gt_before, eq_before);
  const float *sc = p.scores + (size_t)b * p.max_len;
  const int j0 = j_begin + tid * kSlicePer;
  uint32_t kr[kSlicePer];
#pragma unroll
  for (int i = 0; i < kSlicePer; ++i) {
    const int j = j0 + i;
    kr[i] = j < L ? score_key(sc[j]) : 0u;
  }
  compact_slice<kSliceWaves, kSlicePer>(p, L, j0, thr, need, gt_before, eq_before, kr, wave_cnt, out, bt);
}

}  // namespace

hipError_t launch_dsa_scores(const DsaParams &p, int max_len, bool force, hipStream_t st) {
  if (p.B == 0 || max_len == 0) return hipSuccess;
  // a batch that would give fewer than two 64-token workgroups per CU takes
  // 16-token workgroups
  if ((int64_t)((max_len + 63) / 64) * p.B < 512) {
    const dim3 grid((max_len + 15) / 16, p.B);
    hipLaunchKernelGGL(dsa_scores_kernel<16>, grid, dim3(kScoreThreads), 0, st, p, force ? 1 : 0);
  } else {
    const dim3 grid((max_len + 63) / 64, p.B);
    hipLaunchKernelGGL(dsa_scores_kernel<64>, grid, dim3(kScoreThreads), 0, st, p, force ? 1 : 0);
  }
  return hipGetLastError();
}

// Batches whose longest possible sequence reaches this many tokens count
// the radix histograms with many workgroups per sequence.
constexpr int kWideSelectLen = 16384;
constexpr int kWideTokensPerWG = 2048;

// the select kernel holds a whole sequence's keys in registers below this length
static_assert(kSelThreads * kSelPer >= kWideSelectLen, "local select covers every shorter sequence");

hipError_t launch_dsa_select(const DsaParams &p, hipStream_t st) {
  if (p.B == 0) return hipSuccess;
  if (p.max_len >= kWideSelectLen && !p.hist) return hipErrorInvalidValue;  // needs the histograms
  if (p.max_len >= kWideSelectLen) {
    static_assert(kWideTokensPerWG == kSlice, "histogram and compaction slices agree");
    const dim3 grid((p.max_len + kSlice - 1) / kSlice, p.B);
    for (int pass = 0; pass < 4; ++pass)
      hipLaunchKernelGGL(dsa_hist_kernel, grid, dim3(kHistThreads), 0, st, p, pass);
    hipLaunchKernelGGL(dsa_count_kernel, grid, dim3(kSliceThreads), 0, st, p);
    const dim3 cgrid((max(p.max_len, p.topk) + kSlice - 1) / kSlice, p.B);
    hipLaunchKernelGGL(dsa_compact_kernel, cgrid, dim3(kSliceThreads), 0, st, p);
  } else if (p.max_len <= kSmallSelThreads * kSelPer) {  // a short block table: 4 waves hold it all
    hipLaunchKernelGGL(dsa_select_kernel<kSmallSelThreads>, dim3(p.B), dim3(kSmallSelThreads), 0, st, p);
  } else {
    hipLaunchKernelGGL(dsa_select_kernel<kSelThreads>, dim3(p.B), dim3(kSelThreads), 0, st, p);
  }
  return hipGetLastError();
}

bool dsa_wide_select(int max_len) { return max_len >= kWideSelectLen; }

// ints of the long-sequence select's global state: the four radix histograms
// [4, B, 256], the slice counts [B, slices, 2] and the final states [B, 2]
size_t dsa_wide_ints(int B, int max_len) {
  const size_t ns = (size_t)(max_len + kSlice - 1) / kSlice;
  return (size_t)4 * 256 * B + (size_t)B * ns * 2 + (size_t)B * 2;
}

}  // namespace moe
