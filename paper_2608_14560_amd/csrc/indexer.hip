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
constexpr int kSelWaves = kSelThreads / kWave;

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
template <int TPW>
__global__ __launch_bounds__(kScoreThreads) void dsa_scores_kernel(DsaParams p, int force) {
  constexpr int kTokPerWG = TPW;
  constexpr int kHeadsPerThread = kNH / (kScoreThreads / TPW);
  static_assert(kHeadsPerThread % 4 == 0, "heads in groups of four");
  __shared__ __attribute__((aligned(16))) float q_l[kNH * kD];
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

  // the query's 64 x 128 codes, decoded exactly to fp32 (32 per thread)
  {
    const uint8_t *qb = p.q + (size_t)b * kNH * kD;
    const u32x4 a = *reinterpret_cast<const u32x4 *>(qb + tid * 32);
    const u32x4 c = *reinterpret_cast<const u32x4 *>(qb + tid * 32 + 16);
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
        const float4 q4 = *reinterpret_cast<const float4 *>(&q_l[(h0 + g) * kD + d]);
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

// Block-wide exclusive prefix sum of `v` over the workgroup's threads in
// order; returns the prefix and writes the total to *total.  Uses one LDS
// word per wave.
__device__ __forceinline__ int block_excl_sum(int v, int *wave_sum, int *total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  int incl = v;  // inclusive scan inside the wave
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int o = __shfl_up(incl, off);
    incl += (lane >= off) ? o : 0;
  }
  __syncthreads();  // previous users of wave_sum are done
  if (lane == kWave - 1) wave_sum[wave] = incl;
  __syncthreads();
  int before = 0, all = 0;
  for (int w = 0; w < kSelWaves; ++w) {
    const int c = wave_sum[w];
    before += (w < wave) ? c : 0;
    all += c;
  }
  *total = all;
  return before + incl - v;
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
  int suffix = mine;  // sum over lanes >= lane
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int o = __shfl_down(suffix, off);
    suffix += (lane + off < kWave) ? o : 0;
  }
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

// GLOBAL: the four histograms come from dsa_hist_kernel; otherwise this
// workgroup counts every position itself.
template <bool GLOBAL>
__global__ __launch_bounds__(kSelThreads) void dsa_select_kernel(DsaParams p) {
  __shared__ int hist[kSelWaves][256];
  __shared__ int wave_cnt[kSelWaves];
  __shared__ SelState st;
  const int b = blockIdx.x;
  const int L = seq_len_of(p, b);
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  int32_t *out = p.out + (size_t)b * p.topk;
  const int32_t *bt = p.block_table + (size_t)b * p.max_pages;

  if (L <= p.topk) {  // every token, in position order, then -1
    for (int i = tid; i < p.topk; i += kSelThreads)
      out[i] = i < L ? page_of(p, bt[i / p.PS]) * p.PS + i % p.PS : -1;
    return;
  }
  const float *sc = p.scores + (size_t)b * p.max_len;

  // radix select of the topk-th largest key, 8 bits per pass from the top:
  // `prefix` holds the bits fixed so far (under `mask`), `left` how many of
  // the keys matching them are still to be taken
  if (tid == 0) st = SelState{0u, 0u, p.topk};
  __syncthreads();
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (GLOBAL) {
      if (wave == 0) resolve_bin(p.hist + ((size_t)pass * p.B + b) * 256, 1, 0, shift, &st);
    } else {
      for (int i = tid; i < kSelWaves * 256; i += kSelThreads) (&hist[0][0])[i] = 0;
      __syncthreads();
      const SelState s0 = st;
      count_keys(sc, 0, L, kSelThreads, s0, shift, hist[wave]);
      __syncthreads();
      if (wave == 0) resolve_bin(&hist[0][0], kSelWaves, 256, shift, &st);
    }
    __syncthreads();
  }
  const uint32_t thr = st.prefix;   // the topk-th largest key
  const int need = st.left;         // keys equal to it that are taken

  // ordered compaction: position j is taken if its key beats the threshold,
  // or equals it and fewer than `need` equal keys come before it.  Each
  // thread owns kPer consecutive positions of a chunk; two block scans per
  // chunk give the equal-key ranks and the output slots.
  constexpr int kPer = 16;
  int eq_before = 0, sel_before = 0;
  for (int base = 0; base < L; base += kSelThreads * kPer) {
    const int j0 = base + tid * kPer;
    uint32_t k[kPer];
    int neq = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int j = j0 + i;
      k[i] = j < L ? score_key(sc[j]) : 0u;
      neq += (j < L && k[i] == thr) ? 1 : 0;
    }
    int eq_total, sel_total;
    int eq_rank = eq_before + block_excl_sum(neq, wave_cnt, &eq_total);
    uint32_t selm = 0u;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const bool in = j0 + i < L;
      const bool eq = in && k[i] == thr;
      const bool sel = (in && k[i] > thr) || (eq && eq_rank < need);
      eq_rank += eq ? 1 : 0;
      selm |= sel ? (1u << i) : 0u;
    }
    int pos = sel_before + block_excl_sum(__popc(selm), wave_cnt, &sel_total);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (selm & (1u << i)) {
        const int j = j0 + i;
        out[pos++] = page_of(p, bt[j / p.PS]) * p.PS + j % p.PS;
      }
    }
    eq_before += eq_total;
    sel_before += sel_total;
  }
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

hipError_t launch_dsa_select(const DsaParams &p, hipStream_t st) {
  if (p.B == 0) return hipSuccess;
  if (p.max_len >= kWideSelectLen && p.hist) {
    const dim3 grid((p.max_len + kWideTokensPerWG - 1) / kWideTokensPerWG, p.B);
    for (int pass = 0; pass < 4; ++pass)
      hipLaunchKernelGGL(dsa_hist_kernel, grid, dim3(kHistThreads), 0, st, p, pass);
    hipLaunchKernelGGL(dsa_select_kernel<true>, dim3(p.B), dim3(kSelThreads), 0, st, p);
  } else {
    hipLaunchKernelGGL(dsa_select_kernel<false>, dim3(p.B), dim3(kSelThreads), 0, st, p);
  }
  return hipGetLastError();
}

bool dsa_wide_select(int max_len) { return max_len >= kWideSelectLen; }

}  // namespace moe
