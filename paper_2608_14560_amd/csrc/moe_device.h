// moe_device.h -- device helpers and launch-parameter blocks shared by the
// gfx950 kernels of the fused FP8 MoE layer.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

constexpr int kWave = 64;

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- numerics

// Round an fp32 value to bf16 (nearest, ties to even); NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Two fp32 values -> two OCP e4m3fn codes (round to nearest even).  The inputs
// are clamped to +-448 first, so the conversion saturates instead of
// overflowing to NaN.  Result: code(a) in bits [7:0], code(b) in [15:8].
__device__ __forceinline__ uint32_t e4m3x2_rne_sat(float a, float b) {
  a = fminf(fmaxf(a, -448.0f), 448.0f);
  b = fminf(fmaxf(b, -448.0f), 448.0f);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false) & 0xffffu;
}

// GEMM2's expert outputs Y go to memory as fp16 with one power-of-two
// exponent per row and 16-column chunk (kYChunk): the chunk's largest
// magnitude m 2^x (m in [0.5, 1)) is scaled by 2^-(x - 15) into
// [2^14, 2^15), every value of the chunk is rounded to fp16 (nearest even)
// after that exact scaling, and the combine multiplies by 2^e back (exact).
// The rounding error is at most 2^-11 of the chunk's largest magnitude (half
// an fp16 ulp at [2^14, 2^15) is 8), in half of fp32's bytes.  An all-zero chunk gets exponent 0; a chunk below 2^-113
// keeps exponent -128 (its scaled values still stay below 2^15).
constexpr int kYChunk = 16;

__device__ __forceinline__ int y16_exponent(float amax) {
  if (!(amax > 0.0f)) return 0;
  return max(__builtin_amdgcn_frexp_expf(amax) - 15, -128);
}
__device__ __forceinline__ uint16_t y16_code(float y, int e) {
  const _Float16 h = (_Float16)__builtin_amdgcn_ldexpf(y, -e);
  return __builtin_bit_cast(uint16_t, h);
}
// two codes of one chunk packed as (lo, hi) in one dword: the same values as
// y16_code, by the packed fp32 -> fp16 conversion (nearest even)
__device__ __forceinline__ uint32_t y16_code2(float y0, float y1, int e) {
  typedef float f32x2_ __attribute__((ext_vector_type(2)));
  typedef _Float16 f16x2_ __attribute__((ext_vector_type(2)));
  const f32x2_ v = {__builtin_amdgcn_ldexpf(y0, -e), __builtin_amdgcn_ldexpf(y1, -e)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2_));
}
__device__ __forceinline__ float y16_value(uint16_t c, int e) {
  return __builtin_amdgcn_ldexpf((float)__builtin_bit_cast(_Float16, c), e);
}

// fp32 sigmoid with a fixed operation sequence: clamp to [-80, 80],
// e^z for z = -x by Cody-Waite reduction n = rint(z log2 e),
// r = z - n ln2 (two-part ln2), degree-7 Taylor polynomial of e^r in Horner
// form with fused multiply-adds, e^z = p * 2^n, and sigma = 1 / (1 + e^z)
// with a correctly rounded division.  Constants: log2 e, ln 2 split into a
// 12-trailing-zero head and its fp32 remainder, 1/k! rounded to fp32.
__device__ __forceinline__ float sigmoid_spec(float x) {
#pragma clang fp contract(off)
  const float kLog2e = 0x1.715476p+0f;
  const float kLn2Hi = 0x1.62e400p-1f;
  const float kLn2Lo = 0x1.7f7d1cp-20f;
  x = fminf(fmaxf(x, -80.0f), 80.0f);
  const float z = -x;
  const float n = __builtin_rintf(z * kLog2e);
  float r = __builtin_fmaf(-n, kLn2Hi, z);
  r = __builtin_fmaf(-n, kLn2Lo, r);
  float p = 1.0f / 5040.0f;
  p = __builtin_fmaf(p, r, 1.0f / 720.0f);
  p = __builtin_fmaf(p, r, 1.0f / 120.0f);
  p = __builtin_fmaf(p, r, 1.0f / 24.0f);
  p = __builtin_fmaf(p, r, 1.0f / 6.0f);
  p = __builtin_fmaf(p, r, 0.5f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  const float e = __builtin_ldexpf(p, (int)n);
  return 1.0f / (1.0f + e);
}

// SwiGLU of the expert MLP: silu(g) * u with silu(g) = g * sigmoid(g), in
// fp32 with the sigmoid above (a fixed sequence, so the re-quantised codes it
// feeds are reproducible).
__device__ __forceinline__ float swiglu_spec(float g, float u) {
#pragma clang fp contract(off)
  const float silu = g * sigmoid_spec(g);
  return silu * u;
}

// SwiGLU for the large-tile GEMM1 epilogue, where it runs on every element
// of a tile (64 per lane of a 256-row tile) and its cost is not hidden behind
// loads: silu(g) * u with sigma(g) = 1 / (1 + 2^t), t = -g log2(e), from the
// hardware's base-2 exponential and reciprocal (each within about an ulp).
// t is carried in two parts -- its fp32 rounding and the remainder (a fused
// multiply-add, plus -g times the constant's own fp32 tail) -- and
// 2^t = 2^t_hi (1 + t_lo ln 2), so the exponential keeps a few-ulp relative
// accuracy for any |g|; one Newton step refines the reciprocal.  Relative
// error of the result a few u (u = 2^-24), inside the 8 u the re-quantised
// intermediate's admissible set allows; sigma is exactly 1 where 2^t is below
// half an ulp of 1 (g >= 17), so SwiGLU is g * u there.  The routing keeps
// the fixed sequence above (its sigmoid decides expert selection).
__device__ __forceinline__ float swiglu_fast(float g, float u) {
  const float kLog2e = 0x1.715476p+0f;     // log2(e) rounded to fp32
  const float kLog2eLo = 0x1.4ae0c0p-26f;  // log2(e) - kLog2e
  const float kLn2 = 0x1.62e430p-1f;
  const float z = -g;
  const float t = z * kLog2e;
  const float tl = __builtin_fmaf(z, kLog2eLo, __builtin_fmaf(z, kLog2e, -t));
  const float e = __builtin_amdgcn_exp2f(t) * __builtin_fmaf(tl, kLn2, 1.0f);
  const float d = 1.0f + e;
  const float s0 = __builtin_amdgcn_rcpf(d);
  const float s = __builtin_fmaf(s0, __builtin_fmaf(-d, s0, 1.0f), s0);
  return (g * s) * u;
}

// The correctly rounded quotient v / b of several values by one divisor b:
// y = 1 / b (one correctly rounded division per divisor), then per value
// q = v y refined by its exact remainder, q' = q + (v - q b) y (two fused
// multiply-adds) -- with y the rounded reciprocal and q within an ulp, this
// correction rounds to the same result as the division (Markstein's
// theorem for round-to-nearest).  A divisor below 2^-100 has both operands
// scaled by 2^64 first (exact), so y stays finite.
struct DivBy {
  float b, y, pre;
  __device__ __forceinline__ explicit DivBy(float d) {
    pre = d < 0x1p-100f ? 0x1p64f : 1.0f;
    b = d * pre;
    y = 1.0f / b;
  }
  __device__ __forceinline__ float operator()(float v) const {
    const float vv = v * pre;
    const float q = vv * y;
    return __builtin_fmaf(__builtin_fmaf(-q, b, vv), y, q);
  }
};

// Total order used by every selection of the routing stage: the larger value
// wins, equal values go to the lower index.
__device__ __forceinline__ bool beats(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// ---------------------------------------------------------------- launch blocks

struct RouteParams {
  const float *logits;   // [T, E] (unused when `partials` is set)
  const float *bias;     // [E]
  int32_t *topk_ids;     // [T, K]
  float *topk_w;         // [T, K]
  int T, E, G, TG, K;
  float rsf;
  // Router projection path: the projection's per-block sums [T, KB, E] and
  // the hidden rows' block scales [T, KB]; the logits are formed from them.
  const float *partials;
  const float *pscale;
  int KB;
};

// Logits of the lane's experts e = q * 64 + lane (q < EPL) for token t.
// Given the router projection's block sums p_kb, each logit is the fused
// multiply-add chain over the blocks, ascending, from 0:
// acc = fmaf(scale[kb], p_kb, acc) -- the second half of the projection's
// fixed fp32 sequence (the chain inside a block runs in the projection
// kernel).  The block sums are fetched 32 blocks at a time for all slots
// before the chains consume them (fewer blocks per batch for wide routers), so
// the loads overlap.  Experts past E get 0.
template <int EPL>
__device__ __forceinline__ void route_logits(const RouteParams &p, int t, int lane,
                                             float (&lg)[EPL]) {
  // every load is in bounds (clamped indices) and unconditional; values past
  // E or KB are replaced by 0 afterwards
  if (!p.partials) {
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const int e = q * kWave + lane;
      const float x = p.logits[(size_t)t * p.E + min(e, p.E - 1)];
      lg[q] = e < p.E ? x : 0.0f;
    }
    return;
  }
  constexpr int kChunk = EPL >= 8 ? 64 / EPL : 32;
  const float *pp = p.partials + (size_t)t * p.KB * p.E;
  const float *sc = p.pscale + (size_t)t * p.KB;
#pragma unroll
  for (int q = 0; q < EPL; ++q) lg[q] = 0.0f;
  for (int kb0 = 0; kb0 < p.KB; kb0 += kChunk) {
    float v[kChunk][EPL], s[kChunk];
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
      const int kb = min(kb0 + j, p.KB - 1);
      s[j] = sc[kb];
#pragma unroll
      for (int q = 0; q < EPL; ++q) {
        const int e = q * kWave + lane;
        const float x = pp[(size_t)kb * p.E + min(e, p.E - 1)];
        v[j][q] = e < p.E ? x : 0.0f;
      }
    }
#pragma unroll
    for (int j = 0; j < kChunk; ++j)
      if (kb0 + j < p.KB) {
#pragma unroll
        for (int q = 0; q < EPL; ++q) lg[q] = __builtin_fmaf(s[j], v[j][q], lg[q]);
      }
  }
}

// Router projection: block sums of the dequantised-code rows against the
// fp32 router weight rows.
struct RouterParams {
  const uint8_t *hidden;       // [T, H] e4m3fn
  const float *weight;         // [E, H] fp32
  float *partials;             // [T, H/128, E] fp32
  int T, H, E;
};

struct PermuteParams {
  const int32_t *topk_ids;   // [T, K]
  int32_t *chunk_counts;     // [nchunks, El]
  int32_t *expert_offsets;   // [El + 1]
  int32_t *perm_token;       // [T*K]
  int32_t *perm_pair;        // [T*K]  t*K + j of each permuted row
  int32_t *pair_row;         // [T, K]
  int32_t *tile_base;        // [El + 1] first M-tile of each expert
  // [M-tiles, 4]: per M-tile of the batch its expert e, tile_base[e],
  // expert_offsets[e] and e's row count (one 16-byte load per work item)
  int32_t *tile_tab;
  int32_t *n_items;          // [2] work items of GEMM1 and GEMM2
  int T, K, El, offset, nchunks;
  int BM, items_per_tile1, items_per_tile2;
};

constexpr int kChunkTokens = 256;   // tokens per permute workgroup

struct GemmParams {
  // (narrow GEMM1 of at most 16 tokens only) the routing's permutation, built
  // by the GEMM1 workgroups themselves instead of a permutation launch
  PermuteParams perm;
  // A operand: GEMM1 gathers hidden rows through perm_token; GEMM2 reads the
  // permuted activation rows directly.
  const uint8_t *A;          // [rows, K]
  const float *A_scale;      // [rows, K/128]
  // B operand: the expert weights, [El, N_total, K] with [El, N_total/128, K/128] scales
  const uint8_t *B;
  const float *B_scale;
  const int32_t *expert_offsets;
  const int32_t *tile_base;
  const int32_t *tile_tab;   // see PermuteParams
  const int32_t *perm_token;
  const int32_t *n_items;    // device count of work items
  float *abuf;               // GEMM1 column-split SwiGLU output [P_max, I] fp32
  uint8_t *act;              // GEMM1 out: [P_max, I] e4m3
  float *act_scale;          // GEMM1 out: [P_max, I/128]
  float *act_scale_k;        // GEMM1 out (large tiles, optional): [I/128, P_max]
  // The large-tile kernels' activation scales by permuted row r and K block
  // kb: sa_tile[r * sa_row + kb * sa_kb] (a K-block-major copy, so that the
  // scales of one K block of a tile's rows share a few cache lines)
  const float *sa_tile;
  int sa_row, sa_kb;
  uint16_t *Y;               // GEMM2 out: [P_max, H] fp16 codes (see y16_code)
  int8_t *Ye;                // their exponents, [P_max, H / kYChunk]
  int K, KB;                 // reduction length and its 128-blocks
  int N_total;               // rows of one expert's weight matrix (2I or H)
  int I;                     // intermediate size (GEMM1 gate/up split)
  int NB;                    // column blocks per M-tile
  int S;                     // split-K factor (GEMM2: always 1)
  int P_max;                 // row capacity of act / abuf / Y
  int H;                     // GEMM2 output width (row stride of Y)
  int El;
};

struct FinalizeParams {
  const uint16_t *Y;         // [P_max, H] fp16 codes
  const int8_t *Ye;          // [P_max, H / kYChunk] exponents
  const int32_t *pair_row;   // [T, K]
  const float *topk_w;       // [T, K]
  uint16_t *out;             // [T, H] bf16
  int T, H, K;
  int cw;                    // columns per thread: 16 or 8
};

// The weighted combine fused into GEMM2 (batches of at most 16 tokens).
struct CombineParams {
  const int32_t *perm_pair;  // [P] t*K + j of each permuted row
  const float *topk_w;       // [T, K]
  uint16_t *out;             // [T, H] bf16
  int T, K;
  int C;                     // K chunks per tile (divides KB)
};

// DSA TopK indexer: 64 heads of 128, a paged key cache of PS tokens per page
struct DsaParams {
  const uint8_t *q;            // [B, 64, 128] e4m3
  const float *weights;        // [B, 64]
  const uint8_t *k_cache;      // [num_pages, PS, 128] e4m3
  const float *k_scale;        // [num_pages, PS]
  const int32_t *block_table;  // [B, max_pages]
  const int32_t *seq_lens;     // [B]
  float *scores;               // [B, max_len] workspace
  int *hist;                   // [4, B, 256] radix histograms (workspace; long batches)
  int32_t *out;                // [B, topk]
  int B, PS, topk, max_pages, max_len, num_pages;
};

// ---------------------------------------------------------------- launchers
// (defined in the .hip files, called by the C-ABI layer)
hipError_t launch_route(const RouteParams &p, hipStream_t st);
hipError_t launch_router_partials(const RouterParams &p, hipStream_t st);
hipError_t launch_dsa_scores(const DsaParams &p, int max_len, bool force, hipStream_t st);
hipError_t launch_dsa_select(const DsaParams &p, hipStream_t st);
bool dsa_wide_select(int max_len);
hipError_t launch_router_logits(const RouteParams &p, float *logits, hipStream_t st);
hipError_t launch_permute(const PermuteParams &p, hipStream_t st);
// hs_k[kb * P_max + r] = hidden_scale[perm_token[r] * KB + kb] for r < P
hipError_t launch_gather_scales(const int32_t *expert_offsets, int El, const int32_t *perm_token,
                                const float *hidden_scale, float *hs_k, int KB, int P_max,
                                hipStream_t st);
hipError_t launch_gemm1(const GemmParams &p, int BM, int grid, hipStream_t st);
// permute: the workgroups build the permutation themselves (p.perm; at most
// 16 tokens, gate/up-split items) instead of reading a permutation launch's
// k_split: 1, or 2 (each item's K range in two halves on separate waves,
// their sums added in fixed order)
hipError_t launch_gemm1_narrow(const GemmParams &p, int grid, bool gate_up_split, bool permute,
                               int k_split, hipStream_t st);
int gemm1_narrow_cols(bool gate_up_split);
hipError_t launch_requant(const GemmParams &p, int P_max, hipStream_t st);
hipError_t launch_gemm2(const GemmParams &p, int BM, int grid, hipStream_t st);
// large-tile GEMM1 / GEMM2 (BM = 64 or 128 rows x 256 columns, full K per item)
hipError_t launch_gemm_tile(const GemmParams &p, bool g1, int BM, int grid, hipStream_t st);
int gemm_tile_cols();
hipError_t launch_finalize(const FinalizeParams &p, hipStream_t st);
// GEMM2 with the weighted combine in its epilogue (T <= combine_max_tokens())
hipError_t launch_gemm2_combine(const GemmParams &p, const CombineParams &c, hipStream_t st);
int combine_max_tokens();
bool combine_fits(int P_max, int I);  // its LDS staging fits the workgroup

}  // namespace moe
