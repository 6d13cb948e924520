// attention.hip -- DSA sparse attention (paper Section 3.1.2): for each query
// token and head, gather the token's TopK cached entries through its sparse
// index list, form the base-2 logits
//   s_j = (q_nope . Kc_j + q_pe . Kp_j) * sm_scale * log2(e),
// take the softmax over them and accumulate the weights times Kc_j into a
// 512-wide output, with the base-2 log-sum-exp.
//
// Split-K flash decoding in two launches:
//   attn_partial_kernel  workgroup = (64 consecutive entries of the index
//                        list, token, 16 heads).  All 16 heads of a token read
//                        the same gathered rows, so both products are dense
//                        per workgroup and run on bf16 MFMA (16x16x32, fp32
//                        accumulate):
//                          S [16 heads x 64 entries] = Q [16 x 576] . K^T,
//                          wave w the entries 16w..16w+15, 18 steps over the
//                          576 dimensions (Q held in registers);
//                          the split's softmax per head across the 4 waves
//                          (through LDS), weights P = 2^(s - m), summed in
//                          fp32 and rounded to bf16 for the second product;
//                          O^T [512 x 16] = Kc^T . P^T, wave w the columns
//                          128w..128w+127, so that a lane holds 4 consecutive
//                          columns of one head for its store.
//                        The 64 rows (Kc and Kp, 1152 B each) are gathered to
//                        LDS with every load of a thread issued before its
//                        first store.  Writes the split's output normalised
//                        by its own sum, in bf16, and its (max m_s, sum l_s).
//   attn_merge_kernel    one-wave workgroup per (token, head, column range):
//                        the split outputs are loaded while the factors
//                        l_s 2^(m_s - M) / L are formed (L = sum_s l_s
//                        2^(m_s - M)); bf16 output and the LSE M + log2(L).
// Entries with an index outside [0, rows) count as absent (weight 0).
#include "attention_device.h"
#include "moe_device.h"

namespace moe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) uint8_t lds_u8;

constexpr int kThreads = 256;
constexpr int kD = kAttnDC + kAttnDP;          // 576 bf16 per gathered row
constexpr int kRowChunks = kD * 2 / 16;        // 72 chunks of 16 bytes
constexpr int kKSteps = kD / 32;               // 18 MFMA steps over the dimensions
// LDS row stride of the gathered rows: 1152 + 16 bytes (73 chunks, odd), so the
// 16 rows that one MFMA operand read touches start on distinct 4-bank groups
constexpr int kRowStride = kD * 2 + 16;
constexpr int kPStride = 72;                   // bf16 per weight row (144 B, same reason)
static_assert(kThreads == 8 * 32 && kRowChunks % 8 == 0, "gather: 8 threads per row, 32 rows per pass");
static_assert(kAttnHeads == 16 && kAttnEntries == 64, "one 16x16 MFMA tile per wave");

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
// reductions over the 16 lanes of a DPP row (lane bits 0..3): pairs, quads,
// half-row mirror, row mirror
template <int kCtrl>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), kCtrl, 0xF, 0xF, false));
}
__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  return fmaxf(v, dpp<0x140>(v));
}
__device__ __forceinline__ float row_sum16(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  return v + dpp<0x140>(v);
}
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__global__ __launch_bounds__(kThreads) void attn_partial_kernel(AttnParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint8_t *k_l = smem;                                                              // [64][kRowStride]
  uint16_t *p_l = reinterpret_cast<uint16_t *>(smem + kAttnEntries * kRowStride);  // [16][kPStride]
  __shared__ int idx_l[kAttnEntries];
  __shared__ float max_l[4][kAttnHeads];
  __shared__ float sum_l[4][kAttnHeads];

  const int s = blockIdx.x, t = blockIdx.y, hg = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int n = lane & 15, g = lane >> 4;
  const int e0 = s * kAttnEntries;

  if (tid < kAttnEntries) {
    const int slot = e0 + tid;
    const int row = slot < p.topk ? p.indices[(size_t)t * p.topk + slot] : -1;
    idx_l[tid] = (row >= 0 && row < p.rows) ? row : -1;
  }
  // Q as the MFMA A operand: lane (n, g) holds head n, dimensions 32 ks + 8 g .. + 7
  u32x4 qreg[kKSteps];
  {
    const size_t th = (size_t)t * p.H + hg * kAttnHeads + n;
#pragma unroll
    for (int ks = 0; ks < kKSteps; ++ks) {
      const int d = ks * 32 + g * 8;
      const uint16_t *src = d < kAttnDC ? p.q_nope + th * kAttnDC + d : p.q_pe + th * kAttnDP + (d - kAttnDC);
      qreg[ks] = *reinterpret_cast<const u32x4 *>(src);
    }
  }
  __syncthreads();

  // gather: thread (r = tid / 8, q = tid % 8) loads chunks q, q + 8, .., q + 64 of
  // rows r and r + 32 (Kc: chunks 0..63, Kp: 64..71), so each load instruction
  // of a wave covers whole 128-byte lines of 8 rows; absent rows are zero
  {
    const int r = tid >> 3, q = tid & 7;
    u32x4 v[2][kRowChunks / 8];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int row = idx_l[r + 32 * half];
#pragma unroll
      for (int j = 0; j < kRowChunks / 8; ++j) {
        const int c = q + 8 * j;
        v[half][j] = u32x4{0u, 0u, 0u, 0u};
        if (row >= 0) {
          const uint16_t *src = c < 64 ? p.ckv + (size_t)row * kAttnDC + c * 8
                                       : p.kpe + (size_t)row * kAttnDP + (c - 64) * 8;
          v[half][j] = *reinterpret_cast<const u32x4 *>(src);
        }
      }
    }
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int j = 0; j < kRowChunks / 8; ++j)
        *reinterpret_cast<u32x4 *>(k_l + (r + 32 * half) * kRowStride + (q + 8 * j) * 16) = v[half][j];
  }
  __syncthreads();

  // logits: S[head 4g + i][entry 16 wave + n] in sacc[i]
  f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
  {
    const uint8_t *krow = k_l + (wave * 16 + n) * kRowStride + g * 16;
#pragma unroll
    for (int ks = 0; ks < kKSteps; ++ks) {
      const u32x4 kv = *reinterpret_cast<const u32x4 *>(krow + ks * 64);
      sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(qreg[ks]), as_bf16x8(kv), sacc, 0, 0, 0);
    }
  }

  // the split's softmax per head over its 64 entries (4 waves x 16 lanes)
  const bool ok = idx_l[wave * 16 + n] >= 0;
  float sv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sv[i] = ok ? sacc[i] * p.scale_log2 : -INFINITY;
    const float m = row_max16(sv[i]);
    if (n == 0) max_l[wave][4 * g + i] = m;
  }
  __syncthreads();
  float M[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * g + i;
    M[i] = fmaxf(fmaxf(max_l[0][h], max_l[1][h]), fmaxf(max_l[2][h], max_l[3][h]));
    const float w = (ok && M[i] > -INFINITY) ? exp2f(sv[i] - M[i]) : 0.0f;
    p_l[h * kPStride + wave * 16 + n] = f32_to_bf16_rne(w);
    const float l = row_sum16(w);  // the sum (and so the LSE) keeps the fp32 weights
    if (n == 0) sum_l[wave][h] = l;
  }
  __syncthreads();

  // weighted sum, transposed: O^T [512 x 16 heads] = Kc^T . P^T, so that lane
  // (n, g) holds head n, columns 128 wave + 16 nt + 4 g .. + 3 in oacc[nt]
  f32x4 oacc[8];
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) oacc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the Kc^T operand (8 consecutive entries of one column per lane) by the
  // transposing LDS read: within each 16-lane group, lane s addresses row
  // e0 + s / 4, columns 4 (s % 4) .. + 3 of the tile, and lane i receives rows
  // e0 .. e0 + 3 of column i; two reads give the 8 entries
  lds_u8 *kl3 = (lds_u8 *)smem;  // k_l, as an LDS address
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const u32x4 pb = *reinterpret_cast<const u32x4 *>(p_l + n * kPStride + ks * 32 + g * 8);
    const int e0 = ks * 32 + g * 8 + (n >> 2);
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      const int c0 = wave * 128 + nt * 16 + 4 * (n & 3);
      lds_u8 *a = kl3 + e0 * kRowStride + c0 * 2;
      const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)a);
      const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(a + 4 * kRowStride));
      u32x4 ka;
      ka[0] = (uint32_t)(uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
      ka[1] = (uint32_t)(uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
      ka[2] = (uint32_t)(uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
      ka[3] = (uint32_t)(uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
      oacc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka), as_bf16x8(pb), oacc[nt], 0, 0, 0);
    }
  }

  // the split's output normalised by its own sum, bf16, 4 columns per store
  const size_t split_base = ((size_t)t * p.NS + s) * p.H + hg * kAttnHeads;
  const float l_n = (sum_l[0][n] + sum_l[1][n]) + (sum_l[2][n] + sum_l[3][n]);
  const float inv = l_n > 0.0f ? 1.0f / l_n : 0.0f;
  uint16_t *dst = p.part_o + (split_base + n) * kAttnDC + wave * 128 + g * 4;
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) {
    uint2 w;
    w.x = (uint32_t)f32_to_bf16_rne(oacc[nt][0] * inv) | ((uint32_t)f32_to_bf16_rne(oacc[nt][1] * inv) << 16);
    w.y = (uint32_t)f32_to_bf16_rne(oacc[nt][2] * inv) | ((uint32_t)f32_to_bf16_rne(oacc[nt][3] * inv) << 16);
    *reinterpret_cast<uint2 *>(dst + nt * 16) = w;
  }
  if (wave == 0 && n == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * g + i;
      float *ml = p.part_ml + (split_base + h) * 2;
      ml[0] = M[i];
      ml[1] = (sum_l[0][h] + sum_l[1][h]) + (sum_l[2][h] + sum_l[3][h]);
    }
  }
}

// whole-wave reductions: the row result, then rows 0 -> 1 and 2 -> 3
// (row_bcast:15), then rows 0-1 -> 2-3 (row_bcast:31); lane 63 holds the result
template <int kCtrl, int kRows>
__device__ __forceinline__ float dpp_rows(float old, float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old), __builtin_bit_cast(int, v),
                                                               kCtrl, kRows, 0xF, false));
}
__device__ __forceinline__ float wave_max(float v) {
  v = row_max16(v);
  v = fmaxf(v, dpp_rows<0x142, 0xA>(v, v));
  v = fmaxf(v, dpp_rows<0x143, 0xC>(v, v));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float wave_sum(float v) {
  v = row_sum16(v);
  v += dpp_rows<0x142, 0xA>(0.0f, v);
  v += dpp_rows<0x143, 0xC>(0.0f, v);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

constexpr int kMergeBatch = 32;  // split outputs in flight per lane

template <int CPL>
struct Cols;  // CPL bf16 output columns of one split: one load
template <>
struct Cols<2> {
  uint32_t w[1];
  __device__ void load(const uint16_t *p) { w[0] = *reinterpret_cast<const uint32_t *>(p); }
};
template <>
struct Cols<4> {
  uint32_t w[2];
  __device__ void load(const uint16_t *p) {
    const uint2 v = *reinterpret_cast<const uint2 *>(p);
    w[0] = v.x;
    w[1] = v.y;
  }
};
template <>
struct Cols<8> {
  uint32_t w[4];
  __device__ void load(const uint16_t *p) {
    const u32x4 v = *reinterpret_cast<const u32x4 *>(p);
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = v[q];
  }
};

// one wave per workgroup = (token, head, 64 CPL output columns), lane = CPL
// columns: split s enters with the factor l_s 2^(m_s - M) / L on its
// normalised output
template <int CPL>
__global__ __launch_bounds__(kWave) void attn_merge_kernel(AttnParams p) {
  constexpr int kParts = kAttnDC / (kWave * CPL);
  __shared__ float f_l[kAttnMaxSplits];
  const int lane = threadIdx.x;
  const int th = blockIdx.x / kParts, part = blockIdx.x % kParts;  // th < T * H
  const int t = th / p.H, head = th % p.H;
  const int col = (part * kWave + lane) * CPL;
  const size_t split0 = (size_t)t * p.NS * p.H + head;  // split s at split0 + s * H
  const uint16_t *o = p.part_o + split0 * kAttnDC + col;
  const size_t o_stride = (size_t)p.H * kAttnDC;

  // the first batch of split outputs is in flight while the factors are formed
  Cols<CPL> v[kMergeBatch];
#pragma unroll
  for (int k = 0; k < kMergeBatch; ++k) v[k].load(o + (size_t)min(k, p.NS - 1) * o_stride);

  float M = -INFINITY;
  for (int s = lane; s < p.NS; s += kWave) M = fmaxf(M, p.part_ml[(split0 + (size_t)s * p.H) * 2]);
  M = wave_max(M);
  float L = 0.0f;
  for (int s = lane; s < p.NS; s += kWave) {
    const float *ml = p.part_ml + (split0 + (size_t)s * p.H) * 2;
    const float f = (M > -INFINITY && ml[0] > -INFINITY) ? ml[1] * exp2f(ml[0] - M) : 0.0f;
    f_l[s] = f;
    L += f;
  }
  L = wave_sum(L);
  __syncthreads();  // f_l

  float acc[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) acc[k] = 0.0f;
  for (int s0 = 0; s0 < p.NS; s0 += kMergeBatch) {
    if (s0 > 0) {
#pragma unroll
      for (int k = 0; k < kMergeBatch; ++k) v[k].load(o + (size_t)min(s0 + k, p.NS - 1) * o_stride);
    }
#pragma unroll
    for (int k = 0; k < kMergeBatch; ++k) {
      const float f = s0 + k < p.NS ? f_l[s0 + k] : 0.0f;
#pragma unroll
      for (int q = 0; q < CPL / 2; ++q) {
        acc[2 * q] = __builtin_fmaf(f, bf_lo(v[k].w[q]), acc[2 * q]);
        acc[2 * q + 1] = __builtin_fmaf(f, bf_hi(v[k].w[q]), acc[2 * q + 1]);
      }
    }
  }
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  uint16_t *dst = p.out + (size_t)th * kAttnDC + col;
#pragma unroll
  for (int q = 0; q < CPL / 2; ++q)
    reinterpret_cast<uint32_t *>(dst)[q] =
        (uint32_t)f32_to_bf16_rne(acc[2 * q] * inv) | ((uint32_t)f32_to_bf16_rne(acc[2 * q + 1] * inv) << 16);
  if (part == 0 && lane == 0) p.lse[th] = L > 0.0f ? M + log2f(L) : -INFINITY;
}

}  // namespace

hipError_t launch_attention(const AttnParams &p, hipStream_t st) {
  if (p.T == 0) return hipSuccess;
  if (p.NS > kAttnMaxSplits || p.H % kAttnHeads) return hipErrorInvalidValue;
  const size_t lds = (size_t)kAttnEntries * kRowStride + sizeof(uint16_t) * kAttnHeads * kPStride;
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(attn_partial_kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(attn_partial_kernel, dim3(p.NS, p.T, p.H / kAttnHeads), dim3(kThreads), lds, st, p);
  // the merge spreads over at least 256 workgroups where the columns allow
  const int th = p.T * p.H;
  if (th * (kAttnDC / (kWave * 8)) >= 256)
    hipLaunchKernelGGL(attn_merge_kernel<8>, dim3(th * (kAttnDC / (kWave * 8))), dim3(kWave), 0, st, p);
  else if (th * (kAttnDC / (kWave * 4)) >= 256)
    hipLaunchKernelGGL(attn_merge_kernel<4>, dim3(th * (kAttnDC / (kWave * 4))), dim3(kWave), 0, st, p);
  else
    hipLaunchKernelGGL(attn_merge_kernel<2>, dim3(th * (kAttnDC / (kWave * 2))), dim3(kWave), 0, st, p);
  return hipGetLastError();
}

}  // namespace moe
