// attention.hip -- DSA sparse attention (paper Section 3.1.2): for each query
// token and head, gather the token's TopK cached entries through its sparse
// index list, form the base-2 logits
//   s_j = (q_nope . Kc_j + q_pe . Kp_j) * sm_scale * log2(e),
// take the softmax over them and accumulate the weights times Kc_j into a
// 512-wide output, with the base-2 log-sum-exp.
//
// Split-K flash decoding in two launches:
//   attn_partial_kernel  workgroup = (64 consecutive entries of the index
//                        list, token, 16 heads): the 64 gathered rows (Kc and
//                        Kp, bf16) and the 16 query rows (fp32) in LDS; 4
//                        waves, wave w the heads 4w..4w+3, lane = entry for
//                        the logits (fp32 fused multiply-adds over the 576
//                        dimensions) and the split's softmax (wave max and
//                        sum), lane = 8 output columns for the weighted sum;
//                        writes the unnormalised split output and its
//                        (max, sum).
//   attn_merge_kernel    per (token, head): rescales the splits by 2^(m_s - M)
//                        and normalises; bf16 output and the LSE M + log2(L).
// Entries with an index outside [0, rows) count as absent (weight 0).
#include "attention_device.h"
#include "moe_device.h"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kD = kAttnDC + kAttnDP;          // 576 bf16 per gathered row
constexpr int kRowChunks = kD * 2 / 16;        // 72 chunks of 16 bytes
// LDS row stride of the gathered rows in bytes: 1152 + 16 keeps lane-per-row
// 16-byte reads on distinct bank groups (73 chunks, odd)
constexpr int kRowStride = kD * 2 + 16;

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return f32_to_bf16_rne(f); }

__global__ __launch_bounds__(kThreads) void attn_partial_kernel(AttnParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint8_t *k_l = smem;                                              // [64][kRowStride]
  float *q_l = reinterpret_cast<float *>(smem + kAttnEntries * kRowStride);  // [16][576]
  float *p_l = q_l + kAttnHeads * kD;                                // [64][16]
  __shared__ int valid_l[kAttnEntries];

  const int s = blockIdx.x, t = blockIdx.y, hg = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int e0 = s * kAttnEntries;

  // gather: 64 rows x 72 chunks (Kc: chunks 0..63, Kp: 64..71); absent rows zero
  for (int i = tid; i < kAttnEntries * kRowChunks; i += kThreads) {
    const int e = i / kRowChunks, c = i % kRowChunks;
    const int slot = e0 + e;
    int row = slot < p.topk ? p.indices[(size_t)t * p.topk + slot] : -1;
    const bool ok = row >= 0 && row < p.rows;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (ok) {
      const uint16_t *src = c < 64 ? p.ckv + (size_t)row * kAttnDC + c * 8
                                   : p.kpe + (size_t)row * kAttnDP + (c - 64) * 8;
      v = *reinterpret_cast<const u32x4 *>(src);
    }
    *reinterpret_cast<u32x4 *>(k_l + e * kRowStride + c * 16) = v;
    if (c == 0) valid_l[e] = ok ? 1 : 0;
  }
  // the 16 query rows, fp32
  for (int i = tid; i < kAttnHeads * kRowChunks; i += kThreads) {
    const int h = i / kRowChunks, c = i % kRowChunks;
    const size_t th = (size_t)t * p.H + hg * kAttnHeads + h;
    const uint16_t *src = c < 64 ? p.q_nope + th * kAttnDC + c * 8 : p.q_pe + th * kAttnDP + (c - 64) * 8;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(src);
    float *dst = q_l + h * kD + c * 8;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      dst[2 * k] = bf_lo(v[k]);
      dst[2 * k + 1] = bf_hi(v[k]);
    }
  }
  __syncthreads();

  // logits: lane = entry, wave = 4 heads
  const int h0 = wave * 4;
  float lg[4] = {0.f, 0.f, 0.f, 0.f};
  {
    const uint8_t *krow = k_l + lane * kRowStride;
    for (int c = 0; c < kRowChunks; ++c) {
      const u32x4 kv = *reinterpret_cast<const u32x4 *>(krow + c * 16);
      float kf[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        kf[2 * k] = bf_lo(kv[k]);
        kf[2 * k + 1] = bf_hi(kv[k]);
      }
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float4 qa = *reinterpret_cast<const float4 *>(q_l + (h0 + h) * kD + c * 8);
        const float4 qb = *reinterpret_cast<const float4 *>(q_l + (h0 + h) * kD + c * 8 + 4);
        lg[h] = __builtin_fmaf(qa.x, kf[0], lg[h]);
        lg[h] = __builtin_fmaf(qa.y, kf[1], lg[h]);
        lg[h] = __builtin_fmaf(qa.z, kf[2], lg[h]);
        lg[h] = __builtin_fmaf(qa.w, kf[3], lg[h]);
        lg[h] = __builtin_fmaf(qb.x, kf[4], lg[h]);
        lg[h] = __builtin_fmaf(qb.y, kf[5], lg[h]);
        lg[h] = __builtin_fmaf(qb.z, kf[6], lg[h]);
        lg[h] = __builtin_fmaf(qb.w, kf[7], lg[h]);
      }
    }
  }
  // the split's softmax per head: wave max, weights 2^(s - m), wave sum
  const bool ok = valid_l[lane] != 0;
  float m_h[4], l_h[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const float sv = ok ? lg[h] * p.scale_log2 : -INFINITY;
    float m = sv;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    const float w = (ok && m > -INFINITY) ? exp2f(sv - m) : 0.0f;
    float l = w;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) l += __shfl_xor(l, off);
    m_h[h] = m;
    l_h[h] = l;
    p_l[lane * kAttnHeads + h0 + h] = w;
  }
  __syncthreads();

  // weighted sum: lane = output columns 8 lane .. 8 lane + 7, wave = 4 heads
  float acc[4][8];
#pragma unroll
  for (int h = 0; h < 4; ++h)
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[h][k] = 0.0f;
  for (int e = 0; e < kAttnEntries; ++e) {
    const u32x4 kv = *reinterpret_cast<const u32x4 *>(k_l + e * kRowStride + lane * 16);
    float kf[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      kf[2 * k] = bf_lo(kv[k]);
      kf[2 * k + 1] = bf_hi(kv[k]);
    }
    const float4 w4 = *reinterpret_cast<const float4 *>(p_l + e * kAttnHeads + h0);
    const float w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[h][k] = __builtin_fmaf(w[h], kf[k], acc[h][k]);
  }
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int head = hg * kAttnHeads + h0 + h;
    float *dst = p.part_o + (((size_t)t * p.NS + s) * p.H + head) * kAttnDC + lane * 8;
    *reinterpret_cast<float4 *>(dst) = float4{acc[h][0], acc[h][1], acc[h][2], acc[h][3]};
    *reinterpret_cast<float4 *>(dst + 4) = float4{acc[h][4], acc[h][5], acc[h][6], acc[h][7]};
    if (lane == 0) {
      float *ml = p.part_ml + (((size_t)t * p.NS + s) * p.H + head) * 2;
      ml[0] = m_h[h];
      ml[1] = l_h[h];
    }
  }
}

// one wave per (token, head): lane = 8 output columns
__global__ __launch_bounds__(kThreads) void attn_merge_kernel(AttnParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int th = blockIdx.x * (kThreads / kWave) + wave;  // t * H + head
  if (th >= p.T * p.H) return;
  const int t = th / p.H, head = th % p.H;
  float M = -INFINITY;
  for (int s = 0; s < p.NS; ++s) {
    const float m = p.part_ml[(((size_t)t * p.NS + s) * p.H + head) * 2];
    M = fmaxf(M, m);
  }
  float L = 0.0f, acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.0f;
  if (M > -INFINITY) {
    for (int s = 0; s < p.NS; ++s) {
      const size_t base = ((size_t)t * p.NS + s) * p.H + head;
      const float m = p.part_ml[base * 2], l = p.part_ml[base * 2 + 1];
      if (!(m > -INFINITY)) continue;  // a split with no entry
      const float f = exp2f(m - M);
      L = __builtin_fmaf(l, f, L);
      const float *o = p.part_o + base * kAttnDC + lane * 8;
      const float4 a = *reinterpret_cast<const float4 *>(o);
      const float4 b = *reinterpret_cast<const float4 *>(o + 4);
      acc[0] = __builtin_fmaf(a.x, f, acc[0]);
      acc[1] = __builtin_fmaf(a.y, f, acc[1]);
      acc[2] = __builtin_fmaf(a.z, f, acc[2]);
      acc[3] = __builtin_fmaf(a.w, f, acc[3]);
      acc[4] = __builtin_fmaf(b.x, f, acc[4]);
      acc[5] = __builtin_fmaf(b.y, f, acc[5]);
      acc[6] = __builtin_fmaf(b.z, f, acc[6]);
      acc[7] = __builtin_fmaf(b.w, f, acc[7]);
    }
  }
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  uint4 o;
  o.x = (uint32_t)f32_to_bf16(acc[0] * inv) | ((uint32_t)f32_to_bf16(acc[1] * inv) << 16);
  o.y = (uint32_t)f32_to_bf16(acc[2] * inv) | ((uint32_t)f32_to_bf16(acc[3] * inv) << 16);
  o.z = (uint32_t)f32_to_bf16(acc[4] * inv) | ((uint32_t)f32_to_bf16(acc[5] * inv) << 16);
  o.w = (uint32_t)f32_to_bf16(acc[6] * inv) | ((uint32_t)f32_to_bf16(acc[7] * inv) << 16);
  *reinterpret_cast<uint4 *>(p.out + (size_t)th * kAttnDC + lane * 8) = o;
  if (lane == 0) p.lse[th] = L > 0.0f ? M + log2f(L) : -INFINITY;
}

}  // namespace

hipError_t launch_attention(const AttnParams &p, hipStream_t st) {
  if (p.T == 0) return hipSuccess;
  const size_t lds = (size_t)kAttnEntries * kRowStride + sizeof(float) * kAttnHeads * kD +
                     sizeof(float) * kAttnEntries * kAttnHeads;
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(attn_partial_kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(attn_partial_kernel, dim3(p.NS, p.T, p.H / kAttnHeads), dim3(kThreads), lds, st, p);
  const int waves = p.T * p.H;
  hipLaunchKernelGGL(attn_merge_kernel, dim3((waves + kThreads / kWave - 1) / (kThreads / kWave)),
                     dim3(kThreads), 0, st, p);
  return hipGetLastError();
}

}  // namespace moe
