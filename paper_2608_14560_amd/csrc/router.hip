// router.hip -- the router projection of stage (1) of the Fused MoE block
// (paper Section 3.1.1: routing scores start from a lightweight linear
// projection of the token's hidden state).  The hidden rows arrive as FP8
// e4m3fn codes with 1x128 fp32 block scales and the router weight is fp32
// [E, H].  The logits decide the expert choice, so they follow one fixed fp32
// sequence: per 128-element block, a fused multiply-add chain over the
// decoded codes (exact in fp32) times the weights, ascending from 0; then a
// chain over the blocks, acc = fmaf(scale, block sum, acc).
//
// This kernel computes the block sums only, split over (block, 64 experts,
// 16 or 32 tokens) workgroups, so a decode-sized batch spreads the 7 MB weight
// stream over the whole chip; the routing kernel forms each logit from the
// block sums while it routes, so the logits never go to memory.
//
// Built with -ffp-contract=off: only the explicit fmaf calls fuse.
#include "moe_device.h"

namespace moe {
namespace {

constexpr int kProjExperts = 64;  // experts per workgroup (one per lane)
// LDS row stride of the weight tile in floats: 128 + 4 keeps the lanes'
// 16-byte row reads on distinct banks
constexpr int kWStride = 132;

// TPW tokens per wave, 4 waves: 4 TPW tokens per workgroup.  Large batches
// take 8 (the weight tile is then reused by 32 tokens), small ones 4 (more
// workgroups to spread the weight stream).
template <int TPW>
__global__ __launch_bounds__(256) void router_partials_kernel(RouterParams p) {
  constexpr int kProjTokens = 4 * TPW;
  __shared__ __attribute__((aligned(16))) float w_l[kProjExperts * kWStride];
  __shared__ __attribute__((aligned(16))) float x_l[kProjTokens * 128];
  const int kb = blockIdx.x;
  const int e0 = blockIdx.y * kProjExperts;
  const int t0 = blockIdx.z * kProjTokens;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int KB = p.H / 128;

  // weight tile: 64 rows x 128 fp32 of block kb (rows past E read as zero),
  // and hidden tile: 16 rows x 128 codes, decoded exactly to fp32.  Every
  // load is issued before the first LDS store, so they overlap.
  constexpr int kWLoads = kProjExperts * 32 / 256;
  float4 wv[kWLoads];
#pragma unroll
  for (int j = 0; j < kWLoads; ++j) {
    const int i = tid + 256 * j, r = i >> 5, c4 = i & 31;
    wv[j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (e0 + r < p.E)
      wv[j] = *reinterpret_cast<const float4 *>(p.weight + (size_t)(e0 + r) * p.H + kb * 128 + c4 * 4);
  }
  constexpr int kXLoads = kProjTokens * 32 / 256;
  int xq[kXLoads];
#pragma unroll
  for (int j = 0; j < kXLoads; ++j) {
    const int i = tid + 256 * j, r = i >> 5, c4 = i & 31;
    xq[j] = 0;
    if (t0 + r < p.T)
      xq[j] = *reinterpret_cast<const int *>(p.hidden + (size_t)(t0 + r) * p.H + kb * 128 + c4 * 4);
  }
#pragma unroll
  for (int j = 0; j < kWLoads; ++j) {
    const int i = tid + 256 * j, r = i >> 5, c4 = i & 31;
    *reinterpret_cast<float4 *>(&w_l[r * kWStride + c4 * 4]) = wv[j];
  }
#pragma unroll
  for (int j = 0; j < kXLoads; ++j) {
    const int i = tid + 256 * j, r = i >> 5, c4 = i & 31;
    float4 v;
    v.x = __builtin_amdgcn_cvt_f32_fp8(xq[j], 0);
    v.y = __builtin_amdgcn_cvt_f32_fp8(xq[j], 1);
    v.z = __builtin_amdgcn_cvt_f32_fp8(xq[j], 2);
    v.w = __builtin_amdgcn_cvt_f32_fp8(xq[j], 3);
    *reinterpret_cast<float4 *>(&x_l[r * 128 + c4 * 4]) = v;
  }
  __syncthreads();

  // lane = expert e0 + lane, wave = tokens TPW wave .. TPW wave + TPW - 1:
  // TPW independent chains, each ascending over the block's 128 elements
  float acc[TPW];
#pragma unroll
  for (int j = 0; j < TPW; ++j) acc[j] = 0.0f;
  const float *wr = &w_l[lane * kWStride];
  const float *xr = &x_l[wave * TPW * 128];
#pragma unroll 8
  for (int h = 0; h < 128; h += 4) {
    const float4 w4 = *reinterpret_cast<const float4 *>(wr + h);
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const float4 x4 = *reinterpret_cast<const float4 *>(xr + j * 128 + h);
      acc[j] = __builtin_fmaf(x4.x, w4.x, acc[j]);
      acc[j] = __builtin_fmaf(x4.y, w4.y, acc[j]);
      acc[j] = __builtin_fmaf(x4.z, w4.z, acc[j]);
      acc[j] = __builtin_fmaf(x4.w, w4.w, acc[j]);
    }
  }
  const int e = e0 + lane;
  if (e < p.E) {
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const int t = t0 + wave * TPW + j;
      if (t < p.T) p.partials[((size_t)t * KB + kb) * p.E + e] = acc[j];
    }
  }
}

}  // namespace

hipError_t launch_router_partials(const RouterParams &p, hipStream_t st) {
  if (p.T == 0) return hipSuccess;
  const int tpw = p.T >= 512 ? 8 : 4;
  dim3 grid(p.H / 128, (p.E + kProjExperts - 1) / kProjExperts, (p.T + 4 * tpw - 1) / (4 * tpw));
  if (tpw == 8)
    hipLaunchKernelGGL(router_partials_kernel<8>, grid, dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(router_partials_kernel<4>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace moe
