// route.hip -- stage (1) of the Fused MoE block (paper Section 3.1.1):
// sigmoid routing scores, group-limited top-k expert selection and the
// normalised, scaled routing weights.  One wave64 per token; all selections
// are butterfly reductions over the wave.
//
// Built with -ffp-contract=off: the fp32 sequence below is a specification
// (its integer decisions must be reproducible bit for bit), so no
// multiply-add may be fused except the explicit fmaf calls.
#include "moe_device.h"

namespace moe {
namespace {

// Wave-wide argmax of (value, index) under `beats`, carrying a payload.
__device__ __forceinline__ void wave_argmax(float &v, int &i, float &pay) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(i, off);
    const float op = __shfl_xor(pay, off);
    if (beats(ov, oi, v, i)) {
      v = ov;
      i = oi;
      pay = op;
    }
  }
}

constexpr int kNoIdx = 0x7fffffff;

// EPL = experts held per lane (expert e lives in lane e % 64, slot e / 64).
template <int EPL>
__global__ __launch_bounds__(256) void route_kernel(RouteParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int t = blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
  if (t >= p.T) return;  // whole wave leaves; the kernel has no block barrier

  const int gsz = p.E / p.G;
  const float *lrow = p.logits + (size_t)t * p.E;

  float sc[EPL], key[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    if (e < p.E) {
      sc[q] = sigmoid_spec(lrow[e]);
      key[q] = sc[q] + p.bias[e];
    } else {
      sc[q] = 0.0f;
      key[q] = -INFINITY;
    }
  }

  // group score = sum of the two largest keys of the group
  float my_gs = -INFINITY;  // lane g keeps the score of group g
  for (int g = 0; g < p.G; ++g) {
    float v1 = -INFINITY, v2 = -INFINITY, dummy = 0.0f;
    int i1 = kNoIdx, i2 = kNoIdx;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const int e = q * kWave + lane;
      if (e < p.E && e / gsz == g) {
        if (beats(key[q], e, v1, i1)) {
          v2 = v1; i2 = i1;
          v1 = key[q]; i1 = e;
        } else if (beats(key[q], e, v2, i2)) {
          v2 = key[q]; i2 = e;
        }
      }
    }
    // best of the group
    float bv = v1, bp = 0.0f;
    int bi = i1;
    wave_argmax(bv, bi, bp);
    // second best: the lane that held the best offers its runner-up instead
    float sv = (i1 == bi) ? v2 : v1;
    int si = (i1 == bi) ? i2 : i1;
    wave_argmax(sv, si, dummy);
    const float gs = bv + sv;
    if (lane == g) my_gs = gs;
  }

  // keep the topk_group best groups: a group is kept when fewer than
  // topk_group groups beat it
  int rank = 0;
  for (int g = 0; g < p.G; ++g) {
    const float og = __shfl(my_gs, g);
    if (lane < p.G && g != lane && beats(og, g, my_gs, lane)) ++rank;
  }
  const int kept_lane = (lane < p.G && rank < p.TG) ? 1 : 0;
  bool cand[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    const int g = (e < p.E) ? e / gsz : 0;
    cand[q] = (e < p.E) && (__shfl(kept_lane, g) != 0);
  }

  // top-k experts among the kept groups, in selection order
  int my_id = 0;
  float my_s = 0.0f;
  for (int j = 0; j < p.K; ++j) {
    float bv = -INFINITY, bs = 0.0f;
    int bi = kNoIdx;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const int e = q * kWave + lane;
      if (cand[q] && beats(key[q], e, bv, bi)) {
        bv = key[q];
        bi = e;
        bs = sc[q];
      }
    }
    wave_argmax(bv, bi, bs);
#pragma unroll
    for (int q = 0; q < EPL; ++q)
      if (q * kWave + lane == bi) cand[q] = false;
    if (lane == j) {
      my_id = bi;
      my_s = bs;
    }
  }

  // weights: unbiased scores normalised over the k selections (summed in
  // selection order), times the routed scaling factor
  float sum = 0.0f;
  for (int j = 0; j < p.K; ++j) sum += __shfl(my_s, j);
  if (lane < p.K) {
    p.topk_ids[(size_t)t * p.K + lane] = my_id;
    p.topk_w[(size_t)t * p.K + lane] = (my_s / sum) * p.rsf;
  }
}

}  // namespace

hipError_t launch_route(const RouteParams &p, hipStream_t st) {
  if (p.T == 0) return hipSuccess;
  const int waves_per_block = 4;
  dim3 grid((p.T + waves_per_block - 1) / waves_per_block), block(waves_per_block * kWave);
  if (p.E <= 64)
    hipLaunchKernelGGL(route_kernel<1>, grid, block, 0, st, p);
  else if (p.E <= 128)
    hipLaunchKernelGGL(route_kernel<2>, grid, block, 0, st, p);
  else if (p.E <= 256)
    hipLaunchKernelGGL(route_kernel<4>, grid, block, 0, st, p);
  else if (p.E <= 512)
    hipLaunchKernelGGL(route_kernel<8>, grid, block, 0, st, p);
  else
    hipLaunchKernelGGL(route_kernel<16>, grid, block, 0, st, p);
  return hipGetLastError();
}

// Test hook: the routing sigmoid applied elementwise.
namespace {
__global__ void sigmoid_kernel(const float *x, float *y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = sigmoid_spec(x[i]);
}
}  // namespace

hipError_t launch_debug_sigmoid(const float *x, float *y, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(sigmoid_kernel, dim3((unsigned)blocks), dim3(256), 0, st, x, y, n);
  return hipGetLastError();
}

}  // namespace moe
