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

// Wave-wide argmax under `beats` with DPP: (value, index) is packed into one
// 64-bit key that orders like `beats` (value bits mapped to an unsigned order,
// index complemented so that the lower index wins a tie), reduced with
// row_shr 1/2/4/8 inside each 16-lane row and row_bcast 15/31 across rows,
// and read back from lane 63.  Returns the winner's index; every lane gets it.
__device__ __forceinline__ uint32_t ordered_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void dpp_max_step(uint32_t &hi, uint32_t &lo) {
  // lanes whose DPP source is outside the row (or not selected) see key 0,
  // which no packed key of a real score undercuts
  const uint32_t nh = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)hi, CTRL, ROW_MASK, 0xf, false);
  const uint32_t nl = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lo, CTRL, ROW_MASK, 0xf, false);
  const bool take = nh > hi || (nh == hi && nl > lo);
  hi = take ? nh : hi;
  lo = take ? nl : lo;
}

__device__ __forceinline__ int wave_argmax(float v, int idx) {
  uint32_t hi = ordered_bits(v);
  uint32_t lo = ~(uint32_t)idx;
  dpp_max_step<0x111, 0xf>(hi, lo);  // row_shr:1
  dpp_max_step<0x112, 0xf>(hi, lo);  // row_shr:2
  dpp_max_step<0x114, 0xf>(hi, lo);  // row_shr:4
  dpp_max_step<0x118, 0xf>(hi, lo);  // row_shr:8
  dpp_max_step<0x142, 0xa>(hi, lo);  // row_bcast:15 into rows 1 and 3
  dpp_max_step<0x143, 0xc>(hi, lo);  // row_bcast:31 into rows 2 and 3
  return (int)~(uint32_t)__builtin_amdgcn_readlane((int)lo, 63);
}

constexpr int kNoIdx = 0x7fffffff;

// Value of expert `e` (wave-uniform) from the per-lane slots: lane e % 64,
// slot e / 64.
template <int EPL>
__device__ __forceinline__ float key_of(const float (&v)[EPL], int e) {
  const int slot = e / kWave, src = e % kWave;
  float x = v[0];
#pragma unroll
  for (int q = 1; q < EPL; ++q)
    if (q == slot) x = v[q];
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), src));
}

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
    float v1 = -INFINITY, v2 = -INFINITY;
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
    // best of the group, then the second best: the lane that held the best
    // offers its runner-up instead
    const int bi = wave_argmax(v1, i1);
    const bool had = (i1 == bi);
    const int si = wave_argmax(had ? v2 : v1, had ? i2 : i1);
    // both values live in known lanes/slots: fetch them by index
    const float bv = key_of(key, bi);
    const float sv = key_of(key, si);
    const float gs = bv + sv;
    if (lane == g) my_gs = gs;
  }

  // keep the topk_group best groups: a group is kept when fewer than
  // topk_group groups beat it
  int rank = 0;
  for (int g = 0; g < p.G; ++g) {
    const float og = __builtin_bit_cast(
        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_gs), g));
    if (lane < p.G && g != lane && beats(og, g, my_gs, lane)) ++rank;
  }
  const uint64_t kept = __ballot(lane < p.G && rank < p.TG);
  bool cand[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    cand[q] = (e < p.E) && ((kept >> (e / gsz)) & 1ull);
  }

  // top-k experts among the kept groups, in selection order
  int my_id = 0;
  float my_s = 0.0f;
  for (int j = 0; j < p.K; ++j) {
    float bv = -INFINITY;
    int bi = kNoIdx;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const int e = q * kWave + lane;
      if (cand[q] && beats(key[q], e, bv, bi)) {
        bv = key[q];
        bi = e;
      }
    }
    const int win = wave_argmax(bv, bi);
#pragma unroll
    for (int q = 0; q < EPL; ++q)
      if (q * kWave + lane == win) cand[q] = false;
    const float ws = key_of(sc, win);
    if (lane == j) {
      my_id = win;
      my_s = ws;
    }
  }

  // weights: unbiased scores normalised over the k selections (summed in
  // selection order), times the routed scaling factor
  float sum = 0.0f;
  for (int j = 0; j < p.K; ++j)
    sum += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_s), j));
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
