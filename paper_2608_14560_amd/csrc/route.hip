// route.hip -- stage (1) of the Fused MoE block (paper Section 3.1.1):
// sigmoid routing scores, group-limited top-k expert selection and the
// normalised, scaled routing weights.  One wave64 per token: the group
// scores by DPP reductions over the wave, the top-k by a bounded rank through
// LDS (or a ballot radix select); no block barrier.
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

// Top-K experts among the candidates, in selection order: key descending, the
// lower expert id first among equal keys (the order of K successive wave
// arg-maxes, without their K dependent reduction chains).  A bitwise radix
// select over the ordered key bits finds the K-th largest key: per bit, one
// ballot per slot counts the candidates that match the prefix so far with that
// bit set.  Every candidate above the threshold wins, and those equal to it
// win in ascending id order until K are taken.  The winners go to LDS in id
// order, each ranks itself among them, and lane j < K returns winner j.
// K <= 16 (validated on the host); the wave works alone (no block barrier).
constexpr int kRouteWaves = 4;   // waves per routing workgroup
constexpr int kMaxTopK = 16;

__device__ __forceinline__ int lanes_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

//
// With a lower bound (bh, bl) on the K-th largest packed key (value bits, then
// the complemented id) known, only the candidates at or above it can win; when
// at most 64 of them are, each takes a lane and counts the others that beat it
// (LDS broadcast reads): its rank is its output slot, and nothing else runs.
template <int EPL>
__device__ __forceinline__ void select_topk(const float (&key)[EPL], const float (&sc)[EPL],
                                            const bool (&cand)[EPL], int K, int lane, int &my_id,
                                            float &my_s, bool bounded = false, uint32_t bh = 0u,
                                            uint32_t bl = 0u) {
  __shared__ uint32_t sel_hi[kRouteWaves][kWave];
  __shared__ int sel_e[kRouteWaves][kWave];
  __shared__ float sel_s[kRouteWaves][kWave];
  __shared__ int out_e[kRouteWaves][kMaxTopK];
  __shared__ float out_s[kRouteWaves][kMaxTopK];
  const int wave = threadIdx.x / kWave;

  uint32_t hi[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) hi[q] = ordered_bits(key[q]);

  if (bounded) {
    bool f[EPL];
    int n = 0;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const uint32_t lo = ~(uint32_t)(q * kWave + lane);
      f[q] = cand[q] && (hi[q] > bh || (hi[q] == bh && lo >= bl));
      n += __popcll(__ballot(f[q]));
    }
    if (n <= kWave) {
      int pos_base = 0;
#pragma unroll
      for (int q = 0; q < EPL; ++q) {
        const uint64_t fm = __ballot(f[q]);
        const int pos = pos_base + lanes_below(fm);
        if (f[q]) {  // pos < n <= 64
          sel_hi[wave][pos] = hi[q];
          sel_e[wave][pos] = q * kWave + lane;
          sel_s[wave][pos] = sc[q];
        }
        pos_base += __popcll(fm);
      }
      wave_lds_sync();
      if (lane < n) {
        const uint32_t h = sel_hi[wave][lane];
        int rank = 0;
        for (int i = 0; i < n; ++i) {
          const uint32_t hi_i = sel_hi[wave][i];
          rank += (hi_i > h || (hi_i == h && i < lane)) ? 1 : 0;
        }
        if (rank < K) {
          out_e[wave][rank] = sel_e[wave][lane];
          out_s[wave][rank] = sel_s[wave][lane];
        }
      }
      wave_lds_sync();
      if (lane < K) {
        my_id = out_e[wave][lane];
        my_s = out_s[wave][lane];
      }
      return;
    }
  }

  uint32_t thr = 0;
  int need = K;
  for (int b = 31; b >= 0; --b) {
    const uint32_t target = (thr >> b) | 1u;
    int c = 0;
#pragma unroll
    for (int q = 0; q < EPL; ++q) c += __popcll(__ballot(cand[q] && (hi[q] >> b) == target));
    if (c >= need)
      thr |= 1u << b;
    else
      need -= c;
  }
  // winners, then their slots in id order (slot-major: id = q * 64 + lane)
  int tie_base = 0, pos_base = 0;
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const bool eq = cand[q] && hi[q] == thr;
    const uint64_t em = __ballot(eq);
    const bool win = cand[q] && (hi[q] > thr || (eq && tie_base + lanes_below(em) < need));
    tie_base += __popcll(em);
    const uint64_t wm = __ballot(win);
    const int pos = pos_base + lanes_below(wm);
    if (win && pos < kMaxTopK) {  // exactly K winners; the bound only guards the array
      sel_hi[wave][pos] = hi[q];
      sel_e[wave][pos] = q * kWave + lane;
      sel_s[wave][pos] = sc[q];
    }
    pos_base += __popcll(wm);
  }
  wave_lds_sync();
  if (lane < K) {
    const uint32_t h = sel_hi[wave][lane];
    int rank = 0;
    for (int i = 0; i < K; ++i) {
      const uint32_t hi_i = sel_hi[wave][i];
      rank += (hi_i > h || (hi_i == h && i < lane)) ? 1 : 0;
    }
    out_e[wave][rank] = sel_e[wave][lane];
    out_s[wave][rank] = sel_s[wave][lane];
  }
  wave_lds_sync();
  if (lane < K) {
    my_id = out_e[wave][lane];
    my_s = out_s[wave][lane];
  }
}

// The bias of the lane's experts, loaded unconditionally (clamped index) so the
// loads go out with the logits' and the sigmoids below run without branches:
// per-slot branches around a load serialise one round trip per slot.
template <int EPL>
__device__ __forceinline__ void load_bias(const RouteParams &p, int lane, float (&bs)[EPL]) {
#pragma unroll
  for (int q = 0; q < EPL; ++q) bs[q] = p.bias[min(q * kWave + lane, p.E - 1)];
}

// EPL = experts held per lane (expert e lives in lane e % 64, slot e / 64).
// GC = number of groups when known at compile time (its group reductions are
// then independent chains the compiler interleaves), 0 for a runtime count.
template <int EPL, int GC>
__global__ __launch_bounds__(256) void route_kernel(RouteParams p) {
  constexpr int GMAX = GC > 0 ? GC : 64;
  const int G = GC > 0 ? GC : p.G;
  const int lane = threadIdx.x & (kWave - 1);
  // the token is uniform over the wave: readfirstlane lets its row addresses
  // (scales, logits) live in scalar registers
  const int t = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave));
  if (t >= p.T) return;  // whole wave leaves; the kernel has no block barrier

  const int gsz = p.E / G;

  float sc[EPL], key[EPL], lg[EPL], bs[EPL];
  load_bias<EPL>(p, lane, bs);
  route_logits<EPL>(p, t, lane, lg);
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    const float s = sigmoid_spec(lg[q]);
    sc[q] = e < p.E ? s : 0.0f;
    key[q] = e < p.E ? s + bs[q] : -INFINITY;
  }

  // group score = sum of the two largest keys of the group
  float my_gs = -INFINITY;  // lane g keeps the score of group g
  if (GC > 0) {
    float v1[GMAX], v2[GMAX];
    int i1[GMAX], i2[GMAX];
#pragma unroll
    for (int g = 0; g < GMAX; ++g) {
      v1[g] = v2[g] = -INFINITY;
      i1[g] = i2[g] = kNoIdx;
#pragma unroll
      for (int q = 0; q < EPL; ++q) {
        const int e = q * kWave + lane;
        if (e < p.E && e / gsz == g) {
          if (beats(key[q], e, v1[g], i1[g])) {
            v2[g] = v1[g]; i2[g] = i1[g];
            v1[g] = key[q]; i1[g] = e;
          } else if (beats(key[q], e, v2[g], i2[g])) {
            v2[g] = key[q]; i2[g] = e;
          }
        }
      }
    }
    int b[GMAX];
#pragma unroll
    for (int g = 0; g < GMAX; ++g) b[g] = wave_argmax(v1[g], i1[g]);
#pragma unroll
    for (int g = 0; g < GMAX; ++g) {
      const bool had = (i1[g] == b[g]);
      const int si = wave_argmax(had ? v2[g] : v1[g], had ? i2[g] : i1[g]);
      const float gs = key_of(key, b[g]) + key_of(key, si);
      if (lane == g) my_gs = gs;
    }
  } else {
    for (int g = 0; g < G; ++g) {
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
      const float gs = key_of(key, bi) + key_of(key, si);
      if (lane == g) my_gs = gs;
    }
  }

  // keep the topk_group best groups: a group is kept when fewer than
  // topk_group groups beat it
  int rank = 0;
#pragma unroll
  for (int g = 0; g < GMAX; ++g) {
    if (g < G) {
      const float og = __builtin_bit_cast(
          float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_gs), g));
      if (lane < G && g != lane && beats(og, g, my_gs, lane)) ++rank;
    }
  }
  const uint64_t kept = __ballot(lane < G && rank < p.TG);
  bool cand[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    cand[q] = (e < p.E) && ((kept >> (e / gsz)) & 1ull);
  }

  // top-k experts among the kept groups, in selection order
  int my_id = 0;
  float my_s = 0.0f;
  select_topk<EPL>(key, sc, cand, p.K, lane, my_id, my_s);

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

// ---------------------------------------------------------------------------
// Fast path for groups of S = E/G experts, S a power of two dividing 64: the
// experts of a group then sit in S consecutive lanes of one slot, and one
// segmented DPP pass (row_shr 1/2/4/8 masked to the segment, row_bcast 15/31
// for 32- and 64-lane segments) leaves every group's best and runner-up keys
// in the last lane of its segment -- all groups and slots at once instead of
// 2*G wave-wide reductions.  Keys travel as 64-bit ordered words (value bits,
// complemented index) so that every comparison is the `beats` order.
// ---------------------------------------------------------------------------
struct Key2 {  // best (a) and runner-up (b)
  uint32_t ah, al, bh, bl;
};

__device__ __forceinline__ bool key_gt(uint32_t h1, uint32_t l1, uint32_t h0, uint32_t l0) {
  return h1 > h0 || (h1 == h0 && l1 > l0);
}

// merge a neighbour's top-2 (n) into k; `ok` false discards the neighbour
__device__ __forceinline__ void key2_merge(Key2 &k, const Key2 &n, bool ok) {
  const bool nw = ok && key_gt(n.ah, n.al, k.ah, k.al);
  // runner-up candidates: the loser of the two bests, and the winner's own second
  const uint32_t ch = nw ? k.ah : k.bh, cl = nw ? k.al : k.bl;
  const uint32_t dh = nw ? n.bh : (ok ? n.ah : 0u), dl = nw ? n.bl : (ok ? n.al : 0u);
  const bool dw = key_gt(dh, dl, ch, cl);
  k.ah = nw ? n.ah : k.ah;
  k.al = nw ? n.al : k.al;
  k.bh = dw ? dh : ch;
  k.bl = dw ? dl : cl;
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ Key2 key2_dpp(const Key2 &k) {
  Key2 n;
  n.ah = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)k.ah, CTRL, ROW_MASK, 0xf, false);
  n.al = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)k.al, CTRL, ROW_MASK, 0xf, false);
  n.bh = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)k.bh, CTRL, ROW_MASK, 0xf, false);
  n.bl = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)k.bl, CTRL, ROW_MASK, 0xf, false);
  return n;
}

__device__ __forceinline__ float key_value(uint32_t h) {
  const uint32_t u = (h & 0x80000000u) ? (h & 0x7fffffffu) : ~h;
  return __uint_as_float(u);
}

// Routing of token t by one wave (power-of-two group size S): writes the
// token's ids and weights.
template <int EPL, int S>
__device__ __forceinline__ void route_token_seg(const RouteParams &p, int t) {
  const int lane = threadIdx.x & (kWave - 1);
  const int seg_lane = lane & (S - 1);

  float sc[EPL], key[EPL], lg[EPL], bs[EPL];
  Key2 k2[EPL];
  load_bias<EPL>(p, lane, bs);
  route_logits<EPL>(p, t, lane, lg);
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    const bool v = e < p.E;
    const float s = sigmoid_spec(lg[q]);
    sc[q] = v ? s : 0.0f;
    key[q] = v ? s + bs[q] : -INFINITY;
    k2[q].ah = v ? ordered_bits(key[q]) : 0u;
    k2[q].al = ~(uint32_t)e;
    k2[q].bh = 0u;
    k2[q].bl = 0u;
  }
  // segmented top-2: after the steps the last lane of each segment holds its
  // group's best and runner-up
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    if (S >= 2) key2_merge(k2[q], key2_dpp<0x111, 0xf>(k2[q]), seg_lane >= 1);
    if (S >= 4) key2_merge(k2[q], key2_dpp<0x112, 0xf>(k2[q]), seg_lane >= 2);
    if (S >= 8) key2_merge(k2[q], key2_dpp<0x114, 0xf>(k2[q]), seg_lane >= 4);
    if (S >= 16) key2_merge(k2[q], key2_dpp<0x118, 0xf>(k2[q]), seg_lane >= 8);
    if (S >= 32) key2_merge(k2[q], key2_dpp<0x142, 0xa>(k2[q]), seg_lane >= 16);
    if (S >= 64) key2_merge(k2[q], key2_dpp<0x143, 0xc>(k2[q]), seg_lane >= 32);
  }
  // group score of the segment ending in this lane
  float seg_gs[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) seg_gs[q] = key_value(k2[q].ah) + key_value(k2[q].bh);

  // lane g collects the score of group g (group g = slot * 64/S + segment)
  constexpr int SEGS = kWave / S;
  const int G = p.G;
  float my_gs = -INFINITY;
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
#pragma unroll
    for (int sg = 0; sg < SEGS; ++sg) {
      const int g = q * SEGS + sg;
      if (g < G) {
        const float v = __builtin_bit_cast(
            float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, seg_gs[q]), sg * S + S - 1));
        my_gs = (lane == g) ? v : my_gs;
      }
    }
  }
  int rank = 0;
  for (int g = 0; g < G; ++g) {
    const float og = __builtin_bit_cast(
        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_gs), g));
    rank += (lane < G && g != lane && beats(og, g, my_gs, lane)) ? 1 : 0;
  }
  const uint64_t kept = __ballot(lane < G && rank < p.TG);
  bool cand[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * kWave + lane;
    cand[q] = (e < p.E) && ((kept >> (e / S)) & 1ull);
  }

  // top-k experts among the kept groups, in selection order.  When K <= 2 *
  // topk_group the K-th largest key is at least the smallest runner-up of the
  // kept groups (their bests and runner-ups are 2 * topk_group candidates).
  uint32_t bh = 0xffffffffu, bl = 0xffffffffu;
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
#pragma unroll
    for (int sg = 0; sg < SEGS; ++sg) {
      const int g = q * SEGS + sg;
      if (g < G && ((kept >> g) & 1ull)) {
        const uint32_t h = (uint32_t)__builtin_amdgcn_readlane((int)k2[q].bh, sg * S + S - 1);
        const uint32_t l = (uint32_t)__builtin_amdgcn_readlane((int)k2[q].bl, sg * S + S - 1);
        if (key_gt(bh, bl, h, l)) {
          bh = h;
          bl = l;
        }
      }
    }
  }
  int my_id = 0;
  float my_s = 0.0f;
  select_topk<EPL>(key, sc, cand, p.K, lane, my_id, my_s, p.K <= 2 * p.TG, bh, bl);

  float sum = 0.0f;
  for (int j = 0; j < p.K; ++j)
    sum += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_s), j));
  if (lane < p.K) {
    p.topk_ids[(size_t)t * p.K + lane] = my_id;
    p.topk_w[(size_t)t * p.K + lane] = (my_s / sum) * p.rsf;
  }
}

template <int EPL, int S>
__global__ __launch_bounds__(256) void route_seg_kernel(RouteParams p) {
  const int t = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave));
  if (t >= p.T) return;
  route_token_seg<EPL, S>(p, t);
}

template <int EPL>
bool launch_route_seg(const RouteParams &p, dim3 grid, dim3 block, hipStream_t st) {
  const int S = p.E / p.G;
  if (p.E > kWave && p.E % kWave) return false;
  switch (S) {
    case 4: hipLaunchKernelGGL((route_seg_kernel<EPL, 4>), grid, block, 0, st, p); return true;
    case 8: hipLaunchKernelGGL((route_seg_kernel<EPL, 8>), grid, block, 0, st, p); return true;
    case 16: hipLaunchKernelGGL((route_seg_kernel<EPL, 16>), grid, block, 0, st, p); return true;
    case 32: hipLaunchKernelGGL((route_seg_kernel<EPL, 32>), grid, block, 0, st, p); return true;
    case 64: hipLaunchKernelGGL((route_seg_kernel<EPL, 64>), grid, block, 0, st, p); return true;
    default: return false;
  }
}

template <int EPL>
void launch_route_epl(const RouteParams &p, dim3 grid, dim3 block, hipStream_t st) {
  if (launch_route_seg<EPL>(p, grid, block, st)) return;
  switch (p.G) {
    case 8: hipLaunchKernelGGL((route_kernel<EPL, 8>), grid, block, 0, st, p); break;
    case 4: hipLaunchKernelGGL((route_kernel<EPL, 4>), grid, block, 0, st, p); break;
    case 2: hipLaunchKernelGGL((route_kernel<EPL, 2>), grid, block, 0, st, p); break;
    default: hipLaunchKernelGGL((route_kernel<EPL, 0>), grid, block, 0, st, p); break;
  }
}

}  // namespace

hipError_t launch_route(const RouteParams &p, hipStream_t st) {
  if (p.T == 0) return hipSuccess;
  const int waves_per_block = kRouteWaves;
  dim3 grid((p.T + waves_per_block - 1) / waves_per_block), block(waves_per_block * kWave);
  if (p.E <= 64)
    launch_route_epl<1>(p, grid, block, st);
  else if (p.E <= 128)
    launch_route_epl<2>(p, grid, block, st);
  else if (p.E <= 256)
    launch_route_epl<4>(p, grid, block, st);
  else if (p.E <= 512)
    launch_route_epl<8>(p, grid, block, st);
  else
    launch_route_epl<16>(p, grid, block, st);
  return hipGetLastError();
}

// Test hook: the logits the routing kernels form (from the router
// projection's block sums, or as given).
namespace {
template <int EPL>
__global__ __launch_bounds__(256) void logits_kernel(RouteParams p, float *logits) {
  // one wave per token, as in the routing kernels
  const int t = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave);
  const int lane = threadIdx.x & (kWave - 1);
  if (t >= p.T) return;
  float lg[EPL];
  route_logits<EPL>(p, t, lane, lg);
#pragma unroll
  for (int q = 0; q < EPL; ++q)
    if (q * kWave + lane < p.E) logits[(size_t)t * p.E + q * kWave + lane] = lg[q];
}
}  // namespace

hipError_t launch_router_logits(const RouteParams &p, float *logits, hipStream_t st) {
  if (p.T <= 0) return hipSuccess;
  const dim3 grid((p.T + 3) / 4), block(256);
  if (p.E <= 64)
    hipLaunchKernelGGL(logits_kernel<1>, grid, block, 0, st, p, logits);
  else if (p.E <= 128)
    hipLaunchKernelGGL(logits_kernel<2>, grid, block, 0, st, p, logits);
  else if (p.E <= 256)
    hipLaunchKernelGGL(logits_kernel<4>, grid, block, 0, st, p, logits);
  else if (p.E <= 512)
    hipLaunchKernelGGL(logits_kernel<8>, grid, block, 0, st, p, logits);
  else
    hipLaunchKernelGGL(logits_kernel<16>, grid, block, 0, st, p, logits);
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
