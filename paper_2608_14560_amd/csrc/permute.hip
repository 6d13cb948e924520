// permute.hip -- the bookkeeping of stage (2) of the Fused MoE block (paper
// Section 3.1.1): per-expert counts of the resident (token, slot) pairs,
// their exclusive scan, and the stable scatter of the pairs into one
// contiguous per-expert layout.  All sizes that depend on the routing stay
// on the device (no host synchronisation, as the paper's implementation
// keeps all metadata construction on the GPU).
//
// Two launches over chunks of kChunkTokens tokens:
//   count:   LDS histogram of the chunk's resident experts -> chunk_counts
//   scatter: every workgroup rebuilds the expert offsets from all chunk
//            counts, ranks its pairs inside the chunk with per-wave LDS
//            bitmaps (deterministic: a pair's position depends only on the
//            routing, never on timing), and writes perm_token / perm_pair /
//            pair_row.  Workgroup 0 also writes expert_offsets, the M-tile
//            prefix of every expert and the GEMM work-item counts.
#include "scatter_device.h"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxEl = kPermMaxEl;

__global__ __launch_bounds__(kThreads) void count_kernel(PermuteParams p) {
  __shared__ int hist[kMaxEl];
  for (int e = threadIdx.x; e < p.El; e += kThreads) hist[e] = 0;
  __syncthreads();
  const int t = blockIdx.x * kChunkTokens + threadIdx.x;
  if (t < p.T) {
    // the token's ids loaded together (clamped index), then counted
    int ids[kPermMaxK];
#pragma unroll
    for (int j = 0; j < kPermMaxK; ++j) ids[j] = p.topk_ids[(size_t)t * p.K + min(j, p.K - 1)];
#pragma unroll
    for (int j = 0; j < kPermMaxK; ++j) {
      const int le = ids[j] - p.offset;
      if (j < p.K && le >= 0 && le < p.El) atomicAdd(&hist[le], 1);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < p.El; e += kThreads)
    p.chunk_counts[(size_t)blockIdx.x * p.El + e] = hist[e];
}

template <bool SINGLE>
__global__ __launch_bounds__(kThreads) void scatter_kernel(PermuteParams p) {
  __shared__ ScatterLds<kThreads, SINGLE> sh;
  scatter_chunk<kThreads, SINGLE>(p, blockIdx.x, p.topk_ids, sh);
}

// The hidden rows' block scales in permuted order and K-block-major,
// hs_k[kb][r] = hidden_scale[perm_token[r]][kb], for the large-tile GEMM1
// (its per-K-step scale loads then cover a tile's rows with a few cache
// lines instead of one line per row).  Workgroup = 64 permuted rows: their
// scale rows are read whole (consecutive threads, consecutive K blocks of a
// row), transposed through LDS, and written 64 rows at a time per K block.
constexpr int kGatherRows = 64;
constexpr int kGatherMaxKB = 512;  // H <= 65536

__global__ __launch_bounds__(kThreads) void gather_scales_kernel(const int32_t *expert_offsets, int El,
                                                                 const int32_t *perm_token,
                                                                 const float *hidden_scale, float *hs_k,
                                                                 int KB, int P_max) {
  __shared__ int tok[kGatherRows];
  extern __shared__ float tr[];  // [KB][kGatherRows + 1]
  const int P = expert_offsets[El];
  const int r0 = blockIdx.x * kGatherRows;
  if (r0 >= P) return;
  const int n = min(kGatherRows, P - r0);
  if (threadIdx.x < kGatherRows) tok[threadIdx.x] = perm_token[r0 + min((int)threadIdx.x, n - 1)];
  __syncthreads();
  // eight loads per thread go out together before their LDS stores
  for (int i0 = threadIdx.x; i0 < kGatherRows * KB; i0 += 8 * kThreads) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = min(i0 + u * kThreads, kGatherRows * KB - 1);
      v[u] = hidden_scale[(size_t)tok[i / KB] * KB + i % KB];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * kThreads;
      if (i < kGatherRows * KB) tr[(i % KB) * (kGatherRows + 1) + i / KB] = v[u];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kGatherRows * KB; i += kThreads) {
    const int kb = i / kGatherRows, row = i % kGatherRows;
    if (row < n) hs_k[(size_t)kb * P_max + r0 + row] = tr[kb * (kGatherRows + 1) + row];
  }
}

}  // namespace

hipError_t launch_gather_scales(const int32_t *expert_offsets, int El, const int32_t *perm_token,
                                const float *hidden_scale, float *hs_k, int KB, int P_max,
                                hipStream_t st) {
  if (P_max <= 0 || KB <= 0) return hipSuccess;
  if (KB > kGatherMaxKB) return hipErrorInvalidValue;
  const size_t lds = sizeof(float) * (size_t)KB * (kGatherRows + 1);
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void *>(gather_scales_kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)(sizeof(float) * kGatherMaxKB * (kGatherRows + 1)));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(gather_scales_kernel, dim3((P_max + kGatherRows - 1) / kGatherRows), dim3(kThreads),
                     lds, st, expert_offsets, El, perm_token, hidden_scale, hs_k, KB, P_max);
  return hipGetLastError();
}

// A batch of one chunk needs no count launch: the scatter counts for itself.
hipError_t launch_permute_count(const PermuteParams &p, hipStream_t st) {
  if (p.nchunks == 1) return hipSuccess;
  hipLaunchKernelGGL(count_kernel, dim3(p.nchunks), dim3(kThreads), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_permute_scatter(const PermuteParams &p, hipStream_t st) {
  if (p.nchunks == 1)
    hipLaunchKernelGGL(scatter_kernel<true>, dim3(1), dim3(kThreads), 0, st, p);
  else
    hipLaunchKernelGGL(scatter_kernel<false>, dim3(p.nchunks), dim3(kThreads), 0, st, p);
  return hipGetLastError();
}

}  // namespace moe
