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
    for (int j = 0; j < p.K; ++j) {
      const int le = p.topk_ids[(size_t)t * p.K + j] - p.offset;
      if (le >= 0 && le < p.El) atomicAdd(&hist[le], 1);
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

}  // namespace

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
