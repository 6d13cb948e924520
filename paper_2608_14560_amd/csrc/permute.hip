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
#include "moe_device.h"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxEl = 1024;

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

// Exclusive scan of v over the block (one value per thread); returns the
// exclusive prefix and writes the block total to *total.
__device__ int block_exclusive_scan(int v, int *wsum, int *total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  int x = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == kWave - 1) wsum[w] = x;
  __syncthreads();
  int before = 0, all = 0;
  for (int i = 0; i < kWaves; ++i) {
    if (i < w) before += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// SINGLE: the batch is one chunk; the workgroup counts its own pairs (an LDS
// histogram) instead of reading the count kernel's output.
template <bool SINGLE>
__global__ __launch_bounds__(kThreads) void scatter_kernel(PermuteParams p) {
  // per expert: start of this chunk's rows, then per-wave occupancy bitmaps
  __shared__ int base[kMaxEl];
  __shared__ int hist[SINGLE ? kMaxEl : 1];
  __shared__ unsigned long long bits[kWaves][kMaxEl];
  __shared__ int wsum[kWaves];

  const int chunk = blockIdx.x;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;

  for (int e = threadIdx.x; e < p.El; e += kThreads) {
    for (int i = 0; i < kWaves; ++i) bits[i][e] = 0ull;
    if (SINGLE) hist[e] = 0;
  }
  if (SINGLE) {
    __syncthreads();
    const int t = threadIdx.x;
    if (t < p.T)
      for (int j = 0; j < p.K; ++j) {
        const int le = p.topk_ids[(size_t)t * p.K + j] - p.offset;
        if (le >= 0 && le < p.El) atomicAdd(&hist[le], 1);
      }
    __syncthreads();
  }
  // count of local expert e in chunk c
  auto cnt = [&](int c, int e) {
    return SINGLE ? hist[e] : p.chunk_counts[(size_t)c * p.El + e];
  };

  // expert offsets: exclusive scan of the per-expert totals over all chunks.
  // Each thread owns a contiguous run of experts.
  const int per = (p.El + kThreads - 1) / kThreads;
  const int e0 = threadIdx.x * per;
  int tot_run = 0;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0, before = 0;
    for (int c = 0; c < p.nchunks; ++c) {
      const int n = cnt(c, e);
      tot += n;
      if (c < chunk) before += n;
    }
    base[e] = before;   // chunk-local part; the expert offset is added below
    tot_run += tot;
  }
  int P = 0;
  const int run_start = block_exclusive_scan(tot_run, wsum, &P);
  // walk the run again to turn totals into offsets
  int acc = run_start;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0;
    for (int c = 0; c < p.nchunks; ++c) tot += cnt(c, e);
    if (chunk == 0) p.expert_offsets[e] = acc;
    base[e] += acc;
    acc += tot;
  }
  if (chunk == 0 && threadIdx.x == 0) p.expert_offsets[p.El] = P;
  __syncthreads();

  // rank the chunk's pairs: bit `lane` of bits[w][e] marks that the lane's
  // token holds local expert e
  const int t = chunk * kChunkTokens + threadIdx.x;
  const bool live = t < p.T;
  if (live) {
    for (int j = 0; j < p.K; ++j) {
      const int le = p.topk_ids[(size_t)t * p.K + j] - p.offset;
      if (le >= 0 && le < p.El) atomicOr(&bits[w][le], 1ull << lane);
    }
  }
  __syncthreads();
  if (live) {
    const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int j = 0; j < p.K; ++j) {
      const int le = p.topk_ids[(size_t)t * p.K + j] - p.offset;
      int row = -1;
      if (le >= 0 && le < p.El) {
        row = base[le];
        for (int i = 0; i < w; ++i) row += __popcll(bits[i][le]);
        row += __popcll(bits[w][le] & below);
        p.perm_token[row] = t;
        p.perm_pair[row] = t * p.K + j;
      }
      p.pair_row[(size_t)t * p.K + j] = row;
    }
  }

  if (chunk != 0) return;

  // M-tile prefix per expert and the GEMM work-item counts
  __syncthreads();
  int tiles_run = 0;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0;
    for (int c = 0; c < p.nchunks; ++c) tot += cnt(c, e);
    tiles_run += (tot + p.BM - 1) / p.BM;
  }
  int n_tiles = 0;
  int tacc = block_exclusive_scan(tiles_run, wsum, &n_tiles);
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0;
    for (int c = 0; c < p.nchunks; ++c) tot += cnt(c, e);
    p.tile_base[e] = tacc;
    tacc += (tot + p.BM - 1) / p.BM;
  }
  if (threadIdx.x == 0) {
    p.tile_base[p.El] = n_tiles;
    p.n_items[0] = n_tiles * p.items_per_tile1;
    p.n_items[1] = n_tiles * p.items_per_tile2;
  }
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
