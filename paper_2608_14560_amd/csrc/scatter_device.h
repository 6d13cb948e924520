// scatter_device.h -- the stable scatter of stage (2) of the Fused MoE block
// (paper Section 3.1.1): per-expert offsets from the chunk counts, stable
// ranks of a chunk's (token, slot) pairs, and the permuted-order arrays,
// for a workgroup of any size NT >= 256.
#pragma once
#include "moe_device.h"

namespace moe {

constexpr int kPermMaxEl = 1024;
constexpr int kPermTokenWaves = kChunkTokens / kWave;  // waves that hold a chunk's tokens

// LDS of one scatter workgroup of NT threads.  SINGLE: the batch is one chunk
// and the workgroup counts its own pairs.
template <int NT, bool SINGLE>
struct ScatterLds {
  int base[kPermMaxEl];
  int hist[SINGLE ? kPermMaxEl : 1];
  unsigned long long bits[kPermTokenWaves][kPermMaxEl];
  int wsum[NT / kWave];
};

// Exclusive scan of v over the NT threads (one value per thread); returns the
// exclusive prefix and writes the total to *total.  Every thread must call it.
template <int NT>
__device__ int scatter_block_scan(int v, int *wsum, int *total) {
  constexpr int NW = NT / kWave;
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
  for (int i = 0; i < NW; ++i) {
    if (i < w) before += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// Scatter of chunk `chunk` (tokens [256 chunk, 256 chunk + 256)); thread t of
// the first 256 holds token 256 chunk + t.  `ids` is the [T, K] routing
// output (global or LDS).  Workgroup 0 also writes expert_offsets, the M-tile
// prefix of every expert and the GEMM work-item counts.  Every thread of the
// workgroup must call it (it contains barriers).
template <int NT, bool SINGLE>
__device__ void scatter_chunk(const PermuteParams &p, int chunk, const int32_t *ids,
                              ScatterLds<NT, SINGLE> &sh) {
  static_assert(NT >= kChunkTokens, "a thread per token of the chunk");
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;

  for (int e = threadIdx.x; e < p.El; e += NT) {
    for (int i = 0; i < kPermTokenWaves; ++i) sh.bits[i][e] = 0ull;
    if (SINGLE) sh.hist[e] = 0;
  }
  if (SINGLE) {
    __syncthreads();
    const int t = threadIdx.x;
    if (t < p.T && t < kChunkTokens)
      for (int j = 0; j < p.K; ++j) {
        const int le = ids[(size_t)t * p.K + j] - p.offset;
        if (le >= 0 && le < p.El) atomicAdd(&sh.hist[le], 1);
      }
    __syncthreads();
  }
  // count of local expert e in chunk c
  auto cnt = [&](int c, int e) {
    return SINGLE ? sh.hist[e] : p.chunk_counts[(size_t)c * p.El + e];
  };

  // expert offsets: exclusive scan of the per-expert totals over all chunks.
  // Each thread owns a contiguous run of experts.
  const int per = (p.El + NT - 1) / NT;
  const int e0 = threadIdx.x * per;
  int tot_run = 0;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0, before = 0;
    for (int c = 0; c < p.nchunks; ++c) {
      const int n = cnt(c, e);
      tot += n;
      if (c < chunk) before += n;
    }
    sh.base[e] = before;  // chunk-local part; the expert offset is added below
    tot_run += tot;
  }
  int P = 0;
  const int run_start = scatter_block_scan<NT>(tot_run, sh.wsum, &P);
  // walk the run again to turn totals into offsets
  int acc = run_start;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0;
    for (int c = 0; c < p.nchunks; ++c) tot += cnt(c, e);
    if (chunk == 0) p.expert_offsets[e] = acc;
    sh.base[e] += acc;
    acc += tot;
  }
  if (chunk == 0 && threadIdx.x == 0) p.expert_offsets[p.El] = P;
  __syncthreads();

  // rank the chunk's pairs: bit `lane` of bits[w][e] marks that the lane's
  // token holds local expert e
  const int t = chunk * kChunkTokens + threadIdx.x;
  const bool live = threadIdx.x < kChunkTokens && t < p.T;
  if (live) {
    for (int j = 0; j < p.K; ++j) {
      const int le = ids[(size_t)t * p.K + j] - p.offset;
      if (le >= 0 && le < p.El) atomicOr(&sh.bits[w][le], 1ull << lane);
    }
  }
  __syncthreads();
  if (live) {
    const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int j = 0; j < p.K; ++j) {
      const int le = ids[(size_t)t * p.K + j] - p.offset;
      int row = -1;
      if (le >= 0 && le < p.El) {
        row = sh.base[le];
        for (int i = 0; i < w; ++i) row += __popcll(sh.bits[i][le]);
        row += __popcll(sh.bits[w][le] & below);
        p.perm_token[row] = t;
        p.perm_pair[row] = t * p.K + j;
      }
      p.pair_row[(size_t)t * p.K + j] = row;
    }
  }

  if (chunk != 0) return;  // uniform over the workgroup

  // M-tile prefix per expert and the GEMM work-item counts
  __syncthreads();
  int tiles_run = 0;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0;
    for (int c = 0; c < p.nchunks; ++c) tot += cnt(c, e);
    tiles_run += (tot + p.BM - 1) / p.BM;
  }
  int n_tiles = 0;
  int tacc = scatter_block_scan<NT>(tiles_run, sh.wsum, &n_tiles);
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

}  // namespace moe
