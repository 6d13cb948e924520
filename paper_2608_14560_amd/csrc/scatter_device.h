// scatter_device.h -- the stable scatter of stage (2) of the Fused MoE block
// (paper Section 3.1.1): per-expert offsets from the chunk counts, stable
// ranks of a chunk's (token, slot) pairs, and the permuted-order arrays,
// for a workgroup of any size NT >= 256.
#pragma once
#include "moe_device.h"

namespace moe {

constexpr int kPermMaxEl = 1024;
constexpr int kPermTokenWaves = kChunkTokens / kWave;  // waves that hold a chunk's tokens
constexpr int kPermMaxK = 16;                           // top_k limit of the shape check

// LDS of one scatter workgroup of NT threads.  SINGLE: the batch is one chunk
// and the workgroup counts its own pairs.
template <int NT, bool SINGLE>
struct ScatterLds {
  int base[kPermMaxEl];
  int hist[SINGLE ? kPermMaxEl : 1];
  unsigned long long bits[kPermTokenWaves][kPermMaxEl];
  int wsum[NT / kWave][2];
  int cbase[kPermMaxEl];  // chunk-local start of each expert's pairs
  int tot[kPermMaxEl];    // each expert's pairs over all chunks
  int mine[kPermMaxEl];   // each expert's pairs in this chunk
  int srow[kChunkTokens * kPermMaxK];   // the chunk's pairs in output order:
  int spair[kChunkTokens * kPermMaxK];  // row and t K + j
};

// Inclusive scan over the wave with DPP: a window of four lanes (row_shr 1, 2,
// 3 of the original values), then row_shr 4 and 8 into the upper lanes of each
// 16-lane row, then row_bcast 15 and 31 across rows.
template <int kCtrl, int kRows, int kBanks>
__device__ __forceinline__ int scan_dpp(int v) {
  return __builtin_amdgcn_update_dpp(0, v, kCtrl, kRows, kBanks, false);
}
__device__ __forceinline__ int wave_incl_scan(int v) {
  int x = v + scan_dpp<0x111, 0xf, 0xf>(v);
  x += scan_dpp<0x112, 0xf, 0xf>(v);
  x += scan_dpp<0x113, 0xf, 0xf>(v);
  x += scan_dpp<0x114, 0xf, 0xe>(x);
  x += scan_dpp<0x118, 0xf, 0xc>(x);
  x += scan_dpp<0x142, 0xa, 0xf>(x);
  x += scan_dpp<0x143, 0xc, 0xf>(x);
  return x;
}

// Exclusive scans of two values over the NT threads (one pair per thread):
// the prefixes and the totals.  Every thread must call it.
template <int NT>
__device__ void scatter_block_scan2(int a, int b, int (*wsum)[2], int &pa, int &pb, int &ta, int &tb) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int xa = wave_incl_scan(a), xb = wave_incl_scan(b);
  if (lane == kWave - 1) {
    wsum[w][0] = xa;
    wsum[w][1] = xb;
  }
  __syncthreads();
  int ba = 0, bb = 0, aa = 0, ab = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int va = wsum[i][0], vb = wsum[i][1];
    ba += i < w ? va : 0;
    bb += i < w ? vb : 0;
    aa += va;
    ab += vb;
  }
  pa = ba + xa - a;
  pb = bb + xb - b;
  ta = aa;
  tb = ab;
}

// Scatter of chunk `chunk` (tokens [256 chunk, 256 chunk + 256)); thread t of
// the first 256 holds token 256 chunk + t and keeps its K expert ids in
// registers for the three passes (count, mark, rank).  `ids` is the [T, K]
// routing output.  Workgroup 0 also writes expert_offsets, the M-tile prefix
// of every expert, the per-M-tile table and the GEMM work-item counts (one combined scan of the
// per-expert pair counts and tile counts).  Every thread of the workgroup must
// call it (it contains barriers).
template <int NT, bool SINGLE>
__device__ void scatter_chunk(const PermuteParams &p, int chunk, const int32_t *ids,
                              ScatterLds<NT, SINGLE> &sh) {
  static_assert(NT >= kChunkTokens, "a thread per token of the chunk");
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int t = chunk * kChunkTokens + threadIdx.x;
  const bool live = threadIdx.x < kChunkTokens && t < p.T;

  // the token's local expert ids (-1: not resident, or past K); the loads are
  // unconditional (clamped indices) so they all go out at once
  int le[kPermMaxK];
  {
    const int tc = min(t, p.T - 1);
#pragma unroll
    for (int j = 0; j < kPermMaxK; ++j) {
      const int x = ids[(size_t)tc * p.K + min(j, p.K - 1)] - p.offset;
      le[j] = (live && j < p.K && x >= 0 && x < p.El) ? x : -1;
    }
  }

  for (int e = threadIdx.x; e < p.El; e += NT) {
    for (int i = 0; i < kPermTokenWaves; ++i) sh.bits[i][e] = 0ull;
    if (SINGLE) sh.hist[e] = 0;
  }
  __syncthreads();
  if (SINGLE) {
#pragma unroll
    for (int j = 0; j < kPermMaxK; ++j)
      if (le[j] >= 0) atomicAdd(&sh.hist[le[j]], 1);
    __syncthreads();
  }
  // count of local expert e in chunk c
  auto cnt = [&](int c, int e) {
    return SINGLE ? sh.hist[e] : p.chunk_counts[(size_t)c * p.El + e];
  };

  // per-expert totals over all chunks.  Each thread owns a contiguous run of
  // experts: its pair and tile totals enter one block scan.
  const int per = (p.El + NT - 1) / NT;
  const int e0 = threadIdx.x * per;
  int tot_run = 0, tiles_run = 0;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    int tot = 0, before = 0, mine = 0;
    // the chunks' counts eight at a time, so that their loads go out together
    for (int c0 = 0; c0 < p.nchunks; c0 += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = c0 + u < p.nchunks ? cnt(c0 + u, e) : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        tot += v[u];
        before += c0 + u < chunk ? v[u] : 0;
        mine += c0 + u == chunk ? v[u] : 0;
      }
    }
    sh.base[e] = before;  // chunk-local part; the expert offset is added below
    sh.tot[e] = tot;
    sh.mine[e] = mine;
    tot_run += tot;
    tiles_run += (tot + p.BM - 1) / p.BM;
  }
  int run_start, tile_start, P, n_tiles;
  scatter_block_scan2<NT>(tot_run, tiles_run, sh.wsum, run_start, tile_start, P, n_tiles);
  // walk the run again: expert offsets, M-tile prefix
  int acc = run_start, tacc = tile_start;
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    const int tot = sh.tot[e];
    if (chunk == 0) {
      p.expert_offsets[e] = acc;
      p.tile_base[e] = tacc;
      const int nt = (tot + p.BM - 1) / p.BM;
      for (int t = 0; t < nt; ++t)
        reinterpret_cast<int4 *>(p.tile_tab)[tacc + t] = make_int4(e, tacc, acc, tot);
    }
    sh.base[e] += acc;
    acc += tot;
    tacc += (tot + p.BM - 1) / p.BM;
  }
  if (chunk == 0 && threadIdx.x == 0) {
    p.expert_offsets[p.El] = P;
    p.tile_base[p.El] = n_tiles;
    p.n_items[0] = n_tiles * p.items_per_tile1;
    p.n_items[1] = n_tiles * p.items_per_tile2;
  }

  // chunk-local starts of the experts' pair runs: one more scan over the
  // experts' counts in this chunk (same contiguous runs per thread)
  int crun = 0;
  for (int e = e0; e < e0 + per && e < p.El; ++e) crun += sh.mine[e];
  int cstart, dummy_s, cpairs, dummy_t;
  scatter_block_scan2<NT>(crun, 0, sh.wsum, cstart, dummy_s, cpairs, dummy_t);
  for (int e = e0; e < e0 + per && e < p.El; ++e) {
    sh.cbase[e] = cstart;
    cstart += sh.mine[e];
  }

  // rank the chunk's pairs: bit `lane` of bits[w][e] marks that the lane's
  // token holds local expert e
#pragma unroll
  for (int j = 0; j < kPermMaxK; ++j)
    if (le[j] >= 0) atomicOr(&sh.bits[w][le[j]], 1ull << lane);
  __syncthreads();
  if (live) {
    const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
#pragma unroll
    for (int j = 0; j < kPermMaxK; ++j) {
      if (j < p.K) {
        int row = -1;
        const int e = le[j];
        if (e >= 0) {
          int rank = 0;  // among the chunk's pairs of expert e
          for (int i = 0; i < w; ++i) rank += __popcll(sh.bits[i][e]);
          rank += __popcll(sh.bits[w][e] & below);
          row = sh.base[e] + rank;
          // staged in output order: the chunk's pairs of an expert are one
          // contiguous run of rows
          const int li = sh.cbase[e] + rank;
          sh.srow[li] = row;
          sh.spair[li] = t * p.K + j;
        }
        p.pair_row[(size_t)t * p.K + j] = row;
      }
    }
  }
  __syncthreads();
  // coalesced writes: consecutive threads, consecutive rows of a run
  for (int i = threadIdx.x; i < cpairs; i += NT) {
    const int row = sh.srow[i], pr = sh.spair[i];
    p.perm_token[row] = pr / p.K;
    p.perm_pair[row] = pr;
  }
}

}  // namespace moe
