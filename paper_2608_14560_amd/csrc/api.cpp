// api.cpp -- the C-ABI of the fused FP8 MoE layer: argument validation,
// workspace carving and the launch sequence.  No allocation and no host
// synchronisation happen here: every size that depends on the routing stays
// on the device and the grids are sized from host-known upper bounds.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>

#include "../../include/moe.h"
#include "../../include/moe_debug.h"
#include "moe_device.h"

namespace moe {
hipError_t launch_permute_count(const PermuteParams &p, hipStream_t st);
hipError_t launch_permute_scatter(const PermuteParams &p, hipStream_t st);
hipError_t launch_debug_sigmoid(const float *x, float *y, int64_t n, hipStream_t st);
hipError_t launch_debug_e4m3_encode(const float *x, uint8_t *q, int64_t n, hipStream_t st);
hipError_t launch_debug_mfma_block(const uint8_t *a, const uint8_t *b, float *d, int64_t n,
                                   hipStream_t st);
}  // namespace moe

namespace {

using namespace moe;

constexpr int kStages = 7;
const char *const kStageNames[kStages] = {"route",        "permute_count", "permute_scatter",
                                          "gemm1_swiglu", "requant",       "gemm2",
                                          "combine_finalize"};

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

moe_status_t check_shape(const moe_shape_t *s) {
  if (!s) return MOE_ERR_INVALID_ARG;
  if (s->T < 0 || s->H <= 0 || s->I <= 0 || s->H % 128 || s->I % 128) return MOE_ERR_INVALID_ARG;
  if (s->num_experts < 2 || s->n_group < 1 || s->num_experts % s->n_group) return MOE_ERR_INVALID_ARG;
  const int gsz = s->num_experts / s->n_group;
  if (gsz < 2) return MOE_ERR_INVALID_ARG;
  if (s->topk_group < 1 || s->topk_group > s->n_group) return MOE_ERR_INVALID_ARG;
  if (s->top_k < 1 || s->top_k > s->topk_group * gsz) return MOE_ERR_INVALID_ARG;
  if (s->num_local_experts < 1 || s->local_expert_offset < 0 ||
      (int64_t)s->local_expert_offset + s->num_local_experts > s->num_experts)
    return MOE_ERR_INVALID_ARG;
  if (!std::isfinite(s->routed_scaling_factor)) return MOE_ERR_INVALID_ARG;
  // limits of this library
  if (s->num_experts > 1024 || s->num_local_experts > 1024 || s->n_group > 64 || s->top_k > 16)
    return MOE_ERR_UNSUPPORTED;
  if ((int64_t)s->T * s->top_k >= (int64_t)1 << 31) return MOE_ERR_UNSUPPORTED;
  if (s->H > 65536 || s->I > 65536) return MOE_ERR_UNSUPPORTED;  // staged scales fit LDS
  return MOE_OK;
}

// Host-side plan: tile shape, split factors, grid bounds and the workspace map.
struct Plan {
  int BM, S1, S2, NB1, NB2, nchunks, max_tiles;
  bool narrow1;  // GEMM1 split over 32- (or 16-) column groups (small batches)
  bool gu1;      // ... and over gate and up rows (the fewest rows per expert)
  bool tile;     // large-tile kernels (BM >= 64)
  bool fused_combine;  // GEMM2 with the combine in its epilogue (T <= 16)
  bool perm_in_gemm1;  // the narrow GEMM1 builds the permutation itself (T <= 16)
  int ks1;             // narrow GEMM1: K ranges per item, each on its own waves
  int64_t P_max;
  size_t off_ids, off_w, off_offsets, off_perm_token, off_perm_pair, off_pair_row, off_chunk_counts,
      off_tile_base, off_tile_tab, off_n_items, off_act, off_act_scale, off_act_scale_k, off_hs_k, off_abuf, off_Y,
      off_Ye, off_partials, total;
};

Plan make_plan(const moe_shape_t *s) {
  Plan p{};
  const int64_t TK = (int64_t)s->T * s->top_k;
  p.P_max = TK > 0 ? TK : 1;
  // expected rows per resident expert under uniform routing picks the M tile
  const double avg = (double)TK / s->num_experts;
  p.BM = avg <= 16 ? 16 : (avg <= 48 ? 32 : (avg <= 96 ? 64 : (avg <= 192 ? 128 : 256)));
  // the eight-wave tiles (128 and 256 rows) address their operands with
  // 32-bit offsets from per-matrix bases: rows x row length of the activation
  // operands and of one expert's weights must stay below 2^32 bytes
  const uint64_t big = std::max<uint64_t>({(uint64_t)p.P_max * (uint64_t)s->H, (uint64_t)p.P_max * (uint64_t)s->I,
                                           2ull * (uint64_t)s->I * (uint64_t)s->H});
  if (p.BM >= 128 && big >= (1ull << 32)) p.BM = 64;
  p.tile = p.BM >= 64;
  // GEMM1 keeps the whole K range in one item: its epilogue (SwiGLU and the
  // 1x128 re-quantisation) needs complete sums, and a K split would add a
  // reduction pass.  GEMM2 could split K (S2 > 1 planes of Y, summed by the
  // combine), but measured at decode the full-K items are faster and the
  // combine then reads one plane.
  p.S1 = 1;
  p.S2 = 1;
  // 16-row tiles: GEMM1 split over column groups, so that a batch with few
  // rows per expert still gives every CU work items (it streams weights)
  p.narrow1 = p.BM == 16;
  // at most ~2 rows per expert (decode): 16-column items with the gate and up
  // rows on separate waves, twice the streaming waves; above that the doubled
  // re-reads of each activation tile cost more than the waves gain (measured)
  p.gu1 = p.narrow1 && avg <= 2.0;
  p.NB1 = p.narrow1 ? s->I / gemm1_narrow_cols(p.gu1) : s->I / 128;
  // GEMM2 column blocks: 128 wide for the small-tile kernel, 256 otherwise
  p.NB2 = p.BM == 16 ? s->H / 128 : (s->H + 255) / 256;
  // at most 16 tokens: one 16-row tile per expert, and GEMM2 workgroups that
  // own output columns of every token sum the experts themselves
  p.fused_combine = p.BM == 16 && s->T <= combine_max_tokens() && combine_fits((int)p.P_max, s->I);
  // at most 16 tokens with gate/up-split GEMM1 items: the GEMM1 workgroups
  // rebuild the permutation from the routing ids (at most 256 pairs) and the
  // permutation launch is skipped
  p.perm_in_gemm1 = p.fused_combine && p.gu1 && TK <= 256 && s->T <= 16;
  // 32-column items (more than 2 rows per expert): each item's K range in two
  // halves on separate waves (twice the waves streaming; mid GEMM1 188 -> 172
  // us); the two-wave gate/up items measured no better with it (decode)
  p.ks1 = p.gu1 ? 1 : 2;
  p.nchunks = (int)((s->T + kChunkTokens - 1) / kChunkTokens);
  if (p.nchunks < 1) p.nchunks = 1;
  const int64_t touched = TK < s->num_local_experts ? TK : s->num_local_experts;
  p.max_tiles = (int)((p.P_max + p.BM - 1) / p.BM + touched);

  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  p.off_ids = take(sizeof(int32_t) * p.P_max);
  p.off_w = take(sizeof(float) * p.P_max);
  p.off_offsets = take(sizeof(int32_t) * (s->num_local_experts + 1));
  p.off_perm_token = take(sizeof(int32_t) * p.P_max);
  p.off_perm_pair = take(sizeof(int32_t) * p.P_max);
  p.off_pair_row = take(sizeof(int32_t) * p.P_max);
  p.off_chunk_counts = take(sizeof(int32_t) * (size_t)p.nchunks * s->num_local_experts);
  p.off_tile_base = take(sizeof(int32_t) * (s->num_local_experts + 1));
  p.off_tile_tab = take(4 * sizeof(int32_t) * (size_t)p.max_tiles);
  p.off_n_items = take(sizeof(int32_t) * 2);
  p.off_act = take((size_t)p.P_max * s->I);
  p.off_act_scale = take(sizeof(float) * (size_t)p.P_max * (s->I / 128));
  p.off_abuf = take(p.narrow1 ? sizeof(float) * (size_t)p.P_max * s->I : 0);
  // large tiles: K-block-major activation scales, [I/128, P_max] written by
  // GEMM1 for GEMM2 and [H/128, P_max] gathered from the hidden scales
  p.off_act_scale_k = take(p.tile ? sizeof(float) * (size_t)p.P_max * (s->I / 128) : 0);
  p.off_hs_k = take(p.tile ? sizeof(float) * (size_t)p.P_max * (s->H / 128) : 0);
  // Y: fp16 codes [P_max, H] and their chunk exponents [P_max, H/16].  The
  // router projection's block sums [T, H/128, E_g] live in the same region:
  // the routing kernel consumes them before GEMM2 writes Y
  const size_t y_bytes = align_up(sizeof(uint16_t) * (size_t)p.P_max * s->H);
  const size_t ye_bytes = (size_t)p.P_max * (s->H / kYChunk);
  const size_t part_bytes = sizeof(float) * (size_t)(s->T > 0 ? s->T : 1) * (s->H / 128) * s->num_experts;
  p.off_Y = take(y_bytes + ye_bytes > part_bytes ? y_bytes + ye_bytes : part_bytes);
  p.off_Ye = p.off_Y + y_bytes;
  p.off_partials = p.off_Y;
  p.total = o;
  return p;
}

template <class T>
T *at(void *ws, size_t off) {
  return reinterpret_cast<T *>(static_cast<uint8_t *>(ws) + off);
}

int round8(int64_t x) { return (int)((x + 7) / 8 * 8); }

struct Ptrs {
  int32_t *ids;
  float *w;
  int32_t *offsets, *perm_token, *pair_row;
};

Ptrs route_ptrs(const Plan &pl, void *ws, const moe_route_out_t *ro) {
  Ptrs r;
  r.ids = (ro && ro->topk_ids) ? ro->topk_ids : at<int32_t>(ws, pl.off_ids);
  r.w = (ro && ro->topk_weights) ? ro->topk_weights : at<float>(ws, pl.off_w);
  r.offsets = (ro && ro->expert_offsets) ? ro->expert_offsets : at<int32_t>(ws, pl.off_offsets);
  r.perm_token = (ro && ro->perm_token) ? ro->perm_token : at<int32_t>(ws, pl.off_perm_token);
  r.pair_row = (ro && ro->pair_row) ? ro->pair_row : at<int32_t>(ws, pl.off_pair_row);
  return r;
}

moe_status_t check_route_out(const moe_route_out_t *ro) {
  if (!ro) return MOE_OK;
  const void *ps[] = {ro->topk_ids, ro->topk_weights, ro->expert_offsets, ro->perm_token, ro->pair_row};
  for (const void *q : ps)
    if (!q || !aligned(q, 16)) return MOE_ERR_INVALID_ARG;
  return MOE_OK;
}

#define MOE_TRY_HIP(expr)                    \
  do {                                       \
    if ((expr) != hipSuccess) return MOE_ERR_HIP; \
  } while (0)

// Router input: either the logits, or the hidden rows with the router weight
// (the projection then runs first and the routing kernel forms the logits
// from its block sums).
struct RouterIn {
  const float *logits;
  const uint8_t *hidden;
  const float *hidden_scale;
  const float *weight;
};

RouteParams route_params(const moe_shape_t *s, const Plan &pl, const RouterIn &in,
                         const float *bias, const Ptrs &r, void *ws) {
  RouteParams rp{in.logits, bias, r.ids, r.w, s->T, s->num_experts, s->n_group, s->topk_group,
                 s->top_k, s->routed_scaling_factor};
  if (in.weight) {
    rp.partials = at<float>(ws, pl.off_partials);
    rp.pscale = in.hidden_scale;
    rp.KB = s->H / 128;
  }
  return rp;
}

hipError_t enqueue_projection(const moe_shape_t *s, const Plan &pl, const RouterIn &in, void *ws,
                              hipStream_t st) {
  if (!in.weight) return hipSuccess;
  RouterParams q{in.hidden, in.weight, at<float>(ws, pl.off_partials), s->T, s->H,
                 s->num_experts};
  return launch_router_partials(q, st);
}

PermuteParams permute_params(const moe_shape_t *s, const Plan &pl, const Ptrs &r, void *ws) {
  PermuteParams pp{};
  pp.topk_ids = r.ids;
  pp.chunk_counts = at<int32_t>(ws, pl.off_chunk_counts);
  pp.expert_offsets = r.offsets;
  pp.perm_token = r.perm_token;
  pp.perm_pair = at<int32_t>(ws, pl.off_perm_pair);
  pp.pair_row = r.pair_row;
  pp.tile_base = at<int32_t>(ws, pl.off_tile_base);
  pp.tile_tab = at<int32_t>(ws, pl.off_tile_tab);
  pp.n_items = at<int32_t>(ws, pl.off_n_items);
  pp.T = s->T;
  pp.K = s->top_k;
  pp.El = s->num_local_experts;
  pp.offset = s->local_expert_offset;
  pp.nchunks = pl.nchunks;
  pp.BM = pl.BM;
  pp.items_per_tile1 = pl.NB1 * pl.S1;
  pp.items_per_tile2 = pl.NB2 * pl.S2;
  return pp;
}

// Stages (1) and (2); with skip_permute the permutation is left to the
// narrow GEMM1 (its stage events are still recorded, around nothing).
moe_status_t enqueue_route(const moe_shape_t *s, const Plan &pl, const RouterIn &in,
                           const float *bias, const Ptrs &r, void *ws, hipStream_t st,
                           void *const *ev, int &stage, bool skip_permute = false) {
  auto mark = [&]() {
    if (ev) (void)hipEventRecord(static_cast<hipEvent_t>(ev[stage]), st);
    ++stage;
  };
  const RouteParams rp = route_params(s, pl, in, bias, r, ws);
  const PermuteParams pp = permute_params(s, pl, r, ws);
  mark();
  MOE_TRY_HIP(enqueue_projection(s, pl, in, ws, st));
  MOE_TRY_HIP(launch_route(rp, st));
  mark();
  if (!skip_permute) MOE_TRY_HIP(launch_permute_count(pp, st));
  mark();
  if (!skip_permute) MOE_TRY_HIP(launch_permute_scatter(pp, st));
  return MOE_OK;
}

// Stage (3)'s GEMM2 on the permuted intermediate act [P, I] / act_scale
// [P, I/128] and stage (4)'s weighted combine into `out`, after the routing
// and permutation have been enqueued into `ws`.
moe_status_t enqueue_gemm2_combine(const moe_shape_t *s, const Plan &pl, const Ptrs &r,
                                   const uint8_t *act, const float *act_scale,
                                   const float *act_scale_k, const uint8_t *w2,
                                   const float *w2_scale, uint16_t *out, void *ws, hipStream_t st,
                                   void *const *ev, int &stage) {
  auto mark = [&]() {
    if (ev) (void)hipEventRecord(static_cast<hipEvent_t>(ev[stage]), st);
    ++stage;
  };
  GemmParams g2{};
  g2.expert_offsets = r.offsets;
  g2.tile_base = at<int32_t>(ws, pl.off_tile_base);
  g2.tile_tab = at<int32_t>(ws, pl.off_tile_tab);
  g2.perm_token = r.perm_token;
  g2.Y = at<uint16_t>(ws, pl.off_Y);
  g2.Ye = at<int8_t>(ws, pl.off_Ye);
  g2.I = s->I;
  g2.H = s->H;
  g2.P_max = (int)pl.P_max;
  g2.El = s->num_local_experts;
  g2.A = act;
  g2.A_scale = act_scale;
  // the large-tile kernel reads the K-block-major copy when GEMM1 wrote one
  g2.sa_tile = act_scale_k ? act_scale_k : act_scale;
  g2.sa_row = act_scale_k ? 1 : s->I / 128;
  g2.sa_kb = act_scale_k ? (int)pl.P_max : 1;
  g2.B = w2;
  g2.B_scale = w2_scale;
  g2.n_items = at<int32_t>(ws, pl.off_n_items) + 1;
  g2.K = s->I;
  g2.KB = s->I / 128;
  g2.N_total = s->H;
  g2.NB = pl.NB2;
  g2.S = pl.S2;
  mark();
  if (pl.fused_combine) {
    const int KB = s->I / 128;
    CombineParams c{at<int32_t>(ws, pl.off_perm_pair), r.w, out, s->T, s->top_k,
                    KB % 4 == 0 ? 4 : (KB % 2 == 0 ? 2 : 1)};
    MOE_TRY_HIP(launch_gemm2_combine(g2, c, st));
    mark();  // the combine stage enqueues nothing of its own
    return MOE_OK;
  }
  const int grid2 = round8((int64_t)pl.max_tiles * pl.NB2 * pl.S2);
  MOE_TRY_HIP(pl.tile ? launch_gemm_tile(g2, false, pl.BM, grid2, st)
                      : launch_gemm2(g2, pl.BM, grid2, st));

  // weighted combine in slot order, one bf16 rounding per element
  // a chunk of 16 columns per thread where a token has at least 4 resident
  // slots on average, half a chunk otherwise (more threads for the latency of
  // the two dependent round trips when most slots are absent)
  const int cw = (int64_t)s->top_k * s->num_local_experts >= 4 * (int64_t)s->num_experts ? 16 : 8;
  FinalizeParams f{g2.Y, g2.Ye, r.pair_row, r.w, out, s->T, s->H, s->top_k, cw};
  mark();
  MOE_TRY_HIP(launch_finalize(f, st));
  return MOE_OK;
}

moe_status_t fused_impl(const moe_shape_t *s, const uint8_t *hidden, const float *hidden_scale,
                        const float *logits, const float *router_weight, const float *bias,
                        const uint8_t *w13, const float *w13_scale, const uint8_t *w2,
                        const float *w2_scale, uint16_t *out, const moe_route_out_t *ro, void *ws,
                        size_t ws_bytes, void *stream, void *const *ev, int n_ev) {
  moe_status_t rc = check_shape(s);
  if (rc != MOE_OK) return rc;
  if (ev && n_ev != kStages + 1) return MOE_ERR_INVALID_ARG;
  if (s->T == 0) return MOE_OK;
  const float *router_in = logits ? logits : router_weight;
  const void *ptrs[] = {hidden, hidden_scale, router_in, bias, w13, w13_scale, w2, w2_scale, out};
  for (const void *q : ptrs)
    if (!q || !aligned(q, 16)) return MOE_ERR_INVALID_ARG;
  if ((rc = check_route_out(ro)) != MOE_OK) return rc;
  const Plan pl = make_plan(s);
  if (!ws || !aligned(ws, kAlign)) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < pl.total) return MOE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t st = static_cast<hipStream_t>(stream);

  const Ptrs r = route_ptrs(pl, ws, ro);
  int stage = 0;
  const RouterIn rin{logits, hidden, hidden_scale, router_weight};
  if ((rc = enqueue_route(s, pl, rin, bias, r, ws, st, ev, stage, pl.perm_in_gemm1)) != MOE_OK)
    return rc;
  auto mark = [&]() {
    if (ev) (void)hipEventRecord(static_cast<hipEvent_t>(ev[stage]), st);
    ++stage;
  };

  GemmParams g{};
  g.expert_offsets = r.offsets;
  g.tile_base = at<int32_t>(ws, pl.off_tile_base);
  g.tile_tab = at<int32_t>(ws, pl.off_tile_tab);
  g.perm_token = r.perm_token;
  g.abuf = at<float>(ws, pl.off_abuf);
  g.act = at<uint8_t>(ws, pl.off_act);
  g.act_scale = at<float>(ws, pl.off_act_scale);
  g.I = s->I;
  g.H = s->H;
  g.P_max = (int)pl.P_max;
  g.El = s->num_local_experts;

  // large tiles: the gathered hidden scales, K-block-major (part of the
  // permutation stage)
  if (pl.tile)
    MOE_TRY_HIP(launch_gather_scales(r.offsets, s->num_local_experts, r.perm_token, hidden_scale,
                                     at<float>(ws, pl.off_hs_k), s->H / 128, (int)pl.P_max, st));

  // GEMM1: hidden rows (gathered) x W13, SwiGLU + FP8 re-quantisation
  GemmParams g1 = g;
  g1.A = hidden;
  g1.A_scale = hidden_scale;
  g1.sa_tile = at<float>(ws, pl.off_hs_k);
  g1.sa_row = 1;
  g1.sa_kb = (int)pl.P_max;
  g1.act_scale_k = pl.tile ? at<float>(ws, pl.off_act_scale_k) : nullptr;
  g1.B = w13;
  g1.B_scale = w13_scale;
  g1.n_items = at<int32_t>(ws, pl.off_n_items);
  g1.K = s->H;
  g1.KB = s->H / 128;
  g1.N_total = 2 * s->I;
  g1.NB = pl.NB1;
  g1.S = pl.S1;
  mark();
  const int grid1 = round8((int64_t)pl.max_tiles * pl.NB1 * pl.S1);
  if (pl.perm_in_gemm1) g1.perm = permute_params(s, pl, r, ws);
  if (pl.narrow1)
    MOE_TRY_HIP(launch_gemm1_narrow(g1, grid1, pl.gu1, pl.perm_in_gemm1, pl.ks1, st));
  else if (pl.tile)
    MOE_TRY_HIP(launch_gemm_tile(g1, true, pl.BM, grid1, st));
  else
    MOE_TRY_HIP(launch_gemm1(g1, pl.BM, grid1, st));
  // the column-split GEMM1 leaves its re-quantisation to a launch of its own
  mark();
  if (pl.narrow1) MOE_TRY_HIP(launch_requant(g1, (int)pl.P_max, st));

  // GEMM2 and the weighted combine on the intermediate GEMM1 just wrote
  if ((rc = enqueue_gemm2_combine(s, pl, r, g.act, g.act_scale, g1.act_scale_k, w2, w2_scale, out,
                                  ws, st, ev, stage)) != MOE_OK)
    return rc;
  if (ev) (void)hipEventRecord(static_cast<hipEvent_t>(ev[stage]), st);
  return MOE_OK;
}

// ---- the allocation-free entry point's workspace: a file-scope device array
// (each GPU the library runs on holds its own copy until the process ends).
// Host code never uses the array's name as an address: its device address is
// taken once per device with hipGetSymbolAddress, with that device current.
constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

}  // namespace

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

moe_status_t scratch_of_current_device(void **ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MOE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MOE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return MOE_OK;
}

}  // namespace

extern "C" {

size_t moe_workspace_size(const moe_shape_t *s) {
  if (check_shape(s) != MOE_OK) return 0;
  return make_plan(s).total;
}

moe_status_t moe_route(const moe_shape_t *s, const float *router_logits,
                       const float *routing_bias, const moe_route_out_t *out, void *workspace,
                       size_t ws_bytes, void *stream) {
  moe_status_t rc = check_shape(s);
  if (rc != MOE_OK) return rc;
  if (!out) return MOE_ERR_INVALID_ARG;
  if (s->T == 0) {
    // empty batch: only expert_offsets (all zero) is written; the other
    // arrays have zero size and may be null
    if (!out->expert_offsets || !aligned(out->expert_offsets, 16) || !out->perm_token)
      return MOE_ERR_INVALID_ARG;
  } else {
    if (!router_logits || !routing_bias || !aligned(router_logits, 16) ||
        !aligned(routing_bias, 16))
      return MOE_ERR_INVALID_ARG;
    if ((rc = check_route_out(out)) != MOE_OK) return rc;
  }
  const Plan pl = make_plan(s);
  if (!workspace || !aligned(workspace, kAlign)) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < pl.total) return MOE_ERR_WORKSPACE_TOO_SMALL;
  const Ptrs r = route_ptrs(pl, workspace, out);
  int stage = 0;
  const RouterIn rin{router_logits, nullptr, nullptr, nullptr};
  return enqueue_route(s, pl, rin, routing_bias, r, workspace, static_cast<hipStream_t>(stream),
                       nullptr, stage);
}

moe_status_t moe_route_hidden(const moe_shape_t *s, const uint8_t *hidden,
                              const float *hidden_scale, const float *router_weight,
                              const float *routing_bias, const moe_route_out_t *out,
                              void *workspace, size_t ws_bytes, void *stream) {
  moe_status_t rc = check_shape(s);
  if (rc != MOE_OK) return rc;
  if (!out) return MOE_ERR_INVALID_ARG;
  if (s->T == 0) {
    if (!out->expert_offsets || !aligned(out->expert_offsets, 16) || !out->perm_token)
      return MOE_ERR_INVALID_ARG;
  } else {
    const void *ptrs[] = {hidden, hidden_scale, router_weight, routing_bias};
    for (const void *q : ptrs)
      if (!q || !aligned(q, 16)) return MOE_ERR_INVALID_ARG;
    if ((rc = check_route_out(out)) != MOE_OK) return rc;
  }
  const Plan pl = make_plan(s);
  if (!workspace || !aligned(workspace, kAlign)) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < pl.total) return MOE_ERR_WORKSPACE_TOO_SMALL;
  const Ptrs r = route_ptrs(pl, workspace, out);
  int stage = 0;
  const RouterIn rin{nullptr, hidden, hidden_scale, router_weight};
  return enqueue_route(s, pl, rin, routing_bias, r, workspace, static_cast<hipStream_t>(stream),
                       nullptr, stage);
}

moe_status_t moe_fused_fp8(const moe_shape_t *s, const uint8_t *hidden, const float *hidden_scale,
                           const float *router_logits, const float *routing_bias,
                           const uint8_t *w13, const float *w13_scale, const uint8_t *w2,
                           const float *w2_scale, uint16_t *out, const moe_route_out_t *route_out,
                           void *workspace, size_t ws_bytes, void *stream) {
  return fused_impl(s, hidden, hidden_scale, router_logits, nullptr, routing_bias, w13, w13_scale,
                    w2, w2_scale, out, route_out, workspace, ws_bytes, stream, nullptr, 0);
}

moe_status_t moe_fused_fp8_noalloc(const moe_shape_t *s, const uint8_t *hidden,
                                   const float *hidden_scale, const float *router_logits,
                                   const float *routing_bias, const uint8_t *w13,
                                   const float *w13_scale, const uint8_t *w2,
                                   const float *w2_scale, uint16_t *out,
                                   const moe_route_out_t *route_out, void *stream) {
  moe_status_t rc = check_shape(s);
  if (rc != MOE_OK) return rc;
  if (make_plan(s).total > kScratchBytes) return MOE_ERR_UNSUPPORTED;
  void *ws = nullptr;
  if ((rc = scratch_of_current_device(&ws)) != MOE_OK) return rc;
  return fused_impl(s, hidden, hidden_scale, router_logits, nullptr, routing_bias, w13, w13_scale,
                    w2, w2_scale, out, route_out, ws, kScratchBytes, stream, nullptr, 0);
}

moe_status_t moe_fused_fp8_router(const moe_shape_t *s, const uint8_t *hidden,
                                  const float *hidden_scale, const float *router_weight,
                                  const float *routing_bias, const uint8_t *w13,
                                  const float *w13_scale, const uint8_t *w2, const float *w2_scale,
                                  uint16_t *out, const moe_route_out_t *route_out, void *workspace,
                                  size_t ws_bytes, void *stream) {
  return fused_impl(s, hidden, hidden_scale, nullptr, router_weight, routing_bias, w13, w13_scale,
                    w2, w2_scale, out, route_out, workspace, ws_bytes, stream, nullptr, 0);
}

moe_status_t moe_fused_fp8_staged(const moe_shape_t *s, const uint8_t *hidden,
                                  const float *hidden_scale, const float *router_logits,
                                  const float *routing_bias, const uint8_t *w13,
                                  const float *w13_scale, const uint8_t *w2, const float *w2_scale,
                                  uint16_t *out, const moe_route_out_t *route_out, void *workspace,
                                  size_t ws_bytes, void *stream, void *const *stage_events,
                                  int n_events) {
  if (!stage_events) return MOE_ERR_INVALID_ARG;
  for (int i = 0; i < n_events; ++i)
    if (!stage_events[i]) return MOE_ERR_INVALID_ARG;
  return fused_impl(s, hidden, hidden_scale, router_logits, nullptr, routing_bias, w13, w13_scale,
                    w2, w2_scale, out, route_out, workspace, ws_bytes, stream, stage_events,
                    n_events);
}

int moe_num_stages(void) { return kStages; }

const char *moe_stage_name(int i) { return (i >= 0 && i < kStages) ? kStageNames[i] : nullptr; }

const char *moe_status_string(moe_status_t st) {
  switch (st) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported shape";
    case MOE_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case MOE_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

moe_status_t moe_debug_sigmoid(const float *x, float *y, int64_t n, void *stream) {
  if (n < 0 || (n > 0 && (!x || !y))) return MOE_ERR_INVALID_ARG;
  return launch_debug_sigmoid(x, y, n, static_cast<hipStream_t>(stream)) == hipSuccess
             ? MOE_OK
             : MOE_ERR_HIP;
}

moe_status_t moe_debug_e4m3_encode(const float *x, uint8_t *q, int64_t n, void *stream) {
  if (n < 0 || (n > 0 && (!x || !q))) return MOE_ERR_INVALID_ARG;
  return launch_debug_e4m3_encode(x, q, n, static_cast<hipStream_t>(stream)) == hipSuccess
             ? MOE_OK
             : MOE_ERR_HIP;
}

moe_status_t moe_debug_mfma_block(const uint8_t *a, const uint8_t *b, float *d, int64_t n,
                                  void *stream) {
  if (n < 0 || (n > 0 && (!a || !b || !d))) return MOE_ERR_INVALID_ARG;
  if (!aligned(a, 32) || !aligned(b, 32) || !aligned(d, 16)) return MOE_ERR_INVALID_ARG;
  return launch_debug_mfma_block(a, b, d, n, static_cast<hipStream_t>(stream)) == hipSuccess
             ? MOE_OK
             : MOE_ERR_HIP;
}

moe_status_t moe_debug_router_logits(const moe_shape_t *s, const uint8_t *hidden,
                                     const float *hidden_scale, const float *router_weight,
                                     float *logits, void *workspace, size_t ws_bytes,
                                     void *stream) {
  if (check_shape(s) != MOE_OK) return MOE_ERR_INVALID_ARG;
  if (s->T == 0) return MOE_OK;
  const void *ptrs[] = {hidden, hidden_scale, router_weight, logits};
  for (const void *q : ptrs)
    if (!q || !aligned(q, 16)) return MOE_ERR_INVALID_ARG;
  const Plan pl = make_plan(s);
  if (!workspace || !aligned(workspace, kAlign)) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < pl.total) return MOE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const RouterIn rin{nullptr, hidden, hidden_scale, router_weight};
  const Ptrs r{};
  const RouteParams rp = route_params(s, pl, rin, nullptr, r, workspace);
  if (enqueue_projection(s, pl, rin, workspace, st) != hipSuccess) return MOE_ERR_HIP;
  return launch_router_logits(rp, logits, st) == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

moe_status_t moe_debug_combine_from_act(const moe_shape_t *s, const float *router_logits,
                                        const float *routing_bias, const uint8_t *act,
                                        const float *act_scale, const uint8_t *w2,
                                        const float *w2_scale, uint16_t *out, void *workspace,
                                        size_t ws_bytes, void *stream) {
  moe_status_t rc = check_shape(s);
  if (rc != MOE_OK) return rc;
  if (s->T == 0) return MOE_OK;
  const void *ptrs[] = {router_logits, routing_bias, act, act_scale, w2, w2_scale, out};
  for (const void *q : ptrs)
    if (!q || !aligned(q, 16)) return MOE_ERR_INVALID_ARG;
  const Plan pl = make_plan(s);
  if (!workspace || !aligned(workspace, kAlign)) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < pl.total) return MOE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const Ptrs r = route_ptrs(pl, workspace, nullptr);
  int stage = 0;
  const RouterIn rin{router_logits, nullptr, nullptr, nullptr};
  if ((rc = enqueue_route(s, pl, rin, routing_bias, r, workspace, st, nullptr, stage)) != MOE_OK)
    return rc;
  return enqueue_gemm2_combine(s, pl, r, act, act_scale, nullptr, w2, w2_scale, out, workspace, st,
                               nullptr, stage);
}

moe_status_t moe_debug_act_views(const moe_shape_t *s, void *workspace, uint8_t **act,
                                 float **act_scale) {
  if (check_shape(s) != MOE_OK || !workspace || !act || !act_scale) return MOE_ERR_INVALID_ARG;
  const Plan pl = make_plan(s);
  *act = at<uint8_t>(workspace, pl.off_act);
  *act_scale = at<float>(workspace, pl.off_act_scale);
  return MOE_OK;
}

}  // extern "C"
