/*
 * moe.h -- C-ABI of the MI355X (gfx950) fused block-scaled FP8
 * mixture-of-experts layer.
 *
 * The operation is the Fused MoE block of the paper (Section 3.1.1), per
 * token: (1) routing scores = sigmoid(router logits), group-limited top-k
 * expert selection; (2) the token rows of every resident expert gathered into
 * a contiguous FP8 layout with 128-element fp32 block scales; (3) the gated
 * MLP -- FP8 block GEMM1 [rows,H] -> [rows,2I], SwiGLU, re-quantisation to
 * FP8 with 1x128 fp32 scales, FP8 block GEMM2 [rows,I] -> [rows,H]; (4) the
 * expert outputs scattered back to their tokens, weighted by the routing
 * scores, written as bf16.
 *
 * Conventions for every entry point:
 *  - Tensor arguments are DEVICE pointers (the current HIP device), row-major,
 *    16-byte aligned; the caller owns every buffer, including the workspace.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *    asynchronously; no entry point synchronises the host or allocates
 *    device memory.
 *  - Arguments are validated before anything is enqueued; a failed check
 *    returns an error code and enqueues nothing.  Launch failures return
 *    MOE_ERR_HIP.  Faults inside kernels surface at the caller's next
 *    synchronisation.  No C++ exception crosses this interface.
 *  - Floating-point formats: e4m3 = OCP FP8 E4M3FN (max 448), one byte per
 *    value; bf16 results are returned as their 16-bit patterns.
 *  - Block scales: activation scale [t, h/128] multiplies hidden[t, h];
 *    weight scale [e, n/128, h/128] multiplies w[e, n, h].
 */
#ifndef MOE_MI355X_H
#define MOE_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = 1,         /* bad shape, null or misaligned pointer */
  MOE_ERR_UNSUPPORTED = 2,         /* valid but outside the library's limits */
  MOE_ERR_WORKSPACE_TOO_SMALL = 3, /* ws_bytes < moe_workspace_size()        */
  MOE_ERR_HIP = 4                  /* a HIP runtime call or launch failed    */
} moe_status_t;

/* Problem shape.  Router of E_g experts in n_group equal groups; the
 * experts [local_expert_offset, local_expert_offset + E_l) have their weights
 * on this GPU; a (token, expert) pair whose expert is elsewhere contributes
 * zero to this GPU's output but still counts in the weight normalisation.
 * Limits of this library: H, I multiples of 128; 2 <= E_g/n_group;
 * E_g <= 1024; E_l <= 1024; top_k <= 16; T * top_k < 2^31. */
typedef struct {
  int32_t T;                     /* tokens (0 allowed: no-op)              */
  int32_t H;                     /* hidden size                            */
  int32_t I;                     /* expert intermediate size               */
  int32_t num_experts;           /* E_g, router width                      */
  int32_t num_local_experts;     /* E_l                                    */
  int32_t local_expert_offset;   /* first resident global expert id        */
  int32_t n_group;               /* expert groups of the router            */
  int32_t topk_group;            /* groups kept per token                  */
  int32_t top_k;                 /* experts per token                      */
  float routed_scaling_factor;   /* multiplies the normalised weights      */
} moe_shape_t;

/* Routing and permutation results (all device pointers, caller-owned).
 *  topk_ids      [T, top_k] int32  global expert ids; order: larger key
 *                first (key = score + bias), ties -> lower id
 *  topk_weights  [T, top_k] float  score / (sum of the k selected scores,
 *                summed in that order) * routed_scaling_factor; scores are
 *                the sigmoid without bias
 *  expert_offsets[E_l + 1]  int32  first permuted row of each resident
 *                expert; expert_offsets[E_l] = P, the resident pair count
 *  perm_token    [T * top_k] int32 token of each permuted row (first P
 *                entries written); rows of an expert are in token order
 *  pair_row      [T, top_k] int32  permuted row of pair (t, j), -1 when the
 *                expert of that pair is not resident */
typedef struct {
  int32_t *topk_ids;
  float *topk_weights;
  int32_t *expert_offsets;
  int32_t *perm_token;
  int32_t *pair_row;
} moe_route_out_t;

/* Bytes of device workspace that every entry point below needs for `s`
 * (a worst case: every pair resident).  Returns 0 for an invalid shape.
 * The workspace needs no initialisation and is not read across calls. */
size_t moe_workspace_size(const moe_shape_t *s);

/* Stage (1) and the bookkeeping of stage (2) of Section 3.1.1: routing, the
 * per-expert counts, their exclusive scan and the stable permutation.
 *  router_logits [T, E_g] float, routing_bias [E_g] float (used for
 *  selection only).  Every field of `out` must be non-null, except that for
 *  T = 0 the zero-size arrays (logits, topk_ids, topk_weights, pair_row)
 *  may be null; expert_offsets is then written as all zeros.
 * Bitwise deterministic. */
moe_status_t moe_route(const moe_shape_t *s, const float *router_logits,
                       const float *routing_bias, const moe_route_out_t *out,
                       void *workspace, size_t ws_bytes, void *stream);

/* moe_route with the router projection of stage (1) (Section 3.1.1: the
 * routing scores start from a linear projection of the hidden state) done on
 * the device instead of taking logits:
 *  hidden        [T, H] e4m3      hidden_scale [T, H/128] float
 *  router_weight [E_g, H] float   routing_bias [E_g] float
 * logit[t, e] follows one fixed fp32 sequence (the expert choice depends on
 * it bit for bit): for each 128-element block kb, p = fused multiply-add
 * chain over the block's elements in ascending order, starting from 0, of
 * decode(hidden[t, h]) * router_weight[e, h]; then logit = fused multiply-add
 * chain over the blocks in ascending order, starting from 0, of
 * hidden_scale[t, kb] * p.  The logits are not written anywhere.  Outputs,
 * T = 0 handling and determinism as moe_route; the workspace is the same
 * (moe_workspace_size). */
moe_status_t moe_route_hidden(const moe_shape_t *s, const uint8_t *hidden,
                              const float *hidden_scale, const float *router_weight,
                              const float *routing_bias, const moe_route_out_t *out,
                              void *workspace, size_t ws_bytes, void *stream);

/* The whole layer, stages (1)-(4) of Section 3.1.1.
 *  hidden        [T, H] e4m3      hidden_scale [T, H/128] float
 *  router_logits [T, E_g] float   routing_bias [E_g] float
 *  w13           [E_l, 2I, H] e4m3 -- rows [0, I) gate, [I, 2I) up
 *  w13_scale     [E_l, 2I/128, H/128] float
 *  w2            [E_l, H, I] e4m3  w2_scale [E_l, H/128, I/128] float
 *  out           [T, H] bf16, fully overwritten; a token with no resident
 *                expert gets +0
 *  route_out     nullable; when given, the routing results are also written
 *                there (same meaning as for moe_route)
 * The intermediate activation is re-quantised per 1x128 block with
 * scale = amax / 448 (round to nearest even, saturating; an all-zero block
 * gets scale 1).  Accumulation is fp32; each output element is rounded to bf16
 * once.  Routing results are bitwise deterministic; `out` is deterministic
 * (fixed summation orders, no floating-point atomics). */
moe_status_t moe_fused_fp8(const moe_shape_t *s, const uint8_t *hidden,
                           const float *hidden_scale,
                           const float *router_logits,
                           const float *routing_bias, const uint8_t *w13,
                           const float *w13_scale, const uint8_t *w2,
                           const float *w2_scale, uint16_t *out,
                           const moe_route_out_t *route_out, void *workspace,
                           size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * moe_fused_fp8 without a workspace argument.  The workspace is a 32 MiB
 * device array inside the library, one per GPU, held until the process ends
 * (its address is looked up on the first call on each device).  Arguments,
 * outputs and determinism as moe_fused_fp8; shapes whose workspace
 * (moe_workspace_size) exceeds 32 MiB return MOE_ERR_UNSUPPORTED before
 * anything is enqueued (DeepSeek-V3 shapes: up to about 100 tokens).  Every
 * call on one GPU uses that GPU's array: calls that overlap in time on one
 * GPU (other streams, other threads) race and must be serialised by the
 * caller.  The array needs no initialisation; nothing is read across calls.
 * No hipMalloc, hipFree or allocating library routine is called. */
moe_status_t moe_fused_fp8_noalloc(const moe_shape_t *s, const uint8_t *hidden,
                                   const float *hidden_scale,
                                   const float *router_logits,
                                   const float *routing_bias,
                                   const uint8_t *w13, const float *w13_scale,
                                   const uint8_t *w2, const float *w2_scale,
                                   uint16_t *out,
                                   const moe_route_out_t *route_out,
                                   void *stream);

/* moe_fused_fp8 with the router projection of stage (1) on the device:
 * router_weight [E_g, H] float replaces router_logits; the logits are those
 * defined under moe_route_hidden.  Everything else as moe_fused_fp8 (the
 * projection runs inside the "route" stage). */
moe_status_t moe_fused_fp8_router(const moe_shape_t *s, const uint8_t *hidden,
                                  const float *hidden_scale,
                                  const float *router_weight,
                                  const float *routing_bias, const uint8_t *w13,
                                  const float *w13_scale, const uint8_t *w2,
                                  const float *w2_scale, uint16_t *out,
                                  const moe_route_out_t *route_out, void *workspace,
                                  size_t ws_bytes, void *stream);

/* Same as moe_fused_fp8; additionally records `stage_events[i]` (hipEvent_t
 * handles created by the caller) on `stream` before stage i and
 * stage_events[moe_num_stages()] after the last one, so a caller can time
 * each kernel with hipEventElapsedTime.  n_events must be
 * moe_num_stages() + 1. */
moe_status_t moe_fused_fp8_staged(const moe_shape_t *s, const uint8_t *hidden,
                                  const float *hidden_scale,
                                  const float *router_logits,
                                  const float *routing_bias,
                                  const uint8_t *w13, const float *w13_scale,
                                  const uint8_t *w2, const float *w2_scale,
                                  uint16_t *out,
                                  const moe_route_out_t *route_out,
                                  void *workspace, size_t ws_bytes,
                                  void *stream, void *const *stage_events,
                                  int n_events);

/* Number and names of the kernels moe_fused_fp8 enqueues, in order. */
int moe_num_stages(void);
const char *moe_stage_name(int i);

const char *moe_status_string(moe_status_t st);

#ifdef __cplusplus
}
#endif

#endif /* MOE_MI355X_H */
