/*
 * moe_debug.h -- test hooks of the fused FP8 MoE library.  Not part of the
 * layer's interface: they expose single building blocks of the device path
 * so that tests can check them bit for bit against the CPU oracle.
 * Same conventions as moe.h (device pointers, asynchronous on `stream`,
 * arguments checked before anything is enqueued).
 */
#ifndef MOE_MI355X_DEBUG_H
#define MOE_MI355X_DEBUG_H

#include <stdint.h>

#include "moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* y[i] = the routing sigmoid of stage (1) (paper Section 3.1.1) applied to
 * x[i], exactly as the routing kernel evaluates it.  n >= 0 elements. */
moe_status_t moe_debug_sigmoid(const float *x, float *y, int64_t n, void *stream);

/* q[i] = the e4m3 code that the re-quantisation of stage (3) (paper Section
 * 3.1.1) assigns to the fp32 value x[i]: round to nearest even, saturating at
 * +-448.  n >= 0 elements. */
moe_status_t moe_debug_e4m3_encode(const float *x, uint8_t *q, int64_t n, void *stream);

/* One FP8 block product of the GEMM stages (paper Section 3.1.1, stage (3)),
 * exactly as the grouped GEMM kernels issue it: for each of n cases,
 * d[c][i][j] = sum over k < 128 of a[c][i][k] * b[c][j][k], with
 * a, b [n, 16, 128] e4m3 (32-byte aligned) and d [n, 16, 16] float. */
moe_status_t moe_debug_mfma_block(const uint8_t *a, const uint8_t *b, float *d, int64_t n,
                                  void *stream);

/* logits [T, E_g] float = the router projection of stage (1) (paper Section
 * 3.1.1) exactly as moe_route_hidden forms it (the fixed fp32 sequence
 * stated there), from hidden [T, H] e4m3, hidden_scale [T, H/128] float and
 * router_weight [E_g, H] float.  Uses the workspace of `s`. */
moe_status_t moe_debug_router_logits(const moe_shape_t *s, const uint8_t *hidden,
                                     const float *hidden_scale, const float *router_weight,
                                     float *logits, void *workspace, size_t ws_bytes,
                                     void *stream);

/* Stage (3)'s GEMM2 and stage (4)'s weighted combine (paper Section 3.1.1)
 * on a re-quantised intermediate supplied by the caller: the routing and
 * permutation of moe_route are computed from router_logits / routing_bias
 * into the workspace, then GEMM2 and the combine run exactly as in
 * moe_fused_fp8 but read
 *  act       [T * top_k, I] e4m3, rows in the permuted order of moe_route
 *            (the first P = expert_offsets[E_l] rows are read)
 *  act_scale [T * top_k, I/128] float
 * instead of the intermediate GEMM1 would write.  out [T, H] bf16 is fully
 * overwritten.  For checking the GEMM2 and combine kernels on an intermediate
 * that does not come from the device. */
moe_status_t moe_debug_combine_from_act(const moe_shape_t *s, const float *router_logits,
                                        const float *routing_bias, const uint8_t *act,
                                        const float *act_scale, const uint8_t *w2,
                                        const float *w2_scale, uint16_t *out, void *workspace,
                                        size_t ws_bytes, void *stream);

/* Device addresses, inside a workspace used by moe_fused_fp8 for shape `s`,
 * of the re-quantised intermediate activation: act [P, I] e4m3 in permuted
 * row order and act_scale [P, I/128] float.  Valid after the call completes,
 * until the workspace is reused. */
moe_status_t moe_debug_act_views(const moe_shape_t *s, void *workspace, uint8_t **act,
                                 float **act_scale);

#ifdef __cplusplus
}
#endif

#endif /* MOE_MI355X_DEBUG_H */
