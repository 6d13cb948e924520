/*
 * dsa_attention.h -- C-ABI of the MI355X (gfx950) DSA sparse attention: the
 * paged KV-cache batched decoding operator of the paper's Section 3.1.2.
 *
 * For each query token t and head h: gather the token's TopK cached entries
 * through its sparse index list, form the base-2 logits
 *   s_j = (q_nope[t,h] . Kc_j + q_pe[t,h] . Kp_j) * sm_scale * log2(e),
 * and return out[t,h] = sum_j 2^(s_j - lse) * Kc_j (512 wide, bf16) with
 * lse[t,h] = log2(sum_j 2^s_j) (fp32).  A token with no valid index gets
 * out = 0 and lse = -inf.
 *
 * Same conventions as moe.h: device pointers, row-major, 16-byte aligned;
 * the caller owns every buffer including the workspace; asynchronous on
 * `stream`; arguments are checked before anything is enqueued; nothing
 * synchronises the host or allocates.  Status codes are moe_status_t.
 */
#ifndef DSA_ATTENTION_MI355X_H
#define DSA_ATTENTION_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include "moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Problem shape.  Limits of this library: num_heads a positive multiple of 16;
 * 1 <= topk <= 65536; num_rows >= 1; sm_scale finite. */
typedef struct {
  int32_t T;          /* query tokens                                      */
  int32_t num_heads;  /* query heads (16 per GPU in the paper's workloads)  */
  int32_t topk;       /* sparse entries per token (2048)                    */
  int32_t num_rows;   /* cache rows = pages * tokens per page               */
  float sm_scale;     /* logit scale before the base-2 conversion           */
} dsa_attn_shape_t;

/* Bytes of device workspace dsa_sparse_attention needs for `s` (the split
 * outputs); 0 for an invalid shape. */
size_t dsa_attention_workspace_size(const dsa_attn_shape_t *s);

/* DSA sparse attention (Section 3.1.2).
 *  q_nope   [T, H, 512] bf16      q_pe [T, H, 64] bf16
 *  ckv      [num_rows, 512] bf16  kpe  [num_rows, 64] bf16 (a paged cache
 *           addressed by physical row page * page_size + slot)
 *  indices  [T, topk] int32 cache rows; entries outside [0, num_rows) (-1
 *           for padding) are absent
 *  out      [T, H, 512] bf16      lse  [T, H] float (base 2)
 * Arithmetic: both products on the bf16 matrix cores with fp32 accumulation
 * (the logits from the bf16 inputs as given; the weighted sum from the
 * softmax weights rounded to bf16); the softmax is split over groups of 64
 * index entries, each group's output normalised by its own fp32 sum and kept
 * in bf16, and the groups merged with their maxima and sums (flash decoding).
 * The LSE comes from the fp32 sums.  Deterministic (no atomics). */
moe_status_t dsa_sparse_attention(const dsa_attn_shape_t *s, const uint16_t *q_nope,
                                  const uint16_t *q_pe, const uint16_t *ckv, const uint16_t *kpe,
                                  const int32_t *indices, uint16_t *out, float *lse,
                                  void *workspace, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DSA_ATTENTION_MI355X_H */
