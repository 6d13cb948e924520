/*
 * dsa_indexer.h -- C-ABI of the MI355X (gfx950) DSA TopK Indexer: the paged
 * attention indexing stage of DSA sparse attention (paper Section 3.1.3).
 *
 * For each batch element b and each cached token j < seq_lens[b]:
 *   score(j) = sum over heads h of ReLU(q[b, h, :] . k_j) * weights[b, h]
 * where k_j is token j's key row dequantised with its fp32 scale; the
 * operator returns the topk highest-scoring tokens of each sequence.
 *
 * Same conventions as moe.h: device pointers, row-major, 16-byte aligned;
 * the caller owns every buffer including the workspace; asynchronous on
 * `stream`; arguments are checked before anything is enqueued; nothing
 * synchronises the host or allocates.  Status codes are moe_status_t.
 */
#ifndef DSA_INDEXER_MI355X_H
#define DSA_INDEXER_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include "moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Problem shape.  Limits of this library: num_heads 64, head_dim 128 (the
 * paper's operator); page_size >= 1; 1 <= topk <= 65536; B >= 0. */
typedef struct {
  int32_t B;          /* batch elements (sequences)                      */
  int32_t num_heads;  /* query heads (64)                                */
  int32_t head_dim;   /* 128                                             */
  int32_t page_size;  /* tokens per cache page (64 in the paper)         */
  int32_t topk;       /* tokens returned per sequence (2048)             */
  int32_t max_pages;  /* columns of block_table                          */
  int32_t num_pages;  /* pages in the key cache                          */
} dsa_shape_t;

/* Bytes of device workspace dsa_topk_indexer needs for `s` (the scores of
 * every sequence at its longest possible length; for block tables of 16,384
 * tokens or more also the long-sequence select's radix histograms, per-slice
 * counts and final states); 0 for an invalid shape. */
size_t dsa_workspace_size(const dsa_shape_t *s);

/* The indexer (Section 3.1.3).
 *  q            [B, 64, 128] e4m3
 *  weights      [B, 64] float
 *  k_cache      [num_pages, page_size, 128] e4m3
 *  k_scale      [num_pages, page_size] float (one scale per cached token)
 *  block_table  [B, max_pages] int32: token j of sequence b is slot
 *               j % page_size of page block_table[b][j / page_size]
 *  seq_lens     [B] int32 (read on the device; values are clamped into
 *               [0, max_pages * page_size] and page ids into [0, num_pages),
 *               so invalid device data gives wrong indices, never a fault)
 *  out          [B, topk] int32: the selected tokens' physical cache indices
 *               page * page_size + slot, in ascending position order, the
 *               rest of the row -1.  A sequence of at most topk tokens
 *               returns all of its tokens (no scores are computed for it).
 * Scores follow one fixed fp32 sequence (the returned set depends on it bit
 * for bit): kd = decode(k) * scale rounded to fp32; per head a fused
 * multiply-add chain over the 128 dimensions in ascending order from 0 of
 * decode(q) * kd; then a fused multiply-add chain over the heads in
 * ascending order from 0 of (dot > 0 ? dot : 0) * weight.  Selection: larger
 * score first, equal scores to the lower position.  Bitwise deterministic. */
moe_status_t dsa_topk_indexer(const dsa_shape_t *s, const uint8_t *q, const float *weights,
                              const uint8_t *k_cache, const float *k_scale,
                              const int32_t *block_table, const int32_t *seq_lens,
                              int32_t *out, void *workspace, size_t ws_bytes, void *stream);

/* Test hook: scores [B, max_pages * page_size] float of every token of every
 * sequence (also those of at most topk tokens), exactly as dsa_topk_indexer
 * computes them; entries past a sequence's length are not written. */
moe_status_t dsa_debug_scores(const dsa_shape_t *s, const uint8_t *q, const float *weights,
                              const uint8_t *k_cache, const float *k_scale,
                              const int32_t *block_table, const int32_t *seq_lens,
                              float *scores, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DSA_INDEXER_MI355X_H */
