// dsa_api.cpp -- the C-ABI of the DSA TopK indexer (paper Section 3.1.3):
// argument validation, workspace carving and the launches.  No allocation and
// no host synchronisation.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/dsa_indexer.h"
#include "moe_device.h"

namespace moe {
size_t dsa_wide_ints(int B, int max_len);
}  // namespace moe

namespace {

using namespace moe;

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
template <class T>
T *at(void *ws, size_t off) {
  return reinterpret_cast<T *>(static_cast<uint8_t *>(ws) + off);
}

#define MOE_TRY_HIP(expr)                         \
  do {                                            \
    if ((expr) != hipSuccess) return MOE_ERR_HIP; \
  } while (0)

moe_status_t dsa_check(const dsa_shape_t *s) {
  if (!s || s->B < 0 || s->page_size < 1 || s->topk < 1 || s->max_pages < 1 || s->num_pages < 1)
    return MOE_ERR_INVALID_ARG;
  if (s->num_heads != 64 || s->head_dim != 128) return MOE_ERR_UNSUPPORTED;
  if (s->topk > 65536 || (int64_t)s->max_pages * s->page_size > (1 << 30) ||
      (int64_t)s->B * s->max_pages * s->page_size >= ((int64_t)1 << 31))
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

moe_status_t dsa_check_ptrs(const void *const *ptrs, int n) {
  for (int i = 0; i < n; ++i)
    if (!ptrs[i] || !aligned(ptrs[i], 16)) return MOE_ERR_INVALID_ARG;
  return MOE_OK;
}

size_t dsa_scores_bytes(const dsa_shape_t *s) {
  return align_up(sizeof(float) * (size_t)(s->B > 0 ? s->B : 1) * s->max_pages * s->page_size);
}

DsaParams dsa_params(const dsa_shape_t *s, const uint8_t *q, const float *weights,
                     const uint8_t *k_cache, const float *k_scale, const int32_t *block_table,
                     const int32_t *seq_lens, float *scores, int *hist, int32_t *out) {
  DsaParams p{q, weights, k_cache, k_scale, block_table, seq_lens, scores, hist, out, s->B,
              s->page_size, s->topk, s->max_pages, s->max_pages * s->page_size, s->num_pages};
  return p;
}

}  // namespace

extern "C" {

size_t dsa_workspace_size(const dsa_shape_t *s) {
  if (dsa_check(s) != MOE_OK) return 0;
  // the scores, then (batches that may hold long sequences) the select's
  // global state: radix histograms, slice counts, final states
  const size_t hist = dsa_wide_select(s->max_pages * s->page_size)
                          ? align_up(sizeof(int) * dsa_wide_ints(s->B > 0 ? s->B : 1, s->max_pages * s->page_size))
                          : 0;
  return dsa_scores_bytes(s) + hist;
}

moe_status_t dsa_topk_indexer(const dsa_shape_t *s, const uint8_t *q, const float *weights,
                              const uint8_t *k_cache, const float *k_scale,
                              const int32_t *block_table, const int32_t *seq_lens,
                              int32_t *out, void *workspace, size_t ws_bytes, void *stream) {
  moe_status_t rc = dsa_check(s);
  if (rc != MOE_OK) return rc;
  if (s->B == 0) return MOE_OK;
  const void *ptrs[] = {q, weights, k_cache, k_scale, block_table, seq_lens, out, workspace};
  if ((rc = dsa_check_ptrs(ptrs, 8)) != MOE_OK) return rc;
  if (ws_bytes < dsa_workspace_size(s)) return MOE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int *hist = dsa_wide_select(s->max_pages * s->page_size)
                  ? at<int>(workspace, dsa_scores_bytes(s))
                  : nullptr;
  const DsaParams p = dsa_params(s, q, weights, k_cache, k_scale, block_table, seq_lens,
                                 static_cast<float *>(workspace), hist, out);
  MOE_TRY_HIP(launch_dsa_scores(p, p.max_len, false, st));
  MOE_TRY_HIP(launch_dsa_select(p, st));
  return MOE_OK;
}

moe_status_t dsa_debug_scores(const dsa_shape_t *s, const uint8_t *q, const float *weights,
                              const uint8_t *k_cache, const float *k_scale,
                              const int32_t *block_table, const int32_t *seq_lens,
                              float *scores, void *stream) {
  moe_status_t rc = dsa_check(s);
  if (rc != MOE_OK) return rc;
  if (s->B == 0) return MOE_OK;
  const void *ptrs[] = {q, weights, k_cache, k_scale, block_table, seq_lens, scores};
  if ((rc = dsa_check_ptrs(ptrs, 7)) != MOE_OK) return rc;
  const DsaParams p = dsa_params(s, q, weights, k_cache, k_scale, block_table, seq_lens, scores,
                                 nullptr, nullptr);
  return launch_dsa_scores(p, p.max_len, true, static_cast<hipStream_t>(stream)) == hipSuccess
             ? MOE_OK
             : MOE_ERR_HIP;
}

}  // extern "C"
