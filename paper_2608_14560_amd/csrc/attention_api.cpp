// attention_api.cpp -- the C-ABI of the DSA sparse attention: argument
// validation, workspace carving and the two launches.  No allocation and no
// host synchronisation.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/dsa_attention.h"
#include "attention_device.h"

namespace {

using namespace moe;

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

moe_status_t attn_check(const dsa_attn_shape_t *s) {
  if (!s || s->T < 0 || s->num_heads < 1 || s->topk < 1 || s->num_rows < 1 ||
      !std::isfinite(s->sm_scale))
    return MOE_ERR_INVALID_ARG;
  if (s->num_heads % kAttnHeads || s->topk > 65536 || (int64_t)s->T * s->num_heads > (1 << 26))
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

int splits(const dsa_attn_shape_t *s) { return (s->topk + kAttnEntries - 1) / kAttnEntries; }

size_t part_o_bytes(const dsa_attn_shape_t *s) {
  return align_up(sizeof(uint16_t) * (size_t)(s->T > 0 ? s->T : 1) * splits(s) * s->num_heads * kAttnDC);
}

}  // namespace

extern "C" {

size_t dsa_attention_workspace_size(const dsa_attn_shape_t *s) {
  if (attn_check(s) != MOE_OK) return 0;
  return part_o_bytes(s) +
         align_up(sizeof(float) * 2 * (size_t)(s->T > 0 ? s->T : 1) * splits(s) * s->num_heads);
}

moe_status_t dsa_sparse_attention(const dsa_attn_shape_t *s, const uint16_t *q_nope,
                                  const uint16_t *q_pe, const uint16_t *ckv, const uint16_t *kpe,
                                  const int32_t *indices, uint16_t *out, float *lse,
                                  void *workspace, size_t ws_bytes, void *stream) {
  moe_status_t rc = attn_check(s);
  if (rc != MOE_OK) return rc;
  if (s->T == 0) return MOE_OK;
  const void *ptrs[] = {q_nope, q_pe, ckv, kpe, indices, out, lse, workspace};
  for (const void *q : ptrs)
    if (!q || !aligned(q, 16)) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < dsa_attention_workspace_size(s)) return MOE_ERR_WORKSPACE_TOO_SMALL;
  AttnParams p{};
  p.q_nope = q_nope;
  p.q_pe = q_pe;
  p.ckv = ckv;
  p.kpe = kpe;
  p.indices = indices;
  p.part_o = static_cast<uint16_t *>(workspace);
  p.part_ml = reinterpret_cast<float *>(static_cast<uint8_t *>(workspace) + part_o_bytes(s));
  p.out = out;
  p.lse = lse;
  p.T = s->T;
  p.H = s->num_heads;
  p.topk = s->topk;
  p.rows = s->num_rows;
  p.NS = splits(s);
  p.scale_log2 = s->sm_scale * 1.4426950408889634f;
  return launch_attention(p, static_cast<hipStream_t>(stream)) == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

}  // extern "C"
