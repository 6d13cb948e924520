// attention_device.h -- launch parameters of the DSA sparse attention kernels
// (paper Section 3.1.2).  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

struct AttnParams {
  const uint16_t *q_nope;   // [T, H, 512] bf16
  const uint16_t *q_pe;     // [T, H, 64] bf16
  const uint16_t *ckv;      // [rows, 512] bf16 (rows = pages * page size)
  const uint16_t *kpe;      // [rows, 64] bf16
  const int32_t *indices;   // [T, topk]: cache rows, < 0 = none
  uint16_t *part_o;         // [T, NS, H, 512] bf16 split outputs, normalised (workspace)
  float *part_ml;           // [T, NS, H, 2]  split max and sum (workspace)
  uint16_t *out;            // [T, H, 512] bf16
  float *lse;               // [T, H]
  int T, H, topk, rows, NS;
  float scale_log2;         // sm_scale * log2(e)
};

constexpr int kAttnDC = 512;       // Kc / q_nope width
constexpr int kAttnDP = 64;        // Kp / q_pe width
constexpr int kAttnEntries = 64;   // sparse entries per split workgroup
constexpr int kAttnHeads = 16;     // heads per workgroup
constexpr int kAttnMaxSplits = 1024;  // TopK <= 65536

hipError_t launch_attention(const AttnParams &p, hipStream_t st);

}  // namespace moe
