// Internal interface between the C-ABI host code and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mlkv {

struct AppendParams {
  const uint16_t* k_new;     // row b at k_new + b*row_stride: [owned][D]
  const uint16_t* v_new;
  const int32_t* positions;  // [B] slot of the new token
  uint16_t* k;               // key plane
  uint16_t* v;               // value plane
  int B, S, kv_begin, row_stride;
};

struct AttnParams {
  const uint16_t* q;         // [B][h][D]
  const uint16_t* k;         // key plane   [n_kv][B][S][D]
  const uint16_t* v;         // value plane [n_kv][B][S/32][D][32]
  const int32_t* lens;       // [B]; attended length = lens[b] + len_offset
  void* out;                 // [B][h][D] fp32 or bf16
  float* part_acc;           // [B*n_groups][n_split][G][D]  unnormalised partial outputs
  float* part_ml;            // [B*n_groups][n_split][G][2]  (max in log2 units, denominator)
  int* counters;             // [B * n_groups] finished splits per sequence (zero between calls)
  int B, h, S;
  int kv_begin, G, n_groups; // KV heads [kv_begin, kv_begin+n_groups), G query heads each
  int n_split, tiles_per_split;
  int len_offset, out_bf16;
  int fused_combine;         // 1: last workgroup of a sequence merges; 0: combine kernel
  float scale_log2;          // log2(e) / sqrt(D)
};

hipError_t launch_append(const AppendParams& p, int head_dim, int owned_count,
                         hipStream_t stream);
hipError_t launch_attention(const AttnParams& p, int head_dim, hipStream_t stream);
int fused_partial_capacity();  // floats of partial output the fused combine can stage
hipError_t launch_fill(uint32_t* dst, size_t n_words, uint32_t value, hipStream_t stream);

}  // namespace mlkv
