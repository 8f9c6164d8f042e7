// Internal interface between the C-ABI host code and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mlkv {

// Rotary position embedding of the newest token (GPT-NeoX: rotate-half pairs
// (j, j + half) of the first 2*half channels of every head vector).  Once per
// step the cosine and sine of each pair's angle at the token's position are
// tabulated in double, cs[(b*half + j)*2 + {0, 1}]; the attention launches
// rotate their queries and the owners' appends their keys from that table.
// inv_freq[j] = base^(-2j/(2*half)): radians pair j turns by per position.
constexpr int kMaxRopePairs = 64;
struct RopeTableParams {
  const int32_t* pos;        // [B] position of sequence b's newest token
  double* cs;                // [B][half][2] out: cos, sin
  int B, half;
  double inv_freq[kMaxRopePairs];
};

struct AppendParams {
  const uint16_t* k_new;     // row b at k_new + b*row_stride: [owned][D]
  const uint16_t* v_new;
  const int32_t* positions;  // [B] slot of the new token
  uint16_t* k;               // key plane
  uint16_t* v;               // value plane
  int B, S, kv_begin, row_stride;
  const double* rope_cs;     // null, or the step's rotary table: keys rotated before they are stored
  int rope_half;
};

// Whole-plane conversion between logical rows [kv][B][S][D] (row-major) and
// the cache planes (K identical, V in channel-major 32-token blocks), for the
// KV heads [kv_begin, kv_begin + kv_count): to_cache 1 writes the planes from
// the rows, 0 the rows from the planes.
struct CacheRowsParams {
  uint16_t* k_plane;
  uint16_t* v_plane;
  uint16_t* k_rows;          // [kv_count][B][S][D]
  uint16_t* v_rows;
  int B, S, kv_begin, kv_count, to_cache;
};

// Owners' rows of a prompt: row (b, t) at k_new + (b*T + t)*row_stride,
// [owned][D]; stored at slot ctx[b] + t (skipped outside [0, S)).
struct AppendRowsParams {
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* ctx;        // [B] tokens cached before the prompt
  uint16_t* k;               // key plane
  uint16_t* v;               // value plane
  int B, T, S, kv_begin, row_stride;
};

// Causal prefill attention of one layer: token t of sequence b attends
// positions 0 .. ctx[b] + t of the KV heads [kv_begin, kv_begin + n_groups).
// A prefill wave takes prefill_wave_blocks(D) blocks of 16 query rows (token,
// head) of one KV head; a workgroup is four such waves.
constexpr int prefill_wave_blocks(int head_dim) { return head_dim == 64 ? 2 : 1; }
constexpr int prefill_rows_per_workgroup(int head_dim) {
  return 4 * 16 * prefill_wave_blocks(head_dim);
}
struct PrefillParams {
  const uint16_t* q;         // [B][T][h][D]
  const uint16_t* k;         // key plane   [n_kv][B][S][D]
  const uint16_t* v;         // value plane [n_kv][B][S/32][D][32]
  const int32_t* ctx;        // [B] tokens cached before the prompt
  void* out;                 // [B][T][h][D] fp32 or bf16
  int B, T, h, S;
  int kv_begin, G, n_groups;
  int out_bf16;
  float scale_log2;          // log2(e) / sqrt(D)
};

// The MLP's second product of a model layer, y = f W_2 + b_2 ([rows][d],
// fp32), carried by extra workgroups of that layer's attention launch: it
// needs only the layer-in results (GPT-NeoX's parallel residual), so it runs
// beside the attention instead of after it, and the layer-out product adds y.
// Workgroup s of the product takes column block s % (d / 16) (16 outputs)
// and rows 16 (s / (d / 16)) .. +15, and sums exactly as a layer-out
// workgroup does: k-block kb of the [W_o ; W_2] packing by virtual wave kb % 8
// in increasing kb, the eight virtual waves' tiles in order.
struct SideProduct {
  const uint16_t* w;    // layer-out packing: column block blk has kt k-blocks, W_2's from ka
  const uint16_t* f16;  // [rows][ff] bf16
  const uint16_t* b2;   // [d] bf16
  float* y;             // [rows][d]
  int rows, d, ff, ka, kt;
  int n_blocks;         // (d / 16) * ceil(rows / 16); 0: no product
};

struct AttnParams {
  const uint16_t* q;         // [B][h][D]
  const uint16_t* k;         // key plane   [n_kv][B][S][D]
  const uint16_t* v;         // value plane [n_kv][B][S/32][D][32]
  const int32_t* lens;       // [B]; attended length = lens[b] + len_offset
  void* out;                 // [B][h][D] fp32 or bf16
  int* runs;                 // [B] runs per unit of sequence b (written by workgroup 0)
  void* plan;                // [n_blocks] run items to follow, or null: schedule in-kernel
  void* plan_out;            // with plan null: where each workgroup records its run item (or null)
  int* counters;             // [B*n_groups] finished runs per unit (zero between calls)
  float* part_acc;           // [B*n_groups][max_parts][G][D]  unnormalised partial outputs
  float* part_ml;            // [B*n_groups][max_parts][G][2]  (max in log2 units, denominator)
  int B, h, S, D;
  int kv_begin, G, n_groups; // KV heads [kv_begin, kv_begin+n_groups), G query heads each
  int max_len;               // attended lengths are clamped to this (<= S)
  int n_blocks;              // workgroups launched (runs beyond the schedule's count exit)
  int min_tiles;             // least tiles per run
  int max_parts;             // partial slots per unit (bound on its runs)
  int len_offset, out_bf16;
  int fused;                 // 1: the last run of a unit merges its partials when they fit LDS
  int merge_waves;           // waves merging one (sequence, head) row: 1 or 4
  int merge_first;           // partial slots the merge reads before it knows the run count
  int waves;                 // waves per attention workgroup: 4, or wide_waves() for single runs
  int direct;                // 1: n_blocks = B*n_groups, workgroup g is unit g (no schedule)
  float scale_log2;          // log2(e) / sqrt(D)
  // Fused append (owning layer of a decode step), k_new null when none: row
  // of KV head kv for sequence b at k_new + b*new_stride + kv*D; heads
  // [own_begin, own_begin + own_count) are appended at slot lens[b] + len_offset - 1.
  const uint16_t* k_new;
  const uint16_t* v_new;
  int new_stride, own_begin, own_count;
  // Rotary embedding of the step's newest token (null: none): queries are
  // rotated as they are loaded, the owner's new key before it is stored.
  const double* rope_cs;     // [B][rope_half][2] cos, sin at the token's position
  int rope_half;
};

// An attention launch that also carries a SideProduct: workgroups n_blocks ..
// n_blocks + side.n_blocks - 1 compute the product and nothing else.
struct AttnSideParams : AttnParams {
  SideProduct side;
};

// ---- GPT-NeoX layer pieces around attention (model.hip) ----
struct NormParams {  // h1 = LN1(x), h2 = LN2(x), per row
  const float* x;             // [rows][d]
  const uint16_t *w1, *b1, *w2, *b2;  // [d] bf16
  uint16_t *h1, *h2;          // [rows][d] bf16
  int rows, d;
  float eps;
};
struct QkvEpilogueParams {  // bias, rotation at pos[b], bf16 rounding
  const float* q32;           // [rows][q_width] (GEMM result)
  const uint16_t* b_q;        // [q_width]
  uint16_t* q16;              // [rows][q_width]
  const float *k32, *v32;     // [rows][kv_stride], owned block at kv_offset (kv_width wide)
  const uint16_t *b_k, *b_v;  // [kv_width]
  uint16_t *k16, *v16;        // [rows][kv_stride], same block
  const int32_t* pos;         // [rows]
  int rows, q_width, kv_width, kv_stride, kv_offset, D, dims;
  double inv_freq[kMaxRopePairs];
};
struct GeluParams {  // out16 = bf16(GELU(y32 + bias))
  const float* y32;
  const uint16_t* bias;
  uint16_t* out16;
  int rows, width;
};
struct ResidualParams {  // x += (a32 + b_o) + (m32 + b_2)
  float* x;
  const float *a32, *m32;
  const uint16_t *b_o, *b_2;
  int rows, d;
};
// Fused model-step products (B operand = batch rows, padded to 16 per tile).
// Weights are packed at model creation into MFMA A-operand tiles: tile
// (nt, kb) of a matrix with KB k-blocks holds output columns 16 nt .. +15 and
// inputs 32 kb .. +31 at element offset (nt * KB + kb) * 512; inside it,
// element (n, k) sits at ((k % 32) / 8) * 128 + (n % 16) * 8 + k % 8, so lane
// l of a wave reads elements 8 l .. 8 l + 7 (16 contiguous bytes).
constexpr int kPackTile = 512;  // bf16 elements per packed tile
constexpr int kFusedMaxBatch = 2048;  // rows of a model step on the fused path
struct PackParams {  // source W[k_rows][n_cols] row-major -> tiles (nt0 + nt, kb0 + kb)
  const uint16_t* src;
  uint16_t* dst;
  int k_rows, n_cols, kb_total, kb0, nt0, nt_count;  // k_rows % 32 == 0
};
struct LayerInParams {  // LN1/LN2 of x -> [q | k | v | fc1] products and their epilogues
  const float* x;                        // [rows][d] residual stream
  const uint16_t *ln1_w, *ln1_b, *ln2_w, *ln2_b;
  const uint16_t* w;                     // packed, column blocks of D: h q, owned k, owned v, fc1
  const uint16_t *b_q, *b_k, *b_v, *b_fc1;
  uint16_t* q16;                         // [rows][h*D]
  uint16_t *k16, *v16;                   // [rows][kv_stride], owned block at kv_offset
  uint16_t* f16;                         // [rows][ff], bf16(GELU(h2 W_1 + b_1))
  const int32_t* pos;                    // [rows] rotation position
  int rows, d, h, owned, ff, kv_stride, kv_offset, dims;
  float eps;
  double inv_freq[kMaxRopePairs];
};
struct LayerOutParams {  // x += (o W_o + b_o) + (f W_2 + b_2)
  const uint16_t *o16, *f16;  // [rows][hD], [rows][ff] bf16
  const uint16_t* w;          // packed, K = hD + ff (W_o rows, then W_2 rows), N = d
  const uint16_t *b_o, *b_2;
  float* x;
  int rows, d, hD, ff;
  const float* y_mlp;         // [rows][d] f W_2 + b_2 (SideProduct), or null: computed here
};
hipError_t launch_pack(const PackParams& p, hipStream_t stream);
hipError_t launch_layer_in(const LayerInParams& p, int head_dim, hipStream_t stream);
hipError_t launch_layer_out(const LayerOutParams& p, hipStream_t stream);

hipError_t launch_norm2(const NormParams& p, hipStream_t stream);
hipError_t launch_qkv_epilogue(const QkvEpilogueParams& p, hipStream_t stream);
hipError_t launch_gelu(const GeluParams& p, hipStream_t stream);
hipError_t launch_residual(const ResidualParams& p, hipStream_t stream);

hipError_t launch_append(const AppendParams& p, int head_dim, int owned_count,
                         hipStream_t stream);
hipError_t launch_rope_table(const RopeTableParams& p, hipStream_t stream);
hipError_t launch_cache_rows(const CacheRowsParams& p, int head_dim, hipStream_t stream);
hipError_t launch_append_rows(const AppendRowsParams& p, int head_dim, int owned_count,
                              hipStream_t stream);
// start/stop: optional events recorded around the prefill dispatch.
hipError_t launch_prefill(const PrefillParams& p, int head_dim, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop);
// The split-K attention kernel, then (when splits are merged by a separate
// kernel) the merge.
// start/stop: optional events recorded around the attention dispatch.
// side: a product the launch also carries (null or n_blocks 0: none).
hipError_t launch_attention_main(const AttnParams& p, int head_dim, hipStream_t stream,
                                 hipEvent_t start, hipEvent_t stop,
                                 const SideProduct* side = nullptr);
// stop: optional event recorded when the merge kernel completes.
hipError_t launch_attention_merge(const AttnParams& p, int head_dim, hipStream_t stream,
                                  hipEvent_t stop);
int max_batch();
int stage_floats();  // partial-output floats one workgroup can merge in place
int resident_workgroups(int head_dim); // attention workgroups the device holds at once (0: none)
int wide_waves();                      // waves per workgroup of the one-run-per-unit layout
int compute_units();                   // compute units of the current device (0: unknown)
int default_waves();                   // waves per workgroup otherwise
hipError_t launch_fill(uint32_t* dst, size_t n_words, uint32_t value, hipStream_t stream);
// The library's static device scratch (scratch.hip): kScratchBytes per device.
// Returns its device address on the current device, looked up (and zero
// filled on `stream`) on the first call per device.
constexpr size_t kScratchBytes = size_t(16) << 20;
hipError_t scratch_for_current_device(hipStream_t stream, void** ptr);
// An empty kernel bracketed by start/stop (launch-overhead reference).
hipError_t launch_empty_timed(int workgroups, int threads, hipStream_t stream, hipEvent_t start,
                              hipEvent_t stop);
// A streaming read of `bytes` (a multiple of 16) at src bracketed by
// start/stop; sink receives one word only for an impossible data pattern.
hipError_t launch_stream_read_timed(const void* src, size_t bytes, uint32_t* sink, int workgroups,
                                    hipStream_t stream, hipEvent_t start, hipEvent_t stop);

}  // namespace mlkv
