/*
 * mlkv.h — MLKV decode attention on AMD Instinct MI355X (gfx950).
 *
 * Multi-Layer Key-Value sharing (arXiv 2406.09297): query head i of layer n
 * attends to a KV head that is shared by a group of query heads inside the
 * layer (GQA grouping, Section 2.3, Eq. 12) and by a group of consecutive
 * layers (Section 3, Eqs. 13-17).  Only the layer that owns a KV head appends
 * the newest token's key/value to the cache (Section 2.4 caching; the shared
 * head comes from the bottom layer of its group, Figure 2).
 *
 * Everything here is a plain C ABI: device pointers, sizes and a HIP stream.
 * All entry points are synchronous on the host only for argument validation;
 * device work is enqueued on `stream` and nothing synchronizes.  No entry
 * point throws; each returns an mlkv_status and mlkv_last_error() gives a
 * thread-local message for the last failure.  Argument errors are detected
 * before any HIP call is made.
 *
 * Data types: bf16 storage for q, k, v and the cache (raw 16-bit patterns),
 * fp32 accumulation, output fp32 or bf16.
 */
#ifndef MLKV_H_
#define MLKV_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ----------------------------------------------------------------------- */
/* Status                                                                    */
/* ----------------------------------------------------------------------- */

typedef enum {
  MLKV_OK = 0,
  MLKV_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, bad enum     */
  MLKV_ERR_BAD_MAP = 2,     /* layer->KV-head map violates the rules below   */
  MLKV_ERR_ALIGNMENT = 3,   /* a device pointer is not 16-byte aligned       */
  MLKV_ERR_UNSUPPORTED = 4, /* head_dim or query-group size not supported    */
  MLKV_ERR_CAPACITY = 5,    /* capacity / max_len_hint / lengths out of range */
  MLKV_ERR_WORKSPACE = 6,   /* workspace missing or too small                */
  MLKV_ERR_HIP = 7          /* a HIP runtime call or launch failed           */
} mlkv_status;

typedef enum { MLKV_OUT_F32 = 0, MLKV_OUT_BF16 = 1 } mlkv_out_dtype;

/* Static string naming the status.  Never NULL. */
const char* mlkv_status_string(mlkv_status status);
/* Message of the last failing call on this thread ("" if none).  Owned by the
 * library, valid until the next call on the same thread. */
const char* mlkv_last_error(void);

/* ----------------------------------------------------------------------- */
/* Layer -> KV-head map (Section 2.3 Eq. 12, Section 3 Eqs. 15 and 17)       */
/* ----------------------------------------------------------------------- */

typedef struct mlkv_map mlkv_map; /* opaque, host-only, owned by the library */

/*
 * Uniform MLKV map: l layers with h query heads; m of the layers own g KV
 * heads each (n_kv = m*g).  In 0-indexed form of the paper's formulas, layer n
 * belongs to layer-group k = n / (l/m) and its query head i uses in-layer
 * group j = i / (h/g); the global KV head is k*g + j, owned (appended) by the
 * bottom layer of the group, k*(l/m).
 * m = l, g = h gives MHA; m = l, g = 1 gives MQA; m = l gives GQA.
 * Errors: MLKV_ERR_INVALID_ARG if any argument is <= 0, if m does not divide l
 * or g does not divide h, or out is NULL.
 */
mlkv_status mlkv_map_create_uniform(int l, int h, int m, int g, mlkv_map** out);

/*
 * General map from explicit tables (e.g. non-uniform cross-layer patterns).
 * kv_of [l*h]: KV head of query head i in layer n at kv_of[n*h + i].
 * owner_of [n_kv]: the layer that appends KV head kv.
 * The arrays are copied; the caller keeps ownership.  Rules (else
 * MLKV_ERR_BAD_MAP):
 *   - every entry in range; every KV head is read by at least one layer;
 *   - in each layer the heads read form a contiguous range of KV heads
 *     [kv_begin, kv_begin + c) with c dividing h, and query head i reads
 *     kv_begin + i / (h/c)  (GQA grouping within the layer);
 *   - owner_of[kv] <= every layer that reads kv (the owner appends first);
 *   - each layer owns a contiguous range of KV heads.
 */
mlkv_status mlkv_map_create(int l, int h, int n_kv, const int32_t* kv_of,
                            const int32_t* owner_of, mlkv_map** out);
void mlkv_map_destroy(mlkv_map* map); /* NULL is ignored */

int mlkv_map_num_layers(const mlkv_map* map);
int mlkv_map_num_q_heads(const mlkv_map* map);
int mlkv_map_num_kv_heads(const mlkv_map* map);              /* m*g for uniform maps */
int mlkv_map_kv_head(const mlkv_map* map, int layer, int q_head); /* -1 if out of range */
int mlkv_map_owner_layer(const mlkv_map* map, int kv);            /* -1 if out of range */
/* Number of KV heads layer `layer` reads (g for uniform maps), -1 if out of range. */
int mlkv_map_layer_kv_count(const mlkv_map* map, int layer);
/* Number of KV heads layer `layer` appends (0 for non-owning layers). */
int mlkv_map_layer_owned_count(const mlkv_map* map, int layer);
/* First KV head layer `layer` appends (-1 if it owns none). */
int mlkv_map_layer_owned_begin(const mlkv_map* map, int layer);

/* ----------------------------------------------------------------------- */
/* KV cache                                                                  */
/* ----------------------------------------------------------------------- */

/*
 * Caller-owned device memory (e.g. torch tensors); the library never frees it.
 * capacity must be a multiple of 32; head_dim 64 or 128; both planes 16-byte
 * aligned.  Element (kv, b, t, d), t < capacity, lives at
 *   K: k[((kv*batch + b)*capacity + (t & ~31))*head_dim + 8*q(t & 31, d >> 3) + (d & 7)]
 *      with q(u, c) = ((((u >> 2) & 1)*(head_dim/32) + (c >> 2))*64
 *                      + (c & 3)*16 + ((u >> 3) << 2) + (u & 3))
 *      (keys in blocks of 32 tokens; inside a block, the 16-byte chunks of
 *      channels 8c .. 8c+7 are ordered as the matrix-core operands of the
 *      block's two 16-token halves and 32-channel steps, so each 1 KB run of
 *      the block is one load instruction of a wave)
 *   V: v[((kv*batch + b)*capacity + (t & ~31))*head_dim + d*32 + (t & 31)]
 *      (values in blocks of 32 tokens, channel-major inside a block, so a
 *      block is the transposed 32 x head_dim tile)
 * Both planes hold n_kv*batch*capacity*head_dim bf16 values.
 */
typedef struct {
  void* k;
  void* v;
  int n_kv;
  int batch;
  int capacity;
  int head_dim;
} mlkv_cache;

/* Bytes of one cache (both planes): 2 * batch * capacity * n_kv * head_dim * 2,
 * the paper's 2*b*s*m*g*d_k elements (Section 3, Table 1) in bf16.
 * Returns 0 for invalid arguments. */
size_t mlkv_cache_bytes(const mlkv_map* map, int batch, int capacity, int head_dim);

/*
 * Fill cache planes from plain rows, on the device (for a cache filled from
 * outside the decode path, e.g. by a prefill elsewhere, or a migration):
 *   k_rows, v_rows: device bf16 [kv_count][batch][capacity][head_dim], token
 *                   rows in plain row-major order (element (c, b, t, d) at
 *                   ((c*batch + b)*capacity + t)*head_dim + d), 16-byte aligned.
 * KV heads [kv_begin, kv_begin + kv_count) of the cache receive them: the key
 * plane as is, the value plane in its 32-token channel-major blocks (layout
 * above).  Every slot of those heads is written, nothing else.  kv_count 0
 * does nothing.  Errors: MLKV_ERR_INVALID_ARG (NULL pointers, a head range
 * outside [0, n_kv)), MLKV_ERR_ALIGNMENT, MLKV_ERR_CAPACITY (capacity not a
 * multiple of 32, or more than 2^31 - 1 blocks of 32 tokens), MLKV_ERR_UNSUPPORTED
 * (head_dim), MLKV_ERR_HIP.  Enqueued on `stream`; the rows must not overlap
 * the planes.
 */
mlkv_status mlkv_cache_write_rows(const mlkv_cache* cache, int kv_begin, int kv_count,
                                  const void* k_rows, const void* v_rows, hipStream_t stream);
/* The reverse: KV heads [kv_begin, kv_begin + kv_count) of the cache planes
 * out to plain rows in the same [kv_count][batch][capacity][head_dim] order.
 * Same arguments and errors. */
mlkv_status mlkv_cache_read_rows(const mlkv_cache* cache, int kv_begin, int kv_count,
                                 void* k_rows, void* v_rows, hipStream_t stream);

/* Device workspace needed by mlkv_decode_attention / mlkv_decode_step for any
 * max_len_hint <= capacity (split-K partial results and per-sequence split
 * counters), sized for the current device.  0 for invalid args, and 0 when
 * every layer has at least as many (sequence, KV head) units as the device's
 * attention workgroup budget (two per compute unit): those launches give each
 * unit a workgroup of its own and need no workspace. */
size_t mlkv_workspace_bytes(const mlkv_map* map, int batch, int capacity, int head_dim);

/* Zero-fill a workspace before its first use (a fill kernel enqueued on
 * `stream`, no memset, so it may be captured in a graph).  Every decode call
 * leaves the workspace's counters (its first 256 KiB, whatever the batch or
 * map of the call) at zero again, so this is needed once per allocation, also
 * when calls with different batches or maps share the workspace.  Calls that
 * share one workspace must be ordered on one stream. */
mlkv_status mlkv_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Append the newest token of `layer` (Section 2.4) into the KV heads that
 * layer owns; a no-op returning MLKV_OK for layers that own none.
 *   k_new, v_new: device bf16, row b at k_new + b*new_row_stride elements,
 *                 holding the owned heads' rows back to back
 *                 ([owned_count][head_dim]); 16-byte aligned,
 *                 new_row_stride a multiple of 8 and >= owned_count*head_dim.
 *   positions:    device int32 [batch]; the token goes to slot positions[b].
 *                 Slots outside [0, capacity) are skipped (no write).
 * Bit copy: nothing else in the cache changes.
 */
mlkv_status mlkv_cache_append(int layer, const mlkv_map* map, const mlkv_cache* cache,
                              const void* k_new, const void* v_new, int new_row_stride,
                              const int32_t* positions, hipStream_t stream);

/*
 * Decode attention of one layer (Eqs. 1-3 with the MLKV head map, Eq. 14):
 *   out[b][i][:] = softmax(q[b][i] . K_kv[b][t]^T / sqrt(head_dim))_t V_kv[b][t]
 * over t in [0, L_b), kv = kv head of (layer, i), L_b = seq_lens[b] (device
 * int32 [batch]) clamped to [0, capacity]; L_b = 0 gives zeros.
 *   q:   device bf16 [batch][h][head_dim], 16-byte aligned.
 *   out: device [batch][h][head_dim], fp32 or bf16 per out_dtype.
 *   max_len_hint: an upper bound of every L_b (<= 0 means capacity); it sizes
 *        the work plan.  Lengths above it are truncated to it.
 *   batch: any size when the layer's (sequence, KV head) units are at least
 *        the device's workgroup budget (two per compute unit; then each
 *        unit is one workgroup and no workspace is used); otherwise at most
 *        2048 sequences (else MLKV_ERR_UNSUPPORTED, before any launch).
 *   workspace: device memory of at least mlkv_workspace_bytes(...) bytes,
 *        16-byte aligned, zeroed once by mlkv_workspace_init (the split
 *        counters must start at zero; each call returns them to zero).
 * Every query head mapped to one KV head is served from a single pass over
 * that head's cache rows.  The tiles of all sequences are shared equally by
 * the workgroups (ragged batches stay balanced); a sequence spread over
 * several workgroups is merged in a fixed order, by the last of those
 * workgroups to finish when their partial results fit its staging area, else
 * by a second kernel, so results are bitwise reproducible.
 */
mlkv_status mlkv_decode_attention(int layer, const void* q, const mlkv_cache* cache,
                                  const mlkv_map* map, const int32_t* seq_lens, void* out,
                                  mlkv_out_dtype out_dtype, int max_len_hint, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/*
 * One decode step over all layers (Eq. 17): for n = 0..l-1, append the newest
 * token into the heads layer n owns (slot ctx_lens[b]), then attend every
 * query head of layer n over ctx_lens[b] + 1 positions.
 *   q_all:   device bf16 [l][batch][h][head_dim]
 *   k_new_all, v_new_all: device bf16 [batch][n_kv][head_dim]
 *   ctx_lens: device int32 [batch], tokens cached before the step; the caller
 *             increments them after the step.
 *   out_all: device [l][batch][h][head_dim], fp32 or bf16.
 *   max_len_hint: bound of ctx_lens[b] + 1 (<= 0 means capacity).
 */
mlkv_status mlkv_decode_step(const void* q_all, const void* k_new_all, const void* v_new_all,
                             const mlkv_cache* cache, const mlkv_map* map,
                             const int32_t* ctx_lens, void* out_all, mlkv_out_dtype out_dtype,
                             int max_len_hint, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/*
 * mlkv_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops or harnesses that forbid allocation): the
 * same step, arguments and results, but with no workspace argument.  The
 * split runs' counters, run list and partial results live in the library's
 * own static device scratch of 16 MiB per device (allocated with the code
 * object when the library is loaded on a device, held until the process
 * ends); this call allocates nothing.  The first call on a device looks up
 * the scratch's address and zero-fills it on `stream`.
 * A step whose workspace need (that of mlkv_decode_step for these arguments;
 * at most mlkv_workspace_bytes) exceeds 16 MiB is rejected with
 * MLKV_ERR_WORKSPACE before anything is launched.  Every call on a device
 * shares that device's scratch: calls that overlap on one device (on
 * different streams, or from different threads without ordering) race and
 * give wrong results; order them on one stream.
 */
mlkv_status mlkv_decode_step_noalloc(const void* q_all, const void* k_new_all,
                                     const void* v_new_all, const mlkv_cache* cache,
                                     const mlkv_map* map, const int32_t* ctx_lens, void* out_all,
                                     mlkv_out_dtype out_dtype, int max_len_hint,
                                     hipStream_t stream);

/*
 * mlkv_decode_step with the rotary position embedding of the GPT-NeoX
 * architecture that the paper's Pythia models use (Section 4.2) applied to
 * the newest token inside the step: each attention launch rotates the
 * queries it loads and each owning layer rotates the new keys before storing
 * them, so the cache holds rotated keys.  q_all and k_new_all are read only
 * (never written): repeating a call on the same buffers, or replaying it
 * from a captured graph, gives the same outputs and cache.
 * Rotation: channel pairs (j, j + rotary_dims/2), j < rotary_dims/2, of each
 * head vector turn by ctx_lens[b] * rotary_base^(-2j/rotary_dims) radians;
 * the cosine and sine are tabulated once per step in double (in the first
 * mlkv_workspace_bytes_rope - mlkv_workspace_bytes bytes of the workspace),
 * each rotated value is computed in double (products and sum each rounded)
 * and rounded once to bf16, nearest even; channels at or past rotary_dims
 * and the values are not rotated.  Pythia-160M: rotary_dims 16, rotary_base
 * 10000.
 *   rotary_dims: a multiple of 16 in [0, head_dim] (else
 *                MLKV_ERR_UNSUPPORTED); 0 is mlkv_decode_step.
 *   rotary_base: positive and finite (else MLKV_ERR_INVALID_ARG).
 *   workspace:   at least mlkv_workspace_bytes_rope(...) bytes, 16-byte
 *                aligned, initialised once by mlkv_workspace_init (else
 *                MLKV_ERR_WORKSPACE / MLKV_ERR_ALIGNMENT).
 * Other arguments and errors as mlkv_decode_step; every check is made before
 * anything is launched.
 */
mlkv_status mlkv_decode_step_rope(const void* q_all, const void* k_new_all, const void* v_new_all,
                                  const mlkv_cache* cache, const mlkv_map* map,
                                  const int32_t* ctx_lens, int rotary_dims, double rotary_base,
                                  void* out_all, mlkv_out_dtype out_dtype, int max_len_hint,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace of mlkv_decode_step_rope: the rotary table (batch *
 * rotary_dims/2 (cos, sin) pairs in double, rounded up to 256 bytes) followed
 * by a decode workspace of mlkv_workspace_bytes(map, batch, capacity,
 * head_dim) bytes.  0 for invalid arguments (rotary_dims as above). */
size_t mlkv_workspace_bytes_rope(const mlkv_map* map, int batch, int capacity, int head_dim,
                                 int rotary_dims);

/* ----------------------------------------------------------------------- */
/* Prefill: T new tokens per sequence (a prompt, or a chunk of one)          */
/* ----------------------------------------------------------------------- */

/*
 * The cache of Section 2.4 filled from a prompt; under MLKV (Section 3) the
 * owning layer stores the new keys/values and every layer of its group
 * attends to them.  Token t (0 <= t < T) of sequence b sits at position
 * ctx_lens[b] + t and attends causally to positions 0 .. ctx_lens[b] + t
 * (the cached prefix, the earlier new tokens and itself).
 * ctx_lens: device int32 [batch], tokens cached before the call; each must be
 *   in [0, capacity - T].  They are read on the device and validated only
 *   under MLKV_CHECK=1 (which synchronizes); out-of-range values never make
 *   a kernel leave the cache (slots outside [0, capacity) are not written,
 *   positions are clamped to the capacity), but their results are unspecified.
 * T: 0 <= T <= capacity (else MLKV_ERR_CAPACITY); T = 0 does nothing.
 *   T times the query heads per KV head must not exceed 8,388,480 for
 *   head_dim 64 and 4,194,240 for 128 (65535 workgroups of 128 / 64 query
 *   rows; else MLKV_ERR_UNSUPPORTED).  Any group size is accepted (no
 *   16-head limit).
 * No workspace: each query row is finished by one wave.
 */

/* The T new rows of the KV heads `layer` owns, stored at slots
 * ctx_lens[b] + t (bit copy); a no-op for layers that own none.
 *   k_new, v_new: device bf16, row (b, t) at k_new + (b*T + t)*new_row_stride
 *                 elements, holding the owned heads' rows back to back;
 *                 16-byte aligned, new_row_stride a multiple of 8 and
 *                 >= owned_count*head_dim. */
mlkv_status mlkv_cache_append_rows(int layer, const mlkv_map* map, const mlkv_cache* cache,
                                   const void* k_new, const void* v_new, int T,
                                   int new_row_stride, const int32_t* ctx_lens,
                                   hipStream_t stream);

/* Causal attention of every query head of `layer` for the T new tokens.
 *   q:   device bf16 [batch][T][h][head_dim], 16-byte aligned.
 *   out: device [batch][T][h][head_dim] fp32 or bf16 (out_dtype), 16-byte
 *        aligned.
 * The owners' new rows must already be in the cache (mlkv_cache_append_rows
 * of the owning layer). */
mlkv_status mlkv_prefill_attention(int layer, const void* q, const mlkv_cache* cache,
                                   const mlkv_map* map, const int32_t* ctx_lens, int T, void* out,
                                   mlkv_out_dtype out_dtype, hipStream_t stream);

/* The whole prefill of a model (Eq. 17's layer order): for n = 0..l-1 the
 * heads layer n owns take their T new rows, then layer n attends.
 *   q_all:     device bf16 [l][batch][T][h][head_dim].
 *   k_new_all, v_new_all: device bf16 [batch][T][n_kv][head_dim] (every KV
 *              head's new rows; each owner stores its columns).
 *   out_all:   device [l][batch][T][h][head_dim], fp32 or bf16.
 * All 16-byte aligned.  Every check is made before anything is launched. */
mlkv_status mlkv_prefill_step(const void* q_all, const void* k_new_all, const void* v_new_all,
                              const mlkv_cache* cache, const mlkv_map* map,
                              const int32_t* ctx_lens, int T, void* out_all,
                              mlkv_out_dtype out_dtype, hipStream_t stream);

/* ----------------------------------------------------------------------- */
/* Model-level decode step: GPT-NeoX layers around the MLKV attention        */
/* ----------------------------------------------------------------------- */

/*
 * One decode step of a GPT-NeoX model (the architecture of the paper's Pythia
 * models, Section 4.2) whose attention follows an MLKV map (Section 3): per
 * layer n, with x the newest token's residual stream,
 *   h1 = LayerNorm1(x), h2 = LayerNorm2(x)
 *   q  = h1 W_q + b_q; in a layer owning KV heads k = h1 W_k + b_k,
 *   v = h1 W_v + b_v (a layer owning none computes no key or value: the
 *   compute MLKV saves); q and k rotated at position ctx_lens[b] (rotary
 *   embedding of the first rotary_dims channels of each head)
 *   the owner stores k, v at slot ctx_lens[b]; every query head attends over
 *   ctx_lens[b] + 1 positions of its KV head (as mlkv_decode_step)
 *   x += (o W_o + b_o) + (GELU(h2 W_1 + b_1) W_2 + b_2)  (exact GELU; the
 *   parallel residual)
 * Matrix products take bf16 operands and accumulate in fp32.  When the model
 * holds packed weights (mlkv_model_create), they run, for any batch, in two
 * fused kernels per layer around the attention: layer norms, the
 * q/k/v and fc1 products, bias, rotation and GELU in one; the output product,
 * biases and the residual in the other (weights packed into the matrix
 * cores' operand tiles).  The fc2 product runs beside the attention, in
 * extra workgroups of its launch (it needs only the first kernel's results),
 * with the same sums as if the second kernel formed it.  Otherwise the products are library GEMMs (rocBLAS)
 * between the library's layer-norm, epilogue and residual kernels; the
 * environment variable MLKV_MODEL_GEMM=library selects that path for any
 * batch.  Either way stored in bf16: h1, h2, the rotated q and k, v, the
 * attention output and the GELU output (nearest, ties to even); x stays fp32.
 */
typedef struct mlkv_model mlkv_model; /* opaque, owned by the library */

/* Device pointers of one layer's weights, bf16, matrices row-major [in][out].
 * mlkv_model_create copies the matrices into packed tiles (the fused path)
 * and keeps the pointers for the library-GEMM path and the vectors: the
 * caller keeps the memory alive and unchanged while the model exists. */
typedef struct {
  const void* ln1_w; const void* ln1_b;   /* [d_model] */
  const void* ln2_w; const void* ln2_b;   /* [d_model] */
  const void* w_q;   const void* b_q;     /* [d_model][h*head_dim], [h*head_dim] */
  const void* w_k;   const void* b_k;     /* [d_model][owned*head_dim], [owned*head_dim]; */
  const void* w_v;   const void* b_v;     /*   NULL in a layer that owns no KV head */
  const void* w_o;   const void* b_o;     /* [h*head_dim][d_model], [d_model] */
  const void* w_fc1; const void* b_fc1;   /* [d_model][d_ff], [d_ff] */
  const void* w_fc2; const void* b_fc2;   /* [d_ff][d_model], [d_model] */
} mlkv_layer_weights;

/* d_model must equal h * head_dim (head_dim 64 or 128); rotary_dims even, in
 * [0, head_dim]; rotary_base > 0; ln_eps >= 0; layers[l] with the key/value
 * pointers set exactly in the layers that own KV heads.  Creates the GEMM
 * library handle and, when d_ff % 32 == 0 and the layer-norm vectors are
 * 16-byte aligned, allocates device memory for the packed matrices (2 bytes
 * per weight, every layer) and fills it after synchronizing the device (so
 * the caller's writes of the weights on any stream are complete), finished
 * before returning.  mlkv_model_destroy frees both.
 * Errors: MLKV_ERR_INVALID_ARG, MLKV_ERR_UNSUPPORTED, MLKV_ERR_HIP. */
mlkv_status mlkv_model_create(const mlkv_map* map, int d_model, int d_ff, int head_dim,
                              int rotary_dims, double rotary_base, double ln_eps,
                              const mlkv_layer_weights* layers, mlkv_model** out);
void mlkv_model_destroy(mlkv_model* model);

/* Device workspace of mlkv_model_decode_step (intermediate rows plus the
 * attention workspace of mlkv_workspace_bytes); 0 for invalid arguments.
 * Initialise it once with mlkv_workspace_init. */
size_t mlkv_model_workspace_bytes(const mlkv_model* model, int batch, int capacity);

/* One decode step in place: x device fp32 [batch][d_model] (16-byte
 * aligned) is the newest token's residual stream on entry and after the last
 * layer on return; the cache gains the owners' rows at slot ctx_lens[b].
 * ctx_lens, cache, max_len_hint as mlkv_decode_step.  The GEMM library may
 * size its own workspace on the first call. */
mlkv_status mlkv_model_decode_step(mlkv_model* model, float* x, const mlkv_cache* cache,
                                   const int32_t* ctx_lens, int max_len_hint, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/* ----------------------------------------------------------------------- */
/* Introspection (tests and benchmarks)                                      */
/* ----------------------------------------------------------------------- */

/* 1 when mlkv_model_decode_step runs `batch` sequences on the fused kernels
 * (packed weights, MLKV_MODEL_GEMM not "library"), 0 when on
 * library GEMMs or for invalid arguments. */
int mlkv_model_fused_path(const mlkv_model* model, int batch);

/* Work plan mlkv_decode_attention uses for `layer` at this max length: the
 * 32-token tiles of all (sequence, KV head) pairs form one flat list shared
 * equally by `workgroups` workgroups (two per compute unit, or the device's
 * resident capacity if lower; capped at 128 per (sequence, KV head) and at
 * one per 8 tiles; above the compute-unit count a whole multiple of it; at
 * least one per (sequence, KV head); one workgroup for at most 16 tiles;
 * with at least as many (sequence, KV head) pairs as the
 * budget, exactly one workgroup per pair).  A layer whose KV heads were all
 * appended by earlier layers (it re-reads them) gets one eight-wave
 * workgroup per pair instead when the pairs number at least 3/8 of the
 * compute units and fewer than the budget.  `max_parts` bounds the
 * workgroups covering one sequence.
 * Environment overrides, read on every call (tests and tuning):
 *   MLKV_WORKGROUPS=n   workgroup budget n instead of the device's;
 *   MLKV_COMBINE=kernel always merge split runs with the separate merge
 *                       kernel (by default the last run of each unit merges
 *                       them in place when they fit the kernel's staging
 *                       area, at the full workgroup count or, failing that,
 *                       on fewer workgroups, a whole multiple of the compute
 *                       units and at least one per compute unit);
 *   MLKV_COMBINE=fused  merge in place also when that costs up to half of
 *                       the workgroups;
 *   MLKV_WIDE=1 / 0     one eight-wave workgroup per (sequence, KV head) in
 *                       every layer below the budget / in no layer (the
 *                       default: only in re-reading layers, as above).
 * The workspace size from mlkv_workspace_bytes covers every choice.
 * Returns MLKV_ERR_* on invalid arguments. */
mlkv_status mlkv_plan(const mlkv_map* map, int layer, int batch, int capacity, int head_dim,
                      int max_len, int* workgroups, int* max_parts);
/* 1 when that plan finishes split runs with the separate merge kernel after
 * the attention kernel, 0 when the attention launch finishes every
 * (sequence, KV head) itself, -1 for invalid arguments (same arguments and
 * environment overrides as mlkv_plan). */
int mlkv_plan_merge_kernel(const mlkv_map* map, int layer, int batch, int capacity, int head_dim,
                           int max_len);

/* ----------------------------------------------------------------------- */
/* Kernel timing (benchmarks)                                                */
/* ----------------------------------------------------------------------- */

/* While enabled (on the calling thread), every split-K attention kernel that
 * mlkv_decode_attention / mlkv_decode_step launches, and every prefill
 * attention kernel of mlkv_prefill_attention / mlkv_prefill_step, is
 * bracketed by a pair of HIP events recorded on its launch stream; when a
 * separate merge kernel finishes the split runs of that attention launch, the
 * pair brackets both kernels (start with the attention dispatch, stop when
 * the merge completes), so one timed launch is a layer's whole attention.
 * Separate append kernels are outside the pair.  Up to max_launches launches
 * are recorded; later ones are not timed.  Creates the events (host call, not
 * for capture).  Errors: MLKV_ERR_INVALID_ARG (max_launches <= 0),
 * MLKV_ERR_HIP. */
mlkv_status mlkv_profile_enable(int max_launches);
/* Synchronizes on the recorded events and reports the number of timed
 * launches and the sum, minimum and maximum of their durations (ms). */
mlkv_status mlkv_profile_read(int* launches, double* total_ms, double* min_ms, double* max_ms);
/* Synchronizes on the recorded events and writes the duration (ms) of each
 * timed launch, in launch order, to ms[0 .. min(launches, capacity) - 1];
 * *count receives that number.  Errors: MLKV_ERR_INVALID_ARG (count NULL, or
 * ms NULL with capacity > 0), MLKV_ERR_HIP. */
mlkv_status mlkv_profile_durations(double* ms, int capacity, int* count);
/* Stops timing and destroys the events. */
void mlkv_profile_disable(void);
/* The floor of that timing: `reps` launches of an empty kernel with
 * `workgroups` x `threads` work-items, each bracketed by an event pair
 * recorded with its dispatch exactly as above, enqueued on `stream` back to
 * back; synchronizes and returns the median duration (ms).  What no kernel
 * timed this way can go below.  Errors: MLKV_ERR_INVALID_ARG, MLKV_ERR_HIP. */
mlkv_status mlkv_profile_launch_floor(int workgroups, int threads, int reps, hipStream_t stream,
                                      double* median_ms);
/* The achievable read rate the attention kernels are compared with: `reps`
 * back-to-back launches of a plain streaming read (every 16-byte piece of
 * the first bytes - 16 bytes of `buffer` loaded once, eight loads in flight
 * per thread, 8 workgroups of 256 per compute unit), each timed by an event
 * pair recorded with its dispatch; returns the median and the best rate in
 * GB/s.  buffer: caller-owned device memory, 16-byte aligned, at least 16 KiB;
 * its contents are not changed except, for one impossible data pattern, the
 * last 16 bytes.  A buffer several times the 256 MB Infinity Cache measures
 * HBM.  Errors: MLKV_ERR_INVALID_ARG, MLKV_ERR_ALIGNMENT, MLKV_ERR_HIP. */
mlkv_status mlkv_profile_read_bandwidth(const void* buffer, size_t bytes, int reps,
                                        hipStream_t stream, double* median_gbs, double* best_gbs);

#ifdef __cplusplus
}
#endif

#endif /* MLKV_H_ */
