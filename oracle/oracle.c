/*
 * MLKV decode-attention ORACLE — test infrastructure only.
 *
 * Plain, slow, obviously-correct CPU reference for what the decode hot path
 * computes.  Only tests/, the smoke check and the benchmark's CPU-baseline leg
 * may load it; the product path never does.  It shares no code with the HIP
 * library: no headers, no helpers, no tables.
 *
 * All arithmetic is in double precision; bf16 inputs widen exactly.
 * Tensors are in LOGICAL order (the paper's dimensions, batch-major per
 * sequence):
 *   q      [B][h][D]            query of the newest token, one layer
 *   Kc, Vc [n_kv][B][S][D]      cache of every KV head; S = row stride (capacity)
 *   k_new, v_new [B][n_kv][D]   the newest token's key/value for every KV head
 *
 * Paper: "MLKV: Multi-Layer Key-Value Heads for Memory Efficient Transformer
 * Decoding" (arXiv 2406.09297).
 *   MHA definition ......... Section 2.1, Eqs. (1)-(3)
 *   GQA grouping j ......... Section 2.3, Eq. (12)
 *   KV caching ............. Section 2.4
 *   MLKV sharing ........... Section 3, Eqs. (13)-(17); the shared head comes
 *                            from the bottom layer of its group (Figure 2)
 *   prefill ................ the cache of Section 2.4 filled from a prompt of
 *                            T tokens, causally (each token attends to the
 *                            positions up to its own)
 *   rotary embedding ....... the GPT-NeoX architecture of the Pythia models
 *                            (Section 4.2): rotate-half pairs of the first
 *                            rd channels, angle pos * base^(-2j/rd)
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - K/V of a shared head are produced once, by the lowest layer of its
 *     group, appended to the cache, and reused by the other layers.
 *   - The scale is 1/sqrt(D), D = head dimension (d_k).
 *   - The newest token attends to every cached position and to itself; no
 *     mask, window or positional bias.
 *   - Attention over zero positions yields a zero vector.
 *
 * Parity pins (tests/test_oracle.py): identity map == MHA checked against an
 * independent brute-force loop and torch SDPA; one head per layer == MQA;
 * L = 1 gives v; identical keys give mean(V); weights sum to 1; shift and
 * permutation invariance; needle tokens; Table 2 head counts; Table 1
 * cache-size ratios.  Rotary (tests/test_oracle_rope.py): identity at
 * position 0, a four-channel closed form, pair lengths kept, scores that
 * depend only on the position difference, bf16 rounding against an
 * enumeration of neighbouring bf16 values.  Prefill
 * (tests/test_oracle_prefill.py): one token equals the decode step; T tokens
 * equal T decode steps in sequence; torch SDPA with a causal mask; later
 * tokens leave earlier outputs unchanged; a two-token closed form; rows
 * appended at consecutive slots with nothing else touched.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_value(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* ------------------------------------------------------------------------ */
/* Map (Section 2.3 Eq. 12, Section 3 Eqs. 15 and 17).                       */
/* ------------------------------------------------------------------------ */

/*
 * The paper's 1-indexed formulas:
 *   query head i (1..h) of a layer uses KV group j = floor((i-1)/(h/g)) + 1,
 *   layer n (1..l) uses the KV heads of layer-group k = floor((n-1)/(l/m)) + 1.
 * Layer-group k owns g KV heads; its bottom layer (k-1)*(l/m)+1 computes them.
 * Global KV head (1-indexed) = (k-1)*g + j.  Stored 0-indexed.
 * Returns 0 on success, -1 if m does not divide l or g does not divide h.
 */
int oracle_map_uniform(int l, int h, int m, int g, int32_t* kv_of, int32_t* owner_of) {
  if (l <= 0 || h <= 0 || m <= 0 || g <= 0 || l % m != 0 || h % g != 0) return -1;
  int layers_per_group = l / m; /* l/m */
  int heads_per_kv = h / g;     /* h/g */
  for (int n = 1; n <= l; ++n) {
    int k = (n - 1) / layers_per_group + 1;
    for (int i = 1; i <= h; ++i) {
      int j = (i - 1) / heads_per_kv + 1;
      kv_of[(n - 1) * h + (i - 1)] = (k - 1) * g + (j - 1);
    }
  }
  for (int k = 1; k <= m; ++k)
    for (int j = 1; j <= g; ++j)
      owner_of[(k - 1) * g + (j - 1)] = (k - 1) * layers_per_group; /* bottom layer */
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Attention of one query head (Eqs. 2-3; Eq. 14 for the shared head).       */
/* ------------------------------------------------------------------------ */

/*
 * q [D], K [L rows of stride ld][D], V likewise.
 *   s_t = (q . K_t) / sqrt(D)
 *   alpha_t = exp(s_t - max s) / sum_u exp(s_u - max s)
 *   o = sum_t alpha_t V_t
 * Sums run in ascending t and d.  alpha (length L) is optional.
 */
void oracle_attend_one(const uint16_t* q, const uint16_t* K, const uint16_t* V, long L, long ld,
                       int D, double* o, double* alpha) {
  for (int d = 0; d < D; ++d) o[d] = 0.0;
  if (L <= 0) return;
  double* w = alpha ? alpha : (double*)malloc(sizeof(double) * (size_t)L);
  if (!w) return;
  /* scores s_t = q . K_t / sqrt(D), and their maximum */
  double scale = 1.0 / sqrt((double)D);
  double s_max = -INFINITY;
  for (long t = 0; t < L; ++t) {
    double dot = 0.0;
    for (int d = 0; d < D; ++d) dot += bf16_value(q[d]) * bf16_value(K[t * ld + d]);
    w[t] = dot * scale;
    if (w[t] > s_max) s_max = w[t];
  }
  /* unnormalised weights exp(s_t - max) and their sum Z */
  double Z = 0.0;
  for (long t = 0; t < L; ++t) {
    w[t] = exp(w[t] - s_max);
    Z += w[t];
  }
  /* o = sum_t (w_t / Z) V_t */
  for (long t = 0; t < L; ++t)
    for (int d = 0; d < D; ++d) o[d] += w[t] * bf16_value(V[t * ld + d]);
  for (int d = 0; d < D; ++d) o[d] /= Z;
  if (alpha)
    for (long t = 0; t < L; ++t) alpha[t] = w[t] / Z;
  else
    free(w);
}

/* ------------------------------------------------------------------------ */
/* One layer of decode attention (Eqs. 13-17).                               */
/* ------------------------------------------------------------------------ */

/*
 * For every sequence b and query head i of `layer`:
 *   kv = kv_of[layer][i],  L = seq_lens[b]  (clamped to [0, S])
 *   out[b][i][:] = attend(q[b][i], Kc[kv][b][0:L], Vc[kv][b][0:L])
 */
void oracle_decode_attention(int layer, int B, int h, int n_kv, int S, int D,
                             const int32_t* kv_of, const uint16_t* q, const uint16_t* Kc,
                             const uint16_t* Vc, const int32_t* seq_lens, double* out) {
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int i = 0; i < h; ++i) {
      int kv = kv_of[layer * h + i];
      long L = seq_lens[b];
      if (L < 0) L = 0;
      if (L > S) L = S;
      size_t row = ((size_t)kv * B + b) * (size_t)S * D;
      oracle_attend_one(q + ((size_t)b * h + i) * D, Kc + row, Vc + row, L, D, D,
                        out + ((size_t)b * h + i) * D, NULL);
    }
  }
  (void)n_kv;
}

/* ------------------------------------------------------------------------ */
/* Cache append (Section 2.4) in the layers that own KV heads (Section 3).   */
/* ------------------------------------------------------------------------ */

/*
 * For every KV head kv whose owner is `layer` and every sequence b with
 * 0 <= pos[b] < S:  Kc[kv][b][pos[b]] = k_new[b][kv],  Vc likewise (bit copy).
 * Returns the number of KV heads appended.
 */
int oracle_append(int layer, int B, int n_kv, int S, int D, const int32_t* owner_of,
                  uint16_t* Kc, uint16_t* Vc, const uint16_t* k_new, const uint16_t* v_new,
                  const int32_t* pos) {
  int owned = 0;
  for (int kv = 0; kv < n_kv; ++kv) {
    if (owner_of[kv] != layer) continue;
    ++owned;
    for (int b = 0; b < B; ++b) {
      if (pos[b] < 0 || pos[b] >= S) continue;
      size_t dst = (((size_t)kv * B + b) * S + pos[b]) * D;
      size_t src = ((size_t)b * n_kv + kv) * D;
      memcpy(Kc + dst, k_new + src, sizeof(uint16_t) * D);
      memcpy(Vc + dst, v_new + src, sizeof(uint16_t) * D);
    }
  }
  return owned;
}

/* ------------------------------------------------------------------------ */
/* A whole decode step: Layers(x) of Eq. 17 restricted to attention.         */
/* ------------------------------------------------------------------------ */

/*
 * for n = 0 .. l-1:
 *   append the newest token into the heads layer n owns (slot ctx[b]);
 *   attend every query head of layer n over ctx[b] + 1 positions.
 * q_all [l][B][h][D], out_all [l][B][h][D] (double).  Kc/Vc are updated.
 */
void oracle_decode_step(int l, int B, int h, int n_kv, int S, int D, const int32_t* kv_of,
                        const int32_t* owner_of, const uint16_t* q_all, uint16_t* Kc,
                        uint16_t* Vc, const uint16_t* k_new, const uint16_t* v_new,
                        const int32_t* ctx, int32_t* lens_scratch, double* out_all) {
  for (int b = 0; b < B; ++b) lens_scratch[b] = ctx[b] + 1;
  for (int n = 0; n < l; ++n) {
    oracle_append(n, B, n_kv, S, D, owner_of, Kc, Vc, k_new, v_new, ctx);
    oracle_decode_attention(n, B, h, n_kv, S, D, kv_of, q_all + (size_t)n * B * h * D, Kc, Vc,
                            lens_scratch, out_all + (size_t)n * B * h * D);
  }
}

/* ------------------------------------------------------------------------ */
/* Prefill: T new tokens of every sequence in one call.  The cache of        */
/* Section 2.4 is filled from the prompt; under MLKV (Section 3) the owning  */
/* layer stores the new keys/values and every layer of the group attends to  */
/* them.  Token t of sequence b sits at position ctx[b] + t and attends      */
/* causally: positions 0 .. ctx[b] + t (cached tokens, earlier new tokens    */
/* and itself).                                                              */
/* ------------------------------------------------------------------------ */

/*
 * For every sequence b, new token t < T and query head i of `layer`:
 *   kv = kv_of[layer][i],  L = ctx[b] + t + 1  (clamped to [0, S])
 *   out[b][t][i][:] = attend(q[b][t][i], Kc[kv][b][0:L], Vc[kv][b][0:L])
 * q [B][T][h][D], out [B][T][h][D] (double).
 */
void oracle_prefill_attention(int layer, int B, int T, int h, int n_kv, int S, int D,
                              const int32_t* kv_of, const uint16_t* q, const uint16_t* Kc,
                              const uint16_t* Vc, const int32_t* ctx, double* out) {
#pragma omp parallel for collapse(3) schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    for (int t = 0; t < T; ++t) {
      for (int i = 0; i < h; ++i) {
        int kv = kv_of[layer * h + i];
        long L = (long)ctx[b] + t + 1;
        if (L < 0) L = 0;
        if (L > S) L = S;
        size_t row = ((size_t)kv * B + b) * (size_t)S * D;
        size_t qo = (((size_t)b * T + t) * h + i) * D;
        oracle_attend_one(q + qo, Kc + row, Vc + row, L, D, D, out + qo, NULL);
      }
    }
  }
  (void)n_kv;
}

/*
 * For every KV head kv whose owner is `layer`, every b and t < T with
 * 0 <= ctx[b] + t < S:  Kc[kv][b][ctx[b] + t] = k_new[b][t][kv],  Vc likewise.
 * k_new, v_new [B][T][n_kv][D].  Returns the number of KV heads appended.
 */
int oracle_append_rows(int layer, int B, int T, int n_kv, int S, int D, const int32_t* owner_of,
                       uint16_t* Kc, uint16_t* Vc, const uint16_t* k_new, const uint16_t* v_new,
                       const int32_t* ctx) {
  int owned = 0;
  for (int kv = 0; kv < n_kv; ++kv) {
    if (owner_of[kv] != layer) continue;
    ++owned;
    for (int b = 0; b < B; ++b) {
      for (int t = 0; t < T; ++t) {
        long slot = (long)ctx[b] + t;
        if (slot < 0 || slot >= S) continue;
        size_t dst = (((size_t)kv * B + b) * S + (size_t)slot) * D;
        size_t src = (((size_t)b * T + t) * n_kv + kv) * D;
        memcpy(Kc + dst, k_new + src, sizeof(uint16_t) * D);
        memcpy(Vc + dst, v_new + src, sizeof(uint16_t) * D);
      }
    }
  }
  return owned;
}

/*
 * for n = 0 .. l-1:
 *   the heads layer n owns take the T new rows at slots ctx[b] .. ctx[b]+T-1;
 *   every query head of layer n attends causally as above.
 * q_all [l][B][T][h][D], out_all [l][B][T][h][D] (double).  Kc/Vc are updated.
 */
void oracle_prefill_step(int l, int B, int T, int h, int n_kv, int S, int D,
                         const int32_t* kv_of, const int32_t* owner_of, const uint16_t* q_all,
                         uint16_t* Kc, uint16_t* Vc, const uint16_t* k_new,
                         const uint16_t* v_new, const int32_t* ctx, double* out_all) {
  const size_t layer_elems = (size_t)B * T * h * D;
  for (int n = 0; n < l; ++n) {
    oracle_append_rows(n, B, T, n_kv, S, D, owner_of, Kc, Vc, k_new, v_new, ctx);
    oracle_prefill_attention(n, B, T, h, n_kv, S, D, kv_of, q_all + (size_t)n * layer_elems, Kc,
                             Vc, ctx, out_all + (size_t)n * layer_elems);
  }
}

/* ------------------------------------------------------------------------ */
/* Rotary position embedding of the GPT-NeoX architecture that the paper's   */
/* Pythia models use (Section 4.2).                                          */
/* ------------------------------------------------------------------------ */

/* Nearest bf16 (ties to even) of a double, as bits, by rounding the
 * significand to 8 bits directly (no intermediate float rounding). */
uint16_t oracle_bf16_from_double(double x) {
  if (x == 0.0) return signbit(x) ? 0x8000u : 0u;
  int e;
  const double m = frexp(x, &e);          /* x = m * 2^e, 0.5 <= |m| < 1 */
  const double r = nearbyint(m * 256.0);  /* 8 significant bits, ties to even */
  const float f = (float)ldexp(r, e - 8);  /* exact: r has at most 9 bits */
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (uint16_t)(u >> 16);
}

/*
 * One head vector x[0..D) at position pos.  The first rd channels (rd even)
 * form rd/2 pairs (j, j + rd/2); pair j turns by the angle
 *   theta_j = pos * base^(-2j/rd),
 *   y_j        = x_j cos(theta_j) - x_{j+rd/2} sin(theta_j)
 *   y_{j+rd/2} = x_{j+rd/2} cos(theta_j) + x_j sin(theta_j).
 * Channels rd..D-1 are copied.  Arithmetic in double, stored as bf16.
 */
void oracle_rope(const uint16_t* x, int D, int rd, double base, long pos, uint16_t* y) {
  const int half = rd / 2;
  for (int d = rd; d < D; ++d) y[d] = x[d];
  for (int j = 0; j < half; ++j) {
    const double theta = (double)pos * pow(base, -2.0 * j / rd);
    const double c = cos(theta), s = sin(theta);
    const double a = bf16_value(x[j]), b = bf16_value(x[j + half]);
    y[j] = oracle_bf16_from_double(a * c - b * s);
    y[j + half] = oracle_bf16_from_double(b * c + a * s);
  }
}

/* The double-precision rotation itself (for the invariance pins). */
void oracle_rope_f64(const double* x, int D, int rd, double base, double pos, double* y) {
  const int half = rd / 2;
  for (int d = rd; d < D; ++d) y[d] = x[d];
  for (int j = 0; j < half; ++j) {
    const double theta = pos * pow(base, -2.0 * j / rd);
    const double c = cos(theta), s = sin(theta);
    y[j] = x[j] * c - x[j + half] * s;
    y[j + half] = x[j + half] * c + x[j] * s;
  }
}

/*
 * A decode step with rotary embedding: the newest token sits at position
 * ctx[b]; its keys (for every KV head) and its queries (every layer and head)
 * are rotated at that position, then the step runs as above.  q_rot and
 * k_rot are caller scratch of the sizes of q_all and k_new.
 */
void oracle_decode_step_rope(int l, int B, int h, int n_kv, int S, int D, int rd, double base,
                             const int32_t* kv_of, const int32_t* owner_of,
                             const uint16_t* q_all, uint16_t* Kc, uint16_t* Vc,
                             const uint16_t* k_new, const uint16_t* v_new, const int32_t* ctx,
                             uint16_t* q_rot, uint16_t* k_rot, int32_t* lens_scratch,
                             double* out_all) {
  for (int n = 0; n < l; ++n)
    for (int b = 0; b < B; ++b)
      for (int i = 0; i < h; ++i) {
        const size_t off = (((size_t)n * B + b) * h + i) * D;
        oracle_rope(q_all + off, D, rd, base, ctx[b], q_rot + off);
      }
  for (int b = 0; b < B; ++b)
    for (int kv = 0; kv < n_kv; ++kv) {
      const size_t off = ((size_t)b * n_kv + kv) * D;
      oracle_rope(k_new + off, D, rd, base, ctx[b], k_rot + off);
    }
  oracle_decode_step(l, B, h, n_kv, S, D, kv_of, owner_of, q_rot, Kc, Vc, k_rot, v_new, ctx,
                     lens_scratch, out_all);
}

/* Host threads the OpenMP loops above use (n > 0 sets them); returns the
 * count in effect.  Timing only: the arithmetic does not depend on it. */
int oracle_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
}
