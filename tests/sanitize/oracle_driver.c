/* Drives the oracle (oracle/oracle.c, compiled into this program) under
 * AddressSanitizer / UndefinedBehaviorSanitizer on small inputs whose cache
 * slots past each sequence's length hold NaN: any read or write outside the
 * attended rows, or of an appended row outside its slot, shows up as a
 * sanitizer report or as a NaN in an output.  Checks a few fixed facts on the
 * way: L = 1 returns v, L = 0 zeros, rotation at position 0 is the identity.
 * Exits 0 when every expectation holds. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_map_uniform(int l, int h, int m, int g, int32_t* kv_of, int32_t* owner_of);
void oracle_decode_step(int l, int B, int h, int n_kv, int S, int D, const int32_t* kv_of,
                        const int32_t* owner_of, const uint16_t* q_all, uint16_t* Kc,
                        uint16_t* Vc, const uint16_t* k_new, const uint16_t* v_new,
                        const int32_t* ctx, int32_t* lens_scratch, double* out_all);
void oracle_decode_step_rope(int l, int B, int h, int n_kv, int S, int D, int rd, double base,
                             const int32_t* kv_of, const int32_t* owner_of,
                             const uint16_t* q_all, uint16_t* Kc, uint16_t* Vc,
                             const uint16_t* k_new, const uint16_t* v_new, const int32_t* ctx,
                             uint16_t* q_rot, uint16_t* k_rot, int32_t* lens_scratch,
                             double* out_all);
void oracle_prefill_step(int l, int B, int T, int h, int n_kv, int S, int D,
                         const int32_t* kv_of, const int32_t* owner_of, const uint16_t* q_all,
                         uint16_t* Kc, uint16_t* Vc, const uint16_t* k_new,
                         const uint16_t* v_new, const int32_t* ctx, double* out_all);
void oracle_rope(const uint16_t* x, int D, int rd, double base, long pos, uint16_t* y);

static int failures = 0;
#define EXPECT(c)                                                          \
  do {                                                                     \
    if (!(c)) {                                                            \
      fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #c);      \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

static uint64_t state = 0x4D4C4B56u;
static uint16_t rnd_bf16(void) { /* bf16 values in (-2, 2), never NaN */
  state = state * 6364136223846793005ull + 1442695040888963407ull;
  const float f = (float)((double)(state >> 11) / 9007199254740992.0 * 4.0 - 2.0);
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}
static double f64(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

enum { L_ = 4, H = 4, D = 64, B = 4, S = 64 };

int main(void) {
  int32_t kv_of[L_ * H], owner_of[L_ * H];
  EXPECT(oracle_map_uniform(L_, H, 2, 2, kv_of, owner_of) == 0);
  EXPECT(oracle_map_uniform(L_, H, 3, 2, kv_of, owner_of) == -1);
  EXPECT(oracle_map_uniform(L_, H, 2, 2, kv_of, owner_of) == 0);
  const int n_kv = 4;
  const size_t plane = (size_t)n_kv * B * S * D;
  uint16_t* K = malloc(plane * 2);
  uint16_t* V = malloc(plane * 2);
  uint16_t* q = malloc((size_t)L_ * B * H * D * 2);
  uint16_t* kn = malloc((size_t)B * n_kv * D * 2);
  uint16_t* vn = malloc((size_t)B * n_kv * D * 2);
  double* out = malloc((size_t)L_ * B * H * D * sizeof(double));
  int32_t scratch[B];
  /* contexts: nothing cached (L = 1 after the append), one token, ragged, the last slot */
  const int32_t ctx[B] = {0, 1, 37, S - 1};
  for (size_t i = 0; i < plane; ++i) K[i] = V[i] = 0x7FC0; /* NaN */
  for (int kv = 0; kv < n_kv; ++kv)
    for (int b = 0; b < B; ++b)
      for (int t = 0; t < ctx[b]; ++t)
        for (int d = 0; d < D; ++d) {
          const size_t i = (((size_t)kv * B + b) * S + t) * D + d;
          K[i] = rnd_bf16();
          V[i] = rnd_bf16();
        }
  for (size_t i = 0; i < (size_t)L_ * B * H * D; ++i) q[i] = rnd_bf16();
  for (size_t i = 0; i < (size_t)B * n_kv * D; ++i) {
    kn[i] = rnd_bf16();
    vn[i] = rnd_bf16();
  }
  oracle_decode_step(L_, B, H, n_kv, S, D, kv_of, owner_of, q, K, V, kn, vn, ctx, scratch, out);
  for (size_t i = 0; i < (size_t)L_ * B * H * D; ++i) EXPECT(isfinite(out[i]));
  /* sequence 0 attends only its new token: o = v_new of the head's KV head */
  for (int n = 0; n < L_; ++n)
    for (int i = 0; i < H; ++i)
      for (int d = 0; d < D; ++d)
        EXPECT(out[(((size_t)n * B + 0) * H + i) * D + d] ==
               f64(vn[(size_t)kv_of[n * H + i] * D + d]));

  /* rotary step: at position 0 the rotation is the identity */
  uint16_t* q_rot = malloc((size_t)L_ * B * H * D * 2);
  uint16_t* k_rot = malloc((size_t)B * n_kv * D * 2);
  for (size_t i = 0; i < plane; ++i)
    if (K[i] != 0x7FC0) K[i] = rnd_bf16();
  oracle_decode_step_rope(L_, B, H, n_kv, S, D, 16, 1e4, kv_of, owner_of, q, K, V, kn, vn, ctx,
                          q_rot, k_rot, scratch, out);
  for (size_t i = 0; i < (size_t)L_ * B * H * D; ++i) EXPECT(isfinite(out[i]));
  for (int n = 0; n < L_; ++n)
    for (int i = 0; i < H * D; ++i)
      EXPECT(q_rot[((size_t)n * B) * H * D + i] == q[((size_t)n * B) * H * D + i]);
  uint16_t y[D];
  oracle_rope(q, D, D, 1e4, 0, y);
  EXPECT(memcmp(y, q, sizeof y) == 0);

  /* prefill of T = 5 tokens after the same contexts, capped below S */
  enum { T = 5 };
  const int32_t pctx[B] = {0, 1, 37, S - T};
  uint16_t* pq = malloc((size_t)L_ * B * T * H * D * 2);
  uint16_t* pk = malloc((size_t)B * T * n_kv * D * 2);
  uint16_t* pv = malloc((size_t)B * T * n_kv * D * 2);
  double* pout = malloc((size_t)L_ * B * T * H * D * sizeof(double));
  for (size_t i = 0; i < plane; ++i) K[i] = V[i] = 0x7FC0;
  for (int kv = 0; kv < n_kv; ++kv)
    for (int b = 0; b < B; ++b)
      for (int t = 0; t < pctx[b]; ++t)
        for (int d = 0; d < D; ++d) {
          const size_t i = (((size_t)kv * B + b) * S + t) * D + d;
          K[i] = rnd_bf16();
          V[i] = rnd_bf16();
        }
  for (size_t i = 0; i < (size_t)L_ * B * T * H * D; ++i) pq[i] = rnd_bf16();
  for (size_t i = 0; i < (size_t)B * T * n_kv * D; ++i) {
    pk[i] = rnd_bf16();
    pv[i] = rnd_bf16();
  }
  oracle_prefill_step(L_, B, T, H, n_kv, S, D, kv_of, owner_of, pq, K, V, pk, pv, pctx, pout);
  for (size_t i = 0; i < (size_t)L_ * B * T * H * D; ++i) EXPECT(isfinite(pout[i]));

  free(K); free(V); free(q); free(kn); free(vn); free(out); free(q_rot); free(k_rot);
  free(pq); free(pk); free(pv); free(pout);
  printf("oracle driver: %d failure(s)\n", failures);
  return failures == 0 ? 0 : 1;
}
