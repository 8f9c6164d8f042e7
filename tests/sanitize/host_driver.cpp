// Drives the C-ABI host code under AddressSanitizer / UndefinedBehaviorSanitizer
// (with the device side replaced by kernel_stubs.cpp): map construction for
// every Table 2 configuration and the 7B-like map, general-map validation,
// argument validation of every entry point, and the planning / workspace
// layout that runs before a launch (which the stubs then refuse).  Exits 0
// when every expectation holds.
#include <cstdio>
#include <cstdint>
#include <vector>

#include "mlkv.h"

static int g_failures = 0;
#define EXPECT(cond)                                                      \
  do {                                                                    \
    if (!(cond)) {                                                        \
      std::fprintf(stderr, "FAILED %s:%d: %s\n", __FILE__, __LINE__, #cond); \
      ++g_failures;                                                       \
    }                                                                     \
  } while (0)

static void* addr(uintptr_t a) { return reinterpret_cast<void*>(a); }
static const int32_t* lens(uintptr_t a) { return reinterpret_cast<const int32_t*>(a); }

static void maps() {
  // (l, h, m, g) of Table 2 (Pythia-160M variants) and the 7B-like map.
  const int cfg[][4] = {{12, 12, 12, 12}, {12, 12, 12, 4}, {12, 12, 4, 12}, {12, 12, 12, 1},
                        {12, 12, 4, 3},   {12, 12, 6, 1},  {12, 12, 4, 1},  {12, 12, 2, 1},
                        {12, 12, 1, 1},   {32, 32, 8, 8}};
  for (const auto& c : cfg) {
    mlkv_map* m = nullptr;
    EXPECT(mlkv_map_create_uniform(c[0], c[1], c[2], c[3], &m) == MLKV_OK && m);
    if (!m) continue;
    EXPECT(mlkv_map_num_kv_heads(m) == c[2] * c[3]);
    for (int n = 0; n < c[0]; ++n)
      for (int i = 0; i < c[1]; ++i) {
        const int kv = mlkv_map_kv_head(m, n, i);
        EXPECT(kv == (n / (c[0] / c[2])) * c[3] + i / (c[1] / c[3]));
        EXPECT(mlkv_map_owner_layer(m, kv) <= n);
      }
    EXPECT(mlkv_map_kv_head(m, c[0], 0) == -1 && mlkv_map_owner_layer(m, -1) == -1);
    EXPECT(mlkv_cache_bytes(m, 3, 64, 64) == 2ull * 3 * 64 * c[2] * c[3] * 64 * 2);
    mlkv_map_destroy(m);
  }
  mlkv_map* m = nullptr;
  EXPECT(mlkv_map_create_uniform(12, 12, 5, 1, &m) == MLKV_ERR_INVALID_ARG && !m);
  EXPECT(mlkv_map_create_uniform(12, 12, 4, 5, &m) == MLKV_ERR_INVALID_ARG && !m);
  EXPECT(mlkv_map_create_uniform(0, 12, 4, 1, &m) == MLKV_ERR_INVALID_ARG);
  EXPECT(mlkv_map_create_uniform(12, 12, 4, 1, nullptr) == MLKV_ERR_INVALID_ARG);
  // general maps: a valid cross-layer pattern, then rule violations
  const int32_t kv_ok[4 * 4] = {0, 0, 0, 0, 0, 0, 0, 0, 1, 1, 1, 1, 1, 1, 1, 1};
  const int32_t own_ok[2] = {0, 2};
  EXPECT(mlkv_map_create(4, 4, 2, kv_ok, own_ok, &m) == MLKV_OK && m);
  mlkv_map_destroy(m);
  const int32_t own_late[2] = {1, 2};  // head 0 read by layer 0 before its owner
  EXPECT(mlkv_map_create(4, 4, 2, kv_ok, own_late, &m) == MLKV_ERR_BAD_MAP && !m);
  const int32_t kv_bad[4 * 4] = {0, 1, 0, 1, 0, 0, 0, 0, 1, 1, 1, 1, 1, 1, 1, 1};
  EXPECT(mlkv_map_create(4, 4, 2, kv_bad, own_ok, &m) == MLKV_ERR_BAD_MAP);
  const int32_t kv_range[4 * 4] = {0, 0, 0, 0, 0, 0, 0, 0, 1, 1, 1, 1, 2, 2, 2, 2};
  EXPECT(mlkv_map_create(4, 4, 2, kv_range, own_ok, &m) == MLKV_ERR_BAD_MAP);
  const int32_t kv_unread[4 * 4] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  EXPECT(mlkv_map_create(4, 4, 2, kv_unread, own_ok, &m) == MLKV_ERR_BAD_MAP);
  EXPECT(mlkv_map_create(4, 4, 2, nullptr, own_ok, &m) == MLKV_ERR_INVALID_ARG);
  mlkv_map_destroy(nullptr);
}

static void entry_points() {
  mlkv_map* mp = nullptr;
  EXPECT(mlkv_map_create_uniform(12, 12, 4, 1, &mp) == MLKV_OK);
  const uintptr_t K = 0x100000, V = 0x200000, Q = 0x300000, LEN = 0x400000, OUT = 0x500000,
                  WS = 0x600000;
  mlkv_cache c{addr(K), addr(V), 4, 2, 64, 64};
  const size_t big = size_t(1) << 30;
  // argument errors, reported before anything else
  EXPECT(mlkv_decode_attention(0, addr(Q), &c, nullptr, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), big, nullptr) == MLKV_ERR_INVALID_ARG);
  EXPECT(mlkv_decode_attention(12, addr(Q), &c, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), big, nullptr) == MLKV_ERR_INVALID_ARG);
  EXPECT(mlkv_decode_attention(0, addr(Q + 4), &c, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), big, nullptr) == MLKV_ERR_ALIGNMENT);
  EXPECT(mlkv_decode_attention(0, addr(Q), &c, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 65,
                               addr(WS), big, nullptr) == MLKV_ERR_CAPACITY);
  mlkv_cache bad = c;
  bad.capacity = 48;
  EXPECT(mlkv_decode_attention(0, addr(Q), &bad, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), big, nullptr) == MLKV_ERR_CAPACITY);
  bad = c;
  bad.head_dim = 96;
  EXPECT(mlkv_decode_attention(0, addr(Q), &bad, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), big, nullptr) == MLKV_ERR_UNSUPPORTED);
  mlkv_cache large{addr(K), addr(V), 4, 2, 4096, 64};
  EXPECT(mlkv_decode_attention(0, addr(Q), &large, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), 16, nullptr) == MLKV_ERR_WORKSPACE);
  // valid arguments: planning and the workspace layout run, the stub refuses the launch
  EXPECT(mlkv_decode_attention(0, addr(Q), &large, mp, lens(LEN), addr(OUT), MLKV_OUT_F32, 0,
                               addr(WS), big, nullptr) == MLKV_ERR_HIP);
  EXPECT(mlkv_decode_step(addr(Q), addr(Q), addr(Q), &large, mp, lens(LEN), addr(OUT),
                          MLKV_OUT_BF16, 0, addr(WS), big, nullptr) == MLKV_ERR_HIP);
  EXPECT(mlkv_decode_step_rope(addr(Q), addr(Q), addr(Q), &large, mp, lens(LEN), 8, 1e4,
                               addr(OUT), MLKV_OUT_F32, 0, addr(WS), big, nullptr) ==
         MLKV_ERR_UNSUPPORTED);
  EXPECT(mlkv_decode_step_rope(addr(Q), addr(Q), addr(Q), &large, mp, lens(LEN), 16, 1e4,
                               addr(OUT), MLKV_OUT_F32, 0, addr(WS), 64, nullptr) ==
         MLKV_ERR_WORKSPACE);
  EXPECT(mlkv_decode_step_rope(addr(Q), addr(Q), addr(Q), &large, mp, lens(LEN), 16, 1e4,
                               addr(OUT), MLKV_OUT_F32, 0, addr(WS), big, nullptr) == MLKV_ERR_HIP);
  EXPECT(mlkv_cache_append(0, mp, &c, addr(Q), addr(Q), 64, lens(LEN), nullptr) == MLKV_ERR_HIP);
  EXPECT(mlkv_cache_append(0, mp, &c, addr(Q), addr(Q), 60, lens(LEN), nullptr) ==
         MLKV_ERR_INVALID_ARG);
  EXPECT(mlkv_cache_append(1, mp, &c, nullptr, nullptr, 0, nullptr, nullptr) == MLKV_OK);
  EXPECT(mlkv_cache_write_rows(&c, 0, 4, addr(Q), addr(Q), nullptr) == MLKV_ERR_HIP);
  EXPECT(mlkv_cache_read_rows(&c, 3, 2, addr(Q), addr(Q), nullptr) == MLKV_ERR_INVALID_ARG);
  EXPECT(mlkv_prefill_step(addr(Q), addr(Q), addr(Q), &large, mp, lens(LEN), 100, addr(OUT),
                           MLKV_OUT_F32, nullptr) == MLKV_ERR_HIP);
  EXPECT(mlkv_prefill_attention(0, addr(Q), &c, mp, lens(LEN), 65, addr(OUT), MLKV_OUT_F32,
                                nullptr) == MLKV_ERR_CAPACITY);
  EXPECT(mlkv_workspace_init(addr(WS), 4096, nullptr) == MLKV_ERR_HIP);
  // planning and workspace sizes over batches, capacities and head sizes
  for (int B : {1, 2, 7, 128, 2048, 5000})
    for (int S : {32, 96, 2112, 32800})
      for (int D : {64, 128}) {
        const size_t ws = mlkv_workspace_bytes(mp, B, S, D);
        EXPECT(mlkv_workspace_bytes_rope(mp, B, S, D, 16) >= ws + size_t(B) * 8 * 16);
        int wg = 0, parts = 0;
        for (int layer = 0; layer < 12; ++layer) {
          EXPECT(mlkv_plan(mp, layer, B, S, D, S, &wg, &parts) == MLKV_OK);
          EXPECT(wg >= 1 && parts >= 1);
          EXPECT(mlkv_plan_merge_kernel(mp, layer, B, S, D, S) >= 0);
        }
      }
  EXPECT(mlkv_plan_merge_kernel(mp, 12, 2, 64, 64, 0) == -1);
  mlkv_map_destroy(mp);
}

static void model() {
  mlkv_map* mp = nullptr;
  EXPECT(mlkv_map_create_uniform(2, 4, 1, 1, &mp) == MLKV_OK);
  mlkv_model* model = nullptr;
  std::vector<mlkv_layer_weights> w(2);
  EXPECT(mlkv_model_create(mp, 256, 256, 64, 16, 1e4, 1e-5, w.data(), &model) ==
         MLKV_ERR_INVALID_ARG && !model);
  EXPECT(mlkv_model_create(mp, 250, 256, 64, 16, 1e4, 1e-5, w.data(), &model) ==
         MLKV_ERR_INVALID_ARG);
  EXPECT(mlkv_model_create(mp, 256, 256, 96, 16, 1e4, 1e-5, w.data(), &model) ==
         MLKV_ERR_UNSUPPORTED);
  EXPECT(mlkv_model_workspace_bytes(nullptr, 2, 64) == 0);
  mlkv_map_destroy(mp);
}

int main() {
  maps();
  entry_points();
  model();
  std::printf("host driver: %d failure(s)\n", g_failures);
  return g_failures == 0 ? 0 : 1;
}
