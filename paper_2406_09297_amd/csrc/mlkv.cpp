// C ABI of the MLKV decode library: map construction and validation, argument
// checks, split-K planning and the per-layer / per-step launch sequences.
// Every argument error is reported before any HIP call.
#include "mlkv.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include <rocblas/rocblas.h>

#include "kernels.h"

struct mlkv_map {
  int l = 0, h = 0, n_kv = 0;
  std::vector<int32_t> kv_of;     // [l*h]
  std::vector<int32_t> owner_of;  // [n_kv]
  // per layer: the KV heads read form [kv_begin, kv_begin + kv_count), G = h / kv_count
  std::vector<int> kv_begin, kv_count, group;
  // per layer: the KV heads appended form [own_begin, own_begin + own_count)
  std::vector<int> own_begin, own_count;
};

struct mlkv_model {
  const mlkv_map* map = nullptr;
  int d = 0, d_ff = 0, D = 0, dims = 0;
  float eps = 1e-5f;
  double inv_freq[mlkv::kMaxRopePairs] = {};
  std::vector<mlkv_layer_weights> layers;
  rocblas_handle blas = nullptr;
  // Packed weights of the fused path (NULL when d_ff % 32 != 0): per layer
  // the layer-in matrix [W_q | W_k | W_v | W_1] and the layer-out matrix
  // [W_o ; W_2], element offsets into `packed`.
  uint16_t* packed = nullptr;
  std::vector<size_t> in_off, out_off;
};

namespace {

thread_local std::string g_last_error;

mlkv_status fail(mlkv_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
mlkv_status fail(mlkv_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

mlkv_status ok() {
  g_last_error.clear();
  return MLKV_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

constexpr int kTileTokens = 32;

// Derive the per-layer structure of a map; returns an error message or "".
std::string analyse(mlkv_map& m) {
  const int l = m.l, h = m.h, n_kv = m.n_kv;
  m.kv_begin.assign(l, 0);
  m.kv_count.assign(l, 0);
  m.group.assign(l, 0);
  m.own_begin.assign(l, -1);
  m.own_count.assign(l, 0);
  std::vector<int> first_reader(n_kv, l);
  for (int n = 0; n < l; ++n) {
    const int32_t* row = &m.kv_of[static_cast<size_t>(n) * h];
    int lo = row[0], hi = row[0];
    for (int i = 0; i < h; ++i) {
      if (row[i] < 0 || row[i] >= n_kv) return "kv_of entry out of range";
      lo = row[i] < lo ? row[i] : lo;
      hi = row[i] > hi ? row[i] : hi;
    }
    const int c = hi - lo + 1;
    if (h % c != 0) return "a layer reads a number of KV heads that does not divide h";
    const int G = h / c;
    for (int i = 0; i < h; ++i)
      if (row[i] != lo + i / G)
        return "query heads of a layer must read KV heads kv_begin + i/(h/c) (GQA grouping)";
    m.kv_begin[n] = lo;
    m.kv_count[n] = c;
    m.group[n] = G;
    for (int kv = lo; kv <= hi; ++kv) first_reader[kv] = n < first_reader[kv] ? n : first_reader[kv];
  }
  for (int kv = 0; kv < n_kv; ++kv) {
    if (first_reader[kv] == l) return "a KV head is read by no layer";
    const int o = m.owner_of[kv];
    if (o < 0 || o >= l) return "owner_of entry out of range";
    if (o > first_reader[kv]) return "a KV head is read before its owner layer appends it";
  }
  for (int kv = 0; kv < n_kv; ++kv) {
    const int o = m.owner_of[kv];
    if (m.own_count[o] == 0) {
      m.own_begin[o] = kv;
      m.own_count[o] = 1;
    } else if (m.own_begin[o] + m.own_count[o] == kv) {
      ++m.own_count[o];
    } else {
      return "the KV heads a layer owns must be contiguous";
    }
  }
  return "";
}

mlkv_status check_map(const mlkv_map* map) {
  if (!map) return fail(MLKV_ERR_INVALID_ARG, "map is NULL");
  return MLKV_OK;
}

mlkv_status check_cache(const mlkv_cache* c, const mlkv_map* map) {
  if (!c) return fail(MLKV_ERR_INVALID_ARG, "cache is NULL");
  if (!c->k || !c->v) return fail(MLKV_ERR_INVALID_ARG, "cache planes must be non-NULL");
  if (!aligned16(c->k) || !aligned16(c->v))
    return fail(MLKV_ERR_ALIGNMENT, "cache planes must be 16-byte aligned");
  if (c->batch <= 0 || c->capacity <= 0)
    return fail(MLKV_ERR_INVALID_ARG, "cache batch and capacity must be positive");
  if (c->capacity % kTileTokens != 0)
    return fail(MLKV_ERR_CAPACITY, "cache capacity %d is not a multiple of 32", c->capacity);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(MLKV_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", c->head_dim);
  if (c->n_kv != map->n_kv)
    return fail(MLKV_ERR_INVALID_ARG, "cache has %d KV heads, map has %d", c->n_kv, map->n_kv);
  const double elems = 2.0 * c->n_kv * c->batch * static_cast<double>(c->capacity) * c->head_dim;
  if (elems > 9.0e18) return fail(MLKV_ERR_CAPACITY, "cache too large");
  return MLKV_OK;
}

int tiles_of(int len) { return (len + kTileTokens - 1) / kTileTokens; }

// Split-K plan for one layer.  The kernel cuts every (sequence, KV head)
// unit into runs of R tiles, R chosen on the device from the actual lengths
// so that all runs fit the launched workgroups.  The host picks that count:
// the device's resident capacity, capped at 128 per unit (more would only
// multiply partials to merge) and at what runs of kMinTiles tiles need,
// above the compute-unit count a whole multiple of it, but at least one per
// unit; a single unit of at most kSingleUnitTiles tiles takes one workgroup
// (no partials at all).
struct Plan {
  int n_blocks;
  int max_parts;  // bound on the runs of one unit
  int max_tiles;  // tiles of the longest sequence allowed by max_len
  int min_tiles;  // least tiles per run
  int fused;      // 1: every unit's runs are merged in place (no merge kernel)
  int waves;      // waves per attention workgroup
  int direct;     // 1: one workgroup per unit in unit order (no schedule, no workspace)
};
// Runs of at least 8 tiles (two per wave): shorter runs leave each wave one
// tile, which only its first load's latency covers, and multiply partials.
// On MI355X the whole-model step at batch 8 (12 layers of Pythia-160M
// shape, 2000 cached tokens) runs 0.244 / 0.252 / 0.251 ms per step for
// MLKV-4 / MLKV-12 / MQA-12 against 0.252 / 0.270 / 0.259 ms with runs of 4;
// the ragged and long decode batches keep their plans.
constexpr int kMinTiles = 8;
constexpr int kSingleUnitTiles = 16;
constexpr int kMaxRunsPerUnit = 128;
constexpr long kCounterSlots = 65536;  // arrival counters of a workspace
// Launches that schedule their runs on the device use at most this many
// workgroups (the schedule counts runs in 16-bit halves).
constexpr long kMaxScheduledWorkgroups = 16384;
constexpr int kFallbackResident = 768;  // 256 CUs x 3 when no device can be queried
constexpr int kWorkgroupsPerCu = 2;

long compute_units_or_fallback() {
  const long cus = mlkv::compute_units();
  return cus > 0 ? cus : kFallbackResident / 3;
}

long workgroups_for(long resident, long units, long t_max, int min_tiles) {
  long g = resident < kMaxRunsPerUnit * units ? resident : kMaxRunsPerUnit * units;
  // Runs of min_tiles tiles always fit this many workgroups: no more needed.
  const long enough = (t_max + min_tiles - 1) / min_tiles + units;
  g = g < enough ? g : enough;
  // Above the compute units, a whole multiple of them keeps their bandwidth
  // shares equal (MQA-12 at 32 sequences of 2048 tokens: 288 workgroups of
  // 8-tile runs take 135 us per cold-start step, 256 take 127 us).
  const long cus = compute_units_or_fallback();
  if (g > cus) g = g / cus * cus;
  return g > units ? g : units;
}

// Runs of a unit are merged inside the attention kernel (by the last run of
// the unit to finish) when every unit's partials fit the kernel's staging
// area: the run length floor that guarantees it must leave the workgroup
// count of the plain plan unchanged (on MI355X the in-place merge then beats
// the separate merge kernel by about a tenth of a ragged 128-sequence step).
// Otherwise a separate merge kernel runs.  MLKV_COMBINE=kernel forces the
// merge kernel; MLKV_COMBINE=fused also accepts a floor that keeps at least
// half of the workgroups.
// The attention launch's workgroup budget on the current device.  Two
// workgroups per compute unit: on MI355X fewer, longer runs beat filling
// every resident slot (fewer partials, longer pipelines), and a whole
// multiple of the compute units keeps their bandwidth shares equal.
long workgroup_budget(int head_dim) {
  long resident = mlkv::resident_workgroups(head_dim);
  if (resident <= 0) resident = kFallbackResident;
  const long cus = compute_units_or_fallback();
  if (resident > kWorkgroupsPerCu * cus) resident = kWorkgroupsPerCu * cus;
  if (const char* env = std::getenv("MLKV_WORKGROUPS")) {
    const long w = std::atol(env);
    if (w > 0) resident = w;
  }
  return resident < kMaxScheduledWorkgroups ? resident : kMaxScheduledWorkgroups;
}

Plan plan(const mlkv_map* map, int layer, int batch, int max_len, int head_dim) {
  Plan pl{};
  pl.max_tiles = tiles_of(max_len < 1 ? 1 : max_len);
  const long units = static_cast<long>(batch) * map->kv_count[layer];
  const long t_max = units * pl.max_tiles;
  const long resident = workgroup_budget(head_dim);
  pl.min_tiles = kMinTiles;
  pl.fused = 0;
  // A layer that only re-reads KV heads earlier layers of its group have
  // read gives each (sequence, KV head) unit one eight-wave workgroup (no
  // split runs, schedule or merge) when the units fill at least 3/8 of the
  // compute units: on MI355X the Infinity Cache then serves those heads,
  // and the workgroups stream them faster than balanced split runs plus the
  // merge of their partials (12-layer steps back to back: MLKV-4 at 128
  // ragged sequences 136 against 143 us, MLKV-12 at 32 sequences of 2048
  // tokens 136 against 157 us).  Owning layers, which read their heads from
  // HBM first, keep the split runs, as do maps without sharing across
  // layers.  MLKV_WIDE=0 / 1 turns this off / applies it to every layer.
  const char* wide_env = std::getenv("MLKV_WIDE");
  const int wide_mode = wide_env ? (std::atoi(wide_env) != 0 ? 1 : 0) : -1;
  const long cus = compute_units_or_fallback();
  if (wide_mode != 0 && units < resident) {
    bool rereads = true;
    for (int c = 0; c < map->kv_count[layer]; ++c)
      rereads = rereads && map->owner_of[map->kv_begin[layer] + c] < layer;
    if (wide_mode == 1 || (rereads && 8 * units >= 3 * cus)) {
      pl.n_blocks = static_cast<int>(units);
      pl.waves = mlkv::wide_waves();
      pl.min_tiles = pl.max_tiles;
      pl.direct = 1;
      pl.max_parts = 2;
      return pl;
    }
  }
  const long cap_parts = mlkv::stage_floats() / (static_cast<long>(map->group[layer]) * head_dim);
  const char* comb = std::getenv("MLKV_COMBINE");
  const bool force_kernel = comb && std::strcmp(comb, "kernel") == 0;
  const bool force_fused = comb && std::strcmp(comb, "fused") == 0;
  long budget = resident;  // workgroups this plan may use
  if (!force_kernel && cap_parts >= 2) {
    long mt = (pl.max_tiles + cap_parts - 1) / cap_parts;
    mt = mt > kMinTiles ? mt : kMinTiles;
    const long g = workgroups_for(resident, units, t_max, static_cast<int>(mt));
    const long g_plain = workgroups_for(resident, units, t_max, kMinTiles);
    bool accept = force_fused ? 2 * g >= resident || g >= units * ((pl.max_tiles + mt - 1) / mt)
                              : g >= g_plain;
    // A merge in place on fewer workgroups, at least one per compute unit
    // (a whole multiple of them), beats the full count plus the merge
    // kernel's launch: MQA-12 and MLKV-1 at batch 32, context 2048, take
    // 109 / 102 us per 12-layer step instead of 122 / 108 us.
    if (!accept && !force_fused && g >= cus) {
      accept = true;
      budget = g;
    }
    if (accept) {
      pl.min_tiles = static_cast<int>(mt);
      pl.fused = 1;
    }
  }
  long g = workgroups_for(budget, units, t_max, pl.min_tiles);
  if (units == 1 && t_max <= kSingleUnitTiles) g = 1;
  pl.waves = mlkv::default_waves();
  pl.n_blocks = static_cast<int>(g);
  if (g == units) {  // one workgroup per unit: runs cover whole units, nothing to merge
    pl.min_tiles = pl.max_tiles;
    pl.fused = 0;
    // Workgroup g is unit g, except the lone short unit of a one-sequence
    // batch, which keeps the single-workgroup path (first tiles requested
    // before its length arrives).
    pl.direct = !(g == 1 && batch == 1 && map->kv_count[layer] == 1);
  }
  pl.max_parts = (pl.max_tiles + pl.min_tiles - 1) / pl.min_tiles + 1;
  return pl;
}

// Whether launches of this plan record (or follow) a step's run items: split
// runs scheduled on the device; not a workgroup per unit or one workgroup.
bool plan_records(const Plan& pl) { return !pl.direct && pl.n_blocks > 1; }

// Layers of a step share the lengths, so a layer can follow the run items an
// earlier layer recorded exactly when both plans split the same number of KV
// heads' units the same way: equal keys.
struct PlanKey {
  int kv_count = -1, n_blocks = 0, min_tiles = 0, waves = 0, fused = 0;
  bool operator==(const PlanKey& o) const {
    return kv_count == o.kv_count && n_blocks == o.n_blocks && min_tiles == o.min_tiles &&
           waves == o.waves && fused == o.fused;
  }
};
PlanKey plan_key(const Plan& pl, int kv_count) {
  return PlanKey{kv_count, pl.n_blocks, pl.min_tiles, pl.waves, pl.fused};
}

// The work-plan bound of a call: the hint, or the capacity for a hint <= 0.
int max_len_of(const mlkv_cache* cache, int max_len_hint) {
  return max_len_hint <= 0 ? cache->capacity : max_len_hint;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workspace bytes of the rotary table of mlkv_decode_step_rope: (cos, sin)
// in double for each sequence and channel pair.
size_t rope_table_bytes(int batch, int rotary_dims) {
  if (rotary_dims <= 0) return 0;
  return align_up(static_cast<size_t>(batch) * (rotary_dims / 2) * 2 * sizeof(double), 256);
}

// Plans that schedule runs inside the kernel keep per-sequence tables in LDS,
// which bounds the batch; direct plans (a workgroup per unit) have no bound.
// The in-kernel schedule also counts all tiles of a layer in 32 bits (below
// 2^30, far above any cache that fits a device) and gives each workgroup at
// most one sequence with nothing to attend (at least one workgroup per
// sequence, which the plan always launches).
mlkv_status check_plan_batch(const Plan& pl, int batch, int kv_count) {
  if (pl.direct || pl.n_blocks <= 1) return MLKV_OK;
  if (batch > mlkv::max_batch())
    return fail(MLKV_ERR_UNSUPPORTED,
                "batch %d above %d needs one workgroup per (sequence, KV head): %d workgroups "
                "planned", batch, mlkv::max_batch(), pl.n_blocks);
  if (static_cast<long>(batch) * kv_count * pl.max_tiles >= (1L << 30))
    return fail(MLKV_ERR_UNSUPPORTED, "%d sequences x %d KV heads x %d tiles: too many tiles",
                batch, kv_count, pl.max_tiles);
  if (pl.n_blocks < batch)
    return fail(MLKV_ERR_UNSUPPORTED, "plan of %d workgroups for %d sequences", pl.n_blocks, batch);
  return MLKV_OK;
}

// Workspace layout of one call (nothing when one workgroup does all):
//   counters  int32 [kCounterSlots]  finished runs per unit, zero between calls
//   runs      int32 [batch]                          (256-byte aligned blocks)
//   plan      32-byte run items [n_blocks]            (used by mlkv_decode_step)
//   part_acc  fp32  [batch * h * max_parts][head_dim]
//   part_ml   fp32  [batch * h * max_parts][2]
// The counters are the only state a call leaves for the next one (all zero),
// so their region has the same place and size in every call's layout: calls
// with different batches or maps on one workspace never write anything else
// there.  A split plan has fewer units than workgroups and at most
// kCounterSlots workgroups, so every unit has its slot.
constexpr size_t kRunItemBytes = 32;

struct WsLayout {
  size_t counters, runs, plan, acc, ml, total;
};

WsLayout ws_layout(int batch, int h, int head_dim, const Plan& pl) {
  WsLayout w{};
  if (pl.n_blocks <= 1 || pl.direct) return w;
  const size_t rows = static_cast<size_t>(batch) * h * pl.max_parts;
  w.counters = 0;
  w.runs = static_cast<size_t>(kCounterSlots) * sizeof(int32_t);
  w.plan = w.runs + align_up(static_cast<size_t>(batch) * sizeof(int32_t), 256);
  w.acc = w.plan + align_up(static_cast<size_t>(pl.n_blocks) * kRunItemBytes, 256);
  w.ml = w.acc + align_up(rows * head_dim * sizeof(float), 256);
  w.total = w.ml + rows * 2 * sizeof(float);
  return w;
}

size_t workspace_need(int batch, int h, int head_dim, const Plan& pl) {
  return ws_layout(batch, h, head_dim, pl).total;
}

mlkv_status check_lengths_if_requested(const int32_t* lens, int batch, int offset, int limit,
                                       hipStream_t stream) {
  const char* env = std::getenv("MLKV_CHECK");
  if (!env || std::strcmp(env, "1") != 0) return MLKV_OK;
  std::vector<int32_t> host(batch);
  if (hipStreamSynchronize(stream) != hipSuccess ||
      hipMemcpy(host.data(), lens, sizeof(int32_t) * batch, hipMemcpyDeviceToHost) != hipSuccess)
    return fail(MLKV_ERR_HIP, "MLKV_CHECK: could not read lengths back");
  for (int b = 0; b < batch; ++b) {
    const long L = static_cast<long>(host[b]) + offset;
    if (L < 0 || L > limit)
      return fail(MLKV_ERR_CAPACITY, "MLKV_CHECK: sequence %d attends %ld positions, limit %d", b,
                  L, limit);
  }
  return MLKV_OK;
}

// Event pairs around attention launches (mlkv_profile_*).
struct Profile {
  std::vector<hipEvent_t> start, stop;
  int used = 0;
  bool on = false;
};
thread_local Profile g_profile;

// plan_mode: 0 = every workgroup schedules inside the attention kernel;
// 1 = the same, and each workgroup also records its run in the workspace's
// plan; 2 = follow the plan already recorded there (same lengths and launch).
// k_new/v_new (may be null): the step's new rows [B][n_kv][D]; when given,
// the kernel also appends the heads `layer` owns (all inside its read range).
mlkv_status attention_impl(int layer, const void* q, const mlkv_cache* cache, const mlkv_map* map,
                           const int32_t* lens, int len_offset, void* out, mlkv_out_dtype dt,
                           int max_len_hint, void* ws, size_t ws_bytes, hipStream_t stream,
                           int plan_mode = 0, const uint16_t* k_new = nullptr,
                           const uint16_t* v_new = nullptr, const double* rope_cs = nullptr,
                           int rope_half = 0, const mlkv::SideProduct* side = nullptr) {
  const int B = cache->batch, S = cache->capacity, D = cache->head_dim;
  const int max_len = max_len_hint <= 0 ? S : max_len_hint;
  const Plan pl = plan(map, layer, B, max_len, D);
  if (const mlkv_status bs = check_plan_batch(pl, B, map->kv_count[layer]); bs != MLKV_OK)
    return bs;
  const size_t need = workspace_need(B, map->h, D, pl);
  if (need > 0 && (!ws || ws_bytes < need))
    return fail(MLKV_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                ws ? ws_bytes : 0);
  if (need > 0 && !aligned16(ws)) return fail(MLKV_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  mlkv::AttnParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(cache->k);
  p.v = static_cast<const uint16_t*>(cache->v);
  p.lens = lens;
  p.out = out;
  const WsLayout wl = ws_layout(B, map->h, D, pl);
  char* base = static_cast<char*>(ws);
  p.counters = need ? reinterpret_cast<int*>(base + wl.counters) : nullptr;
  p.runs = need ? reinterpret_cast<int*>(base + wl.runs) : nullptr;
  p.plan = need && plan_mode == 2 ? base + wl.plan : nullptr;
  p.plan_out = need && plan_mode == 1 ? base + wl.plan : nullptr;
  p.part_acc = need ? reinterpret_cast<float*>(base + wl.acc) : nullptr;
  p.part_ml = need ? reinterpret_cast<float*>(base + wl.ml) : nullptr;
  p.B = B;
  p.h = map->h;
  p.S = S;
  p.kv_begin = map->kv_begin[layer];
  p.G = map->group[layer];
  p.n_groups = map->kv_count[layer];
  p.max_len = max_len;
  p.n_blocks = pl.n_blocks;
  p.min_tiles = pl.min_tiles;
  p.max_parts = pl.max_parts;
  p.fused = pl.fused;
  p.waves = pl.waves;
  p.direct = pl.direct;
  // One wave merges a row when units average at most 16 runs, else four;
  // the merge's first reads cover twice the average runs per unit.
  const long units = static_cast<long>(B) * map->kv_count[layer];
  p.merge_waves = pl.n_blocks <= 16L * units ? 1 : 4;
  const long avg_runs = (pl.n_blocks + units - 1) / units;
  p.merge_first = static_cast<int>(2 * avg_runs < pl.max_parts ? 2 * avg_runs : pl.max_parts);
  p.D = D;
  p.len_offset = len_offset;
  p.out_bf16 = dt == MLKV_OUT_BF16 ? 1 : 0;
  p.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  if (k_new && map->own_count[layer] > 0) {
    p.k_new = k_new;
    p.v_new = v_new;
    p.new_stride = map->n_kv * D;
    p.own_begin = map->own_begin[layer];
    p.own_count = map->own_count[layer];
  }
  p.rope_cs = rope_half > 0 ? rope_cs : nullptr;
  p.rope_half = rope_half > 0 ? rope_half : 0;
  hipError_t err = hipSuccess;
  Profile& prof = g_profile;
  const bool timed = prof.on && prof.used < static_cast<int>(prof.start.size());
  // A layer's attention is one launch, or two when split runs are merged by
  // the separate merge kernel: the timing pair then brackets both.
  const bool single_runs = pl.n_blocks == B * map->kv_count[layer];
  const bool merge_kernel = !pl.fused && !single_runs && pl.n_blocks > 1;
  hipEvent_t t0 = timed ? prof.start[prof.used] : nullptr;
  hipEvent_t t1 = timed ? prof.stop[prof.used] : nullptr;
  err = mlkv::launch_attention_main(p, D, stream, t0, merge_kernel ? nullptr : t1, side);
  if (err == hipSuccess && merge_kernel) err = mlkv::launch_attention_merge(p, D, stream, t1);
  if (err == hipSuccess && timed) ++prof.used;
  if (err != hipSuccess) return fail(MLKV_ERR_HIP, "attention launch: %s", hipGetErrorString(err));
  return MLKV_OK;
}

mlkv_status append_impl(int layer, const mlkv_map* map, const mlkv_cache* cache, const void* k_new,
                        const void* v_new, int row_stride, const int32_t* positions,
                        hipStream_t stream, const double* rope_cs = nullptr, int rope_half = 0) {
  const int owned = map->own_count[layer];
  if (owned == 0) return MLKV_OK;
  mlkv::AppendParams p{};
  p.k_new = static_cast<const uint16_t*>(k_new);
  p.v_new = static_cast<const uint16_t*>(v_new);
  p.positions = positions;
  p.k = static_cast<uint16_t*>(cache->k);
  p.v = static_cast<uint16_t*>(cache->v);
  p.B = cache->batch;
  p.S = cache->capacity;
  p.kv_begin = map->own_begin[layer];
  p.row_stride = row_stride;
  p.rope_cs = rope_half > 0 ? rope_cs : nullptr;
  p.rope_half = rope_half > 0 ? rope_half : 0;
  const hipError_t err = mlkv::launch_append(p, cache->head_dim, owned, stream);
  if (err != hipSuccess) return fail(MLKV_ERR_HIP, "append launch: %s", hipGetErrorString(err));
  return MLKV_OK;
}

mlkv_status append_rows_impl(int layer, const mlkv_map* map, const mlkv_cache* cache,
                             const void* k_new, const void* v_new, int T, int row_stride,
                             const int32_t* ctx_lens, hipStream_t stream) {
  const int owned = map->own_count[layer];
  if (owned == 0 || T == 0) return MLKV_OK;
  mlkv::AppendRowsParams p{};
  p.k_new = static_cast<const uint16_t*>(k_new);
  p.v_new = static_cast<const uint16_t*>(v_new);
  p.ctx = ctx_lens;
  p.k = static_cast<uint16_t*>(cache->k);
  p.v = static_cast<uint16_t*>(cache->v);
  p.B = cache->batch;
  p.T = T;
  p.S = cache->capacity;
  p.kv_begin = map->own_begin[layer];
  p.row_stride = row_stride;
  const hipError_t err = mlkv::launch_append_rows(p, cache->head_dim, owned, stream);
  if (err != hipSuccess) return fail(MLKV_ERR_HIP, "append launch: %s", hipGetErrorString(err));
  return MLKV_OK;
}

// Prefill shape checks shared by the entry points: 0 <= T <= capacity and the
// launch grid within its limits for every layer.
constexpr long kMaxGridY = 65535;
mlkv_status check_prefill_shape(const mlkv_map* map, const mlkv_cache* cache, int T) {
  if (T < 0 || T > cache->capacity)
    return fail(MLKV_ERR_CAPACITY, "T = %d new tokens: must be in [0, capacity %d]", T,
                cache->capacity);
  const long per_wg = mlkv::prefill_rows_per_workgroup(cache->head_dim);
  for (int n = 0; n < map->l; ++n) {
    const long blocks = (static_cast<long>(T) * map->group[n] + per_wg - 1) / per_wg;
    if (blocks > kMaxGridY)
      return fail(MLKV_ERR_UNSUPPORTED, "T * (query heads per KV head) = %ld rows: at most %ld",
                  static_cast<long>(T) * map->group[n], kMaxGridY * per_wg);
  }
  return MLKV_OK;
}

// MLKV_CHECK=1: every ctx_lens[b] in [0, capacity - T] (synchronizes).
mlkv_status check_prefill_lengths_if_requested(const int32_t* ctx, int batch, int T, int S,
                                               hipStream_t stream) {
  const char* env = std::getenv("MLKV_CHECK");
  if (!env || std::strcmp(env, "1") != 0) return MLKV_OK;
  std::vector<int32_t> host(batch);
  if (hipStreamSynchronize(stream) != hipSuccess ||
      hipMemcpy(host.data(), ctx, sizeof(int32_t) * batch, hipMemcpyDeviceToHost) != hipSuccess)
    return fail(MLKV_ERR_HIP, "MLKV_CHECK: could not read lengths back");
  for (int b = 0; b < batch; ++b)
    if (host[b] < 0 || static_cast<long>(host[b]) + T > S)
      return fail(MLKV_ERR_CAPACITY, "MLKV_CHECK: sequence %d has %d cached + %d new tokens, "
                  "capacity %d", b, host[b], T, S);
  return MLKV_OK;
}

mlkv_status prefill_impl(int layer, const void* q, const mlkv_cache* cache, const mlkv_map* map,
                         const int32_t* ctx_lens, int T, void* out, mlkv_out_dtype dt,
                         hipStream_t stream) {
  if (T == 0) return MLKV_OK;
  const int D = cache->head_dim;
  mlkv::PrefillParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(cache->k);
  p.v = static_cast<const uint16_t*>(cache->v);
  p.ctx = ctx_lens;
  p.out = out;
  p.B = cache->batch;
  p.T = T;
  p.h = map->h;
  p.S = cache->capacity;
  p.kv_begin = map->kv_begin[layer];
  p.G = map->group[layer];
  p.n_groups = map->kv_count[layer];
  p.out_bf16 = dt == MLKV_OUT_BF16 ? 1 : 0;
  p.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(D)));
  Profile& prof = g_profile;
  const bool timed = prof.on && prof.used < static_cast<int>(prof.start.size());
  const hipError_t err = mlkv::launch_prefill(p, D, stream, timed ? prof.start[prof.used] : nullptr,
                                              timed ? prof.stop[prof.used] : nullptr);
  if (err == hipSuccess && timed) ++prof.used;
  if (err != hipSuccess) return fail(MLKV_ERR_HIP, "prefill launch: %s", hipGetErrorString(err));
  return MLKV_OK;
}

mlkv_status check_group_size(const mlkv_map* map, int layer) {
  if (map->group[layer] > 16)
    return fail(MLKV_ERR_UNSUPPORTED,
                "layer %d maps %d query heads to one KV head; at most 16 are supported", layer,
                map->group[layer]);
  return MLKV_OK;
}

}  // namespace

extern "C" {

const char* mlkv_status_string(mlkv_status s) {
  switch (s) {
    case MLKV_OK: return "MLKV_OK";
    case MLKV_ERR_INVALID_ARG: return "MLKV_ERR_INVALID_ARG";
    case MLKV_ERR_BAD_MAP: return "MLKV_ERR_BAD_MAP";
    case MLKV_ERR_ALIGNMENT: return "MLKV_ERR_ALIGNMENT";
    case MLKV_ERR_UNSUPPORTED: return "MLKV_ERR_UNSUPPORTED";
    case MLKV_ERR_CAPACITY: return "MLKV_ERR_CAPACITY";
    case MLKV_ERR_WORKSPACE: return "MLKV_ERR_WORKSPACE";
    case MLKV_ERR_HIP: return "MLKV_ERR_HIP";
  }
  return "MLKV_ERR_UNKNOWN";
}

const char* mlkv_last_error(void) { return g_last_error.c_str(); }

mlkv_status mlkv_map_create_uniform(int l, int h, int m, int g, mlkv_map** out) {
  if (!out) return fail(MLKV_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (l <= 0 || h <= 0 || m <= 0 || g <= 0)
    return fail(MLKV_ERR_INVALID_ARG, "l, h, m, g must be positive");
  if (l % m != 0 || h % g != 0)
    return fail(MLKV_ERR_INVALID_ARG, "uniform map needs m | l and g | h (l=%d h=%d m=%d g=%d)", l,
                h, m, g);
  if (static_cast<long>(l) * h > (1L << 24))
    return fail(MLKV_ERR_INVALID_ARG, "too many query heads");
  mlkv_map* map = new (std::nothrow) mlkv_map;
  if (!map) return fail(MLKV_ERR_INVALID_ARG, "out of host memory");
  map->l = l;
  map->h = h;
  map->n_kv = m * g;
  map->kv_of.resize(static_cast<size_t>(l) * h);
  map->owner_of.resize(map->n_kv);
  const int layers_per_group = l / m, heads_per_kv = h / g;
  for (int n = 0; n < l; ++n)
    for (int i = 0; i < h; ++i)
      map->kv_of[static_cast<size_t>(n) * h + i] = (n / layers_per_group) * g + i / heads_per_kv;
  for (int kv = 0; kv < map->n_kv; ++kv) map->owner_of[kv] = (kv / g) * layers_per_group;
  const std::string err = analyse(*map);
  if (!err.empty()) {
    delete map;
    return fail(MLKV_ERR_BAD_MAP, "%s", err.c_str());
  }
  *out = map;
  return ok();
}

mlkv_status mlkv_map_create(int l, int h, int n_kv, const int32_t* kv_of, const int32_t* owner_of,
                            mlkv_map** out) {
  if (!out) return fail(MLKV_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (l <= 0 || h <= 0 || n_kv <= 0) return fail(MLKV_ERR_INVALID_ARG, "l, h, n_kv must be positive");
  if (!kv_of || !owner_of) return fail(MLKV_ERR_INVALID_ARG, "kv_of and owner_of must be non-NULL");
  if (static_cast<long>(l) * h > (1L << 24))
    return fail(MLKV_ERR_INVALID_ARG, "too many query heads");
  mlkv_map* map = new (std::nothrow) mlkv_map;
  if (!map) return fail(MLKV_ERR_INVALID_ARG, "out of host memory");
  map->l = l;
  map->h = h;
  map->n_kv = n_kv;
  map->kv_of.assign(kv_of, kv_of + static_cast<size_t>(l) * h);
  map->owner_of.assign(owner_of, owner_of + n_kv);
  const std::string err = analyse(*map);
  if (!err.empty()) {
    delete map;
    return fail(MLKV_ERR_BAD_MAP, "%s", err.c_str());
  }
  *out = map;
  return ok();
}

void mlkv_map_destroy(mlkv_map* map) { delete map; }

int mlkv_map_num_layers(const mlkv_map* map) { return map ? map->l : -1; }
int mlkv_map_num_q_heads(const mlkv_map* map) { return map ? map->h : -1; }
int mlkv_map_num_kv_heads(const mlkv_map* map) { return map ? map->n_kv : -1; }

int mlkv_map_kv_head(const mlkv_map* map, int layer, int q_head) {
  if (!map || layer < 0 || layer >= map->l || q_head < 0 || q_head >= map->h) return -1;
  return map->kv_of[static_cast<size_t>(layer) * map->h + q_head];
}

int mlkv_map_owner_layer(const mlkv_map* map, int kv) {
  if (!map || kv < 0 || kv >= map->n_kv) return -1;
  return map->owner_of[kv];
}

int mlkv_map_layer_kv_count(const mlkv_map* map, int layer) {
  if (!map || layer < 0 || layer >= map->l) return -1;
  return map->kv_count[layer];
}

int mlkv_map_layer_owned_count(const mlkv_map* map, int layer) {
  if (!map || layer < 0 || layer >= map->l) return -1;
  return map->own_count[layer];
}

int mlkv_map_layer_owned_begin(const mlkv_map* map, int layer) {
  if (!map || layer < 0 || layer >= map->l) return -1;
  return map->own_begin[layer];
}

size_t mlkv_cache_bytes(const mlkv_map* map, int batch, int capacity, int head_dim) {
  if (!map || batch <= 0 || capacity <= 0 || head_dim <= 0) return 0;
  return 2ull * static_cast<size_t>(batch) * capacity * map->n_kv * head_dim * 2ull;
}

size_t mlkv_workspace_bytes(const mlkv_map* map, int batch, int capacity, int head_dim) {
  if (!map || batch <= 0 || capacity <= 0 || (head_dim != 64 && head_dim != 128)) return 0;
  size_t best = 0;
  const long budget = workgroup_budget(head_dim);
  for (int n = 0; n < map->l; ++n) {
    // At least as many units as the device's workgroup budget: every plan is
    // one workgroup per unit, which needs no workspace.
    const long units = static_cast<long>(batch) * map->kv_count[n];
    if (units > 1 && units >= budget) continue;
    // Otherwise the largest plan any launch layout can pick: the most
    // workgroups (kMaxRunsPerUnit per unit) and the shortest runs (kMinTiles).
    Plan pl{};
    pl.max_tiles = tiles_of(capacity);
    pl.min_tiles = kMinTiles;
    pl.max_parts = (pl.max_tiles + kMinTiles - 1) / kMinTiles + 1;
    pl.n_blocks = kMaxRunsPerUnit * batch * map->kv_count[n];
    pl.n_blocks = pl.n_blocks > 2 ? pl.n_blocks : 2;
    const size_t need = workspace_need(batch, map->h, head_dim, pl);
    best = need > best ? need : best;
  }
  return best;
}

size_t mlkv_workspace_bytes_rope(const mlkv_map* map, int batch, int capacity, int head_dim,
                                 int rotary_dims) {
  if (!map || batch <= 0 || capacity <= 0 || (head_dim != 64 && head_dim != 128) ||
      rotary_dims < 0 || rotary_dims > head_dim || rotary_dims % 16 != 0)
    return 0;
  return rope_table_bytes(batch, rotary_dims) +
         mlkv_workspace_bytes(map, batch, capacity, head_dim);
}

mlkv_status mlkv_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!workspace && workspace_bytes > 0) return fail(MLKV_ERR_INVALID_ARG, "workspace is NULL");
  if (workspace_bytes == 0) return ok();
  if (!aligned16(workspace)) return fail(MLKV_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  const hipError_t err = mlkv::launch_fill(static_cast<uint32_t*>(workspace), workspace_bytes / 4,
                                           0u, stream);
  if (err != hipSuccess) return fail(MLKV_ERR_HIP, "fill launch: %s", hipGetErrorString(err));
  return ok();
}

mlkv_status mlkv_plan(const mlkv_map* map, int layer, int batch, int capacity, int head_dim,
                      int max_len, int* workgroups, int* max_parts) {
  if (check_map(map) != MLKV_OK) return MLKV_ERR_INVALID_ARG;
  if (layer < 0 || layer >= map->l) return fail(MLKV_ERR_INVALID_ARG, "layer out of range");
  if (batch <= 0 || capacity <= 0 || !workgroups || !max_parts)
    return fail(MLKV_ERR_INVALID_ARG, "bad arguments");
  if (head_dim != 64 && head_dim != 128) return fail(MLKV_ERR_UNSUPPORTED, "head_dim");
  if (max_len <= 0) max_len = capacity;
  if (max_len > capacity) return fail(MLKV_ERR_CAPACITY, "max_len above capacity");
  const Plan pl = plan(map, layer, batch, max_len, head_dim);
  *workgroups = pl.n_blocks;
  *max_parts = pl.max_parts;
  return ok();
}

int mlkv_plan_merge_kernel(const mlkv_map* map, int layer, int batch, int capacity, int head_dim,
                           int max_len) {
  if (!map || layer < 0 || layer >= map->l || batch <= 0 || capacity <= 0 ||
      (head_dim != 64 && head_dim != 128) || max_len > capacity)
    return -1;
  if (max_len <= 0) max_len = capacity;
  const Plan pl = plan(map, layer, batch, max_len, head_dim);
  const bool single_runs = pl.n_blocks == batch * map->kv_count[layer];
  return !pl.fused && !single_runs && pl.n_blocks > 1 ? 1 : 0;
}

mlkv_status mlkv_cache_append(int layer, const mlkv_map* map, const mlkv_cache* cache,
                              const void* k_new, const void* v_new, int new_row_stride,
                              const int32_t* positions, hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if (layer < 0 || layer >= map->l) return fail(MLKV_ERR_INVALID_ARG, "layer %d out of range", layer);
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  const int owned = map->own_count[layer];
  if (owned == 0) return ok();
  if (!k_new || !v_new || !positions)
    return fail(MLKV_ERR_INVALID_ARG, "k_new, v_new and positions must be non-NULL");
  if (!aligned16(k_new) || !aligned16(v_new))
    return fail(MLKV_ERR_ALIGNMENT, "k_new and v_new must be 16-byte aligned");
  if (!aligned4(positions)) return fail(MLKV_ERR_ALIGNMENT, "positions must be 4-byte aligned");
  if (new_row_stride % 8 != 0 || new_row_stride < owned * cache->head_dim)
    return fail(MLKV_ERR_INVALID_ARG, "new_row_stride %d must be a multiple of 8 and >= %d",
                new_row_stride, owned * cache->head_dim);
  if ((s = append_impl(layer, map, cache, k_new, v_new, new_row_stride, positions, stream)) !=
      MLKV_OK)
    return s;
  return ok();
}

namespace {

mlkv_status cache_rows(const mlkv_cache* cache, int kv_begin, int kv_count, const void* k_rows,
                       const void* v_rows, int to_cache, hipStream_t stream) {
  if (!cache) return fail(MLKV_ERR_INVALID_ARG, "cache is NULL");
  if (!cache->k || !cache->v) return fail(MLKV_ERR_INVALID_ARG, "cache planes must be non-NULL");
  if (!aligned16(cache->k) || !aligned16(cache->v))
    return fail(MLKV_ERR_ALIGNMENT, "cache planes must be 16-byte aligned");
  if (cache->batch <= 0 || cache->capacity <= 0 || cache->n_kv <= 0)
    return fail(MLKV_ERR_INVALID_ARG, "cache n_kv, batch and capacity must be positive");
  if (cache->capacity % kTileTokens != 0)
    return fail(MLKV_ERR_CAPACITY, "cache capacity %d is not a multiple of 32", cache->capacity);
  if (cache->head_dim != 64 && cache->head_dim != 128)
    return fail(MLKV_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", cache->head_dim);
  if (kv_begin < 0 || kv_count < 0 || kv_begin + static_cast<long>(kv_count) > cache->n_kv)
    return fail(MLKV_ERR_INVALID_ARG, "KV heads [%d, %d + %d) outside [0, %d)", kv_begin, kv_begin,
                kv_count, cache->n_kv);
  if (kv_count == 0) return ok();
  if (!k_rows || !v_rows) return fail(MLKV_ERR_INVALID_ARG, "k_rows and v_rows must be non-NULL");
  if (!aligned16(k_rows) || !aligned16(v_rows))
    return fail(MLKV_ERR_ALIGNMENT, "k_rows and v_rows must be 16-byte aligned");
  const double blocks = static_cast<double>(kv_count) * cache->batch * (cache->capacity / 32);
  if (blocks >= 2147483647.0)
    return fail(MLKV_ERR_CAPACITY, "more than 2^31 - 1 blocks of 32 tokens in one call");
  mlkv::CacheRowsParams p{};
  p.k_plane = static_cast<uint16_t*>(cache->k);
  p.v_plane = static_cast<uint16_t*>(cache->v);
  p.k_rows = static_cast<uint16_t*>(const_cast<void*>(k_rows));
  p.v_rows = static_cast<uint16_t*>(const_cast<void*>(v_rows));
  p.B = cache->batch;
  p.S = cache->capacity;
  p.kv_begin = kv_begin;
  p.kv_count = kv_count;
  p.to_cache = to_cache;
  const hipError_t err = mlkv::launch_cache_rows(p, cache->head_dim, stream);
  if (err != hipSuccess) return fail(MLKV_ERR_HIP, "cache rows launch: %s", hipGetErrorString(err));
  return ok();
}

}  // namespace

mlkv_status mlkv_cache_write_rows(const mlkv_cache* cache, int kv_begin, int kv_count,
                                  const void* k_rows, const void* v_rows, hipStream_t stream) {
  return cache_rows(cache, kv_begin, kv_count, k_rows, v_rows, 1, stream);
}

mlkv_status mlkv_cache_read_rows(const mlkv_cache* cache, int kv_begin, int kv_count,
                                 void* k_rows, void* v_rows, hipStream_t stream) {
  return cache_rows(cache, kv_begin, kv_count, k_rows, v_rows, 0, stream);
}

mlkv_status mlkv_decode_attention(int layer, const void* q, const mlkv_cache* cache,
                                  const mlkv_map* map, const int32_t* seq_lens, void* out,
                                  mlkv_out_dtype out_dtype, int max_len_hint, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if (layer < 0 || layer >= map->l) return fail(MLKV_ERR_INVALID_ARG, "layer %d out of range", layer);
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  if ((s = check_group_size(map, layer)) != MLKV_OK) return s;
  if (!q || !seq_lens || !out) return fail(MLKV_ERR_INVALID_ARG, "q, seq_lens, out must be non-NULL");
  if (!aligned16(q) || !aligned16(out)) return fail(MLKV_ERR_ALIGNMENT, "q and out must be 16-byte aligned");
  if (!aligned4(seq_lens)) return fail(MLKV_ERR_ALIGNMENT, "seq_lens must be 4-byte aligned");
  if (out_dtype != MLKV_OUT_F32 && out_dtype != MLKV_OUT_BF16)
    return fail(MLKV_ERR_INVALID_ARG, "bad out_dtype");
  if (max_len_hint > cache->capacity)
    return fail(MLKV_ERR_CAPACITY, "max_len_hint %d above capacity %d", max_len_hint,
                cache->capacity);
  const int limit = max_len_hint <= 0 ? cache->capacity : max_len_hint;
  if ((s = check_lengths_if_requested(seq_lens, cache->batch, 0, limit, stream)) != MLKV_OK) return s;
  if ((s = attention_impl(layer, q, cache, map, seq_lens, 0, out, out_dtype, max_len_hint,
                          workspace, workspace_bytes, stream)) != MLKV_OK)
    return s;
  return ok();
}

namespace {

// Argument checks of a decode step, done before anything is launched.
mlkv_status decode_step_check(const void* q_all, const void* k_new_all, const void* v_new_all,
                              const mlkv_cache* cache, const mlkv_map* map,
                              const int32_t* ctx_lens, void* out_all, mlkv_out_dtype out_dtype,
                              int max_len_hint, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  for (int n = 0; n < map->l; ++n)
    if ((s = check_group_size(map, n)) != MLKV_OK) return s;
  if (!q_all || !k_new_all || !v_new_all || !ctx_lens || !out_all)
    return fail(MLKV_ERR_INVALID_ARG, "q_all, k_new_all, v_new_all, ctx_lens, out_all must be non-NULL");
  if (!aligned16(q_all) || !aligned16(k_new_all) || !aligned16(v_new_all) || !aligned16(out_all))
    return fail(MLKV_ERR_ALIGNMENT, "q_all, k/v_new_all and out_all must be 16-byte aligned");
  if (!aligned4(ctx_lens)) return fail(MLKV_ERR_ALIGNMENT, "ctx_lens must be 4-byte aligned");
  if (out_dtype != MLKV_OUT_F32 && out_dtype != MLKV_OUT_BF16)
    return fail(MLKV_ERR_INVALID_ARG, "bad out_dtype");
  if (max_len_hint > cache->capacity)
    return fail(MLKV_ERR_CAPACITY, "max_len_hint %d above capacity %d", max_len_hint,
                cache->capacity);
  const int B = cache->batch, h = map->h, D = cache->head_dim;
  // Workspace check up front so that no layer is half-launched.
  {
    const int max_len = max_len_hint <= 0 ? cache->capacity : max_len_hint;
    for (int n = 0; n < map->l; ++n) {
      const Plan pl = plan(map, n, B, max_len, D);
      if ((s = check_plan_batch(pl, B, map->kv_count[n])) != MLKV_OK) return s;
      const size_t need = workspace_need(B, h, D, pl);
      if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(MLKV_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : 0);
    }
    if (workspace && !aligned16(workspace))
      return fail(MLKV_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  }
  const int limit = (max_len_hint <= 0 ? cache->capacity : max_len_hint);
  if ((s = check_lengths_if_requested(ctx_lens, B, 1, limit, stream)) != MLKV_OK) return s;
  return MLKV_OK;
}

// The step's launches: per layer, the append it owns (when not fused) and
// its attention.
mlkv_status decode_step_launch(const void* q_all, const void* k_new_all, const void* v_new_all,
                               const mlkv_cache* cache, const mlkv_map* map,
                               const int32_t* ctx_lens, void* out_all, mlkv_out_dtype out_dtype,
                               int max_len_hint, void* workspace, size_t workspace_bytes,
                               hipStream_t stream, const double* rope_cs = nullptr,
                               int rope_half = 0) {
  mlkv_status s;
  const int B = cache->batch, h = map->h, D = cache->head_dim, n_kv = map->n_kv;
  const size_t layer_elems = static_cast<size_t>(B) * h * D;
  const size_t out_elem_bytes = out_dtype == MLKV_OUT_BF16 ? 2 : 4;
  const uint16_t* k_new = static_cast<const uint16_t*>(k_new_all);
  const uint16_t* v_new = static_cast<const uint16_t*>(v_new_all);
  PlanKey planned_key;
  for (int n = 0; n < map->l; ++n) {
    // The attention launch appends the heads the layer owns when it reads
    // them all; otherwise a separate append runs first.
    const bool fused_append = map->own_count[n] > 0 && map->own_begin[n] >= map->kv_begin[n] &&
                              map->own_begin[n] + map->own_count[n] <=
                                  map->kv_begin[n] + map->kv_count[n];
    if (map->own_count[n] > 0 && !fused_append) {
      const size_t col = static_cast<size_t>(map->own_begin[n]) * D;
      if ((s = append_impl(n, map, cache, k_new + col, v_new + col, n_kv * D, ctx_lens, stream,
                           rope_cs, rope_half)) != MLKV_OK)
        return s;
    }
    const void* q = static_cast<const uint16_t*>(q_all) + layer_elems * n;
    void* out = static_cast<char*>(out_all) + layer_elems * out_elem_bytes * n;
    // One recorded plan serves every later layer whose plan has the same
    // key; layers with a workgroup per unit record and follow nothing.
    const Plan pl = plan(map, n, B, max_len_of(cache, max_len_hint), D);
    const bool records = plan_records(pl);
    const PlanKey key = plan_key(pl, map->kv_count[n]);
    const int mode = !records ? 0 : key == planned_key ? 2 : 1;
    if ((s = attention_impl(n, q, cache, map, ctx_lens, 1, out, out_dtype, max_len_hint, workspace,
                            workspace_bytes, stream, mode, fused_append ? k_new : nullptr,
                            fused_append ? v_new : nullptr, rope_cs, rope_half)) != MLKV_OK)
      return s;
    if (records) planned_key = key;
  }
  return ok();
}

}  // namespace

mlkv_status mlkv_decode_step(const void* q_all, const void* k_new_all, const void* v_new_all,
                             const mlkv_cache* cache, const mlkv_map* map, const int32_t* ctx_lens,
                             void* out_all, mlkv_out_dtype out_dtype, int max_len_hint,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const mlkv_status s =
      decode_step_check(q_all, k_new_all, v_new_all, cache, map, ctx_lens, out_all, out_dtype,
                        max_len_hint, workspace, workspace_bytes, stream);
  if (s != MLKV_OK) return s;
  return decode_step_launch(q_all, k_new_all, v_new_all, cache, map, ctx_lens, out_all, out_dtype,
                            max_len_hint, workspace, workspace_bytes, stream);
}

mlkv_status mlkv_decode_step_noalloc(const void* q_all, const void* k_new_all,
                                     const void* v_new_all, const mlkv_cache* cache,
                                     const mlkv_map* map, const int32_t* ctx_lens, void* out_all,
                                     mlkv_out_dtype out_dtype, int max_len_hint,
                                     hipStream_t stream) {
  // Every argument, and the step's need against the scratch's fixed size,
  // is checked before the scratch is looked up or anything is launched.
  // decode_step_check only compares pointers and sizes: the address below
  // stands in for the scratch until its device address is known.
  void* const stand_in = reinterpret_cast<void*>(uintptr_t(256));
  mlkv_status s = decode_step_check(q_all, k_new_all, v_new_all, cache, map, ctx_lens, out_all,
                                    out_dtype, max_len_hint, stand_in, mlkv::kScratchBytes,
                                    stream);
  if (s != MLKV_OK) {
    if (s == MLKV_ERR_WORKSPACE)
      return fail(MLKV_ERR_WORKSPACE, "this step needs more than the library's %zu-byte static "
                  "scratch (%s); use mlkv_decode_step with a workspace",
                  mlkv::kScratchBytes, g_last_error.c_str());
    return s;
  }
  void* scratch = nullptr;
  const hipError_t err = mlkv::scratch_for_current_device(stream, &scratch);
  if (err != hipSuccess)
    return fail(MLKV_ERR_HIP, "static scratch set-up: %s", hipGetErrorString(err));
  return decode_step_launch(q_all, k_new_all, v_new_all, cache, map, ctx_lens, out_all, out_dtype,
                            max_len_hint, scratch, mlkv::kScratchBytes, stream);
}

mlkv_status mlkv_decode_step_rope(const void* q_all, const void* k_new_all, const void* v_new_all,
                                  const mlkv_cache* cache, const mlkv_map* map,
                                  const int32_t* ctx_lens, int rotary_dims, double rotary_base,
                                  void* out_all, mlkv_out_dtype out_dtype, int max_len_hint,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  if (rotary_dims < 0 || rotary_dims > cache->head_dim || rotary_dims % 16 != 0)
    return fail(MLKV_ERR_UNSUPPORTED, "rotary_dims %d: a multiple of 16 in [0, head_dim] required",
                rotary_dims);
  if (!(rotary_base > 0.0) || !std::isfinite(rotary_base))
    return fail(MLKV_ERR_INVALID_ARG, "rotary_base must be positive and finite");
  // The rotary table heads the workspace; the decode workspace follows it.
  const size_t table = rope_table_bytes(cache->batch, rotary_dims);
  if (table > 0 && (!workspace || workspace_bytes < table))
    return fail(MLKV_ERR_WORKSPACE, "workspace of at least %zu bytes needed for the rotary table, "
                "%zu given", table, workspace ? workspace_bytes : 0);
  if (table > 0 && !aligned16(workspace))
    return fail(MLKV_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  void* ws = table > 0 ? static_cast<char*>(workspace) + table : workspace;
  const size_t ws_bytes = table > 0 ? workspace_bytes - table : workspace_bytes;
  if ((s = decode_step_check(q_all, k_new_all, v_new_all, cache, map, ctx_lens, out_all, out_dtype,
                             max_len_hint, ws, ws_bytes, stream)) != MLKV_OK)
    return s;
  const int half = rotary_dims / 2;
  double* cs = static_cast<double*>(workspace);
  if (half > 0) {
    mlkv::RopeTableParams p{};
    p.pos = ctx_lens;
    p.cs = cs;
    p.B = cache->batch;
    p.half = half;
    for (int j = 0; j < half; ++j) p.inv_freq[j] = std::pow(rotary_base, -2.0 * j / rotary_dims);
    const hipError_t err = mlkv::launch_rope_table(p, stream);
    if (err != hipSuccess) return fail(MLKV_ERR_HIP, "rotary table launch: %s", hipGetErrorString(err));
  }
  return decode_step_launch(q_all, k_new_all, v_new_all, cache, map, ctx_lens, out_all, out_dtype,
                            max_len_hint, ws, ws_bytes, stream, half > 0 ? cs : nullptr, half);
}

mlkv_status mlkv_cache_append_rows(int layer, const mlkv_map* map, const mlkv_cache* cache,
                                   const void* k_new, const void* v_new, int T,
                                   int new_row_stride, const int32_t* ctx_lens,
                                   hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if (layer < 0 || layer >= map->l) return fail(MLKV_ERR_INVALID_ARG, "layer %d out of range", layer);
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  if ((s = check_prefill_shape(map, cache, T)) != MLKV_OK) return s;
  const int owned = map->own_count[layer];
  if (owned == 0 || T == 0) return ok();
  if (!k_new || !v_new || !ctx_lens)
    return fail(MLKV_ERR_INVALID_ARG, "k_new, v_new and ctx_lens must be non-NULL");
  if (!aligned16(k_new) || !aligned16(v_new))
    return fail(MLKV_ERR_ALIGNMENT, "k_new and v_new must be 16-byte aligned");
  if (!aligned4(ctx_lens)) return fail(MLKV_ERR_ALIGNMENT, "ctx_lens must be 4-byte aligned");
  if (new_row_stride % 8 != 0 || new_row_stride < owned * cache->head_dim)
    return fail(MLKV_ERR_INVALID_ARG, "new_row_stride %d must be a multiple of 8 and >= %d",
                new_row_stride, owned * cache->head_dim);
  if ((s = check_prefill_lengths_if_requested(ctx_lens, cache->batch, T, cache->capacity,
                                              stream)) != MLKV_OK)
    return s;
  if ((s = append_rows_impl(layer, map, cache, k_new, v_new, T, new_row_stride, ctx_lens,
                            stream)) != MLKV_OK)
    return s;
  return ok();
}

mlkv_status mlkv_prefill_attention(int layer, const void* q, const mlkv_cache* cache,
                                   const mlkv_map* map, const int32_t* ctx_lens, int T, void* out,
                                   mlkv_out_dtype out_dtype, hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if (layer < 0 || layer >= map->l) return fail(MLKV_ERR_INVALID_ARG, "layer %d out of range", layer);
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  if ((s = check_prefill_shape(map, cache, T)) != MLKV_OK) return s;
  if (!q || !ctx_lens || !out) return fail(MLKV_ERR_INVALID_ARG, "q, ctx_lens, out must be non-NULL");
  if (!aligned16(q) || !aligned16(out)) return fail(MLKV_ERR_ALIGNMENT, "q and out must be 16-byte aligned");
  if (!aligned4(ctx_lens)) return fail(MLKV_ERR_ALIGNMENT, "ctx_lens must be 4-byte aligned");
  if (out_dtype != MLKV_OUT_F32 && out_dtype != MLKV_OUT_BF16)
    return fail(MLKV_ERR_INVALID_ARG, "bad out_dtype");
  if ((s = check_prefill_lengths_if_requested(ctx_lens, cache->batch, T, cache->capacity,
                                              stream)) != MLKV_OK)
    return s;
  if ((s = prefill_impl(layer, q, cache, map, ctx_lens, T, out, out_dtype, stream)) != MLKV_OK)
    return s;
  return ok();
}

mlkv_status mlkv_prefill_step(const void* q_all, const void* k_new_all, const void* v_new_all,
                              const mlkv_cache* cache, const mlkv_map* map,
                              const int32_t* ctx_lens, int T, void* out_all,
                              mlkv_out_dtype out_dtype, hipStream_t stream) {
  mlkv_status s;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  if ((s = check_prefill_shape(map, cache, T)) != MLKV_OK) return s;
  if (!q_all || !k_new_all || !v_new_all || !ctx_lens || !out_all)
    return fail(MLKV_ERR_INVALID_ARG, "q_all, k_new_all, v_new_all, ctx_lens, out_all must be non-NULL");
  if (!aligned16(q_all) || !aligned16(k_new_all) || !aligned16(v_new_all) || !aligned16(out_all))
    return fail(MLKV_ERR_ALIGNMENT, "q_all, k/v_new_all and out_all must be 16-byte aligned");
  if (!aligned4(ctx_lens)) return fail(MLKV_ERR_ALIGNMENT, "ctx_lens must be 4-byte aligned");
  if (out_dtype != MLKV_OUT_F32 && out_dtype != MLKV_OUT_BF16)
    return fail(MLKV_ERR_INVALID_ARG, "bad out_dtype");
  if ((s = check_prefill_lengths_if_requested(ctx_lens, cache->batch, T, cache->capacity,
                                              stream)) != MLKV_OK)
    return s;
  const int B = cache->batch, h = map->h, D = cache->head_dim, n_kv = map->n_kv;
  const size_t layer_elems = static_cast<size_t>(B) * T * h * D;
  const size_t out_elem_bytes = out_dtype == MLKV_OUT_BF16 ? 2 : 4;
  const uint16_t* k_new = static_cast<const uint16_t*>(k_new_all);
  const uint16_t* v_new = static_cast<const uint16_t*>(v_new_all);
  for (int n = 0; n < map->l; ++n) {
    if (map->own_count[n] > 0) {
      const size_t col = static_cast<size_t>(map->own_begin[n]) * D;
      if ((s = append_rows_impl(n, map, cache, k_new + col, v_new + col, T, n_kv * D, ctx_lens,
                                stream)) != MLKV_OK)
        return s;
    }
    const void* q = static_cast<const uint16_t*>(q_all) + layer_elems * n;
    void* out = static_cast<char*>(out_all) + layer_elems * out_elem_bytes * n;
    if ((s = prefill_impl(n, q, cache, map, ctx_lens, T, out, out_dtype, stream)) != MLKV_OK)
      return s;
  }
  return ok();
}

// ---------------------------------------------------------------------------
// Model-level decode step
// ---------------------------------------------------------------------------

namespace {

// Workspace of a model step: intermediate rows, then the attention workspace.
struct ModelWs {
  size_t h1, h2, q32, k32, v32, q16, k16, v16, o16, a32, f32, f16, m32, attn, attn_bytes, total;
};

ModelWs model_ws(const mlkv_model* m, int B, int S) {
  ModelWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  const size_t b = static_cast<size_t>(B), d = m->d, hD = static_cast<size_t>(m->map->h) * m->D;
  const size_t kvD = static_cast<size_t>(m->map->n_kv) * m->D, ff = m->d_ff;
  w.h1 = take(b * d * 2);
  w.h2 = take(b * d * 2);
  w.q32 = take(b * hD * 4);
  w.k32 = take(b * kvD * 4);
  w.v32 = take(b * kvD * 4);
  w.q16 = take(b * hD * 2);
  w.k16 = take(b * kvD * 2);
  w.v16 = take(b * kvD * 2);
  w.o16 = take(b * hD * 2);
  w.a32 = take(b * d * 4);
  w.f32 = take(b * ff * 4);
  w.f16 = take(b * ff * 2);
  w.m32 = take(b * d * 4);
  w.attn = off;
  w.attn_bytes = mlkv_workspace_bytes(m->map, B, S, m->D);
  w.total = off + w.attn_bytes;
  return w;
}

// Y[rows][n] (fp32, row stride ldy) = X[rows][k] (bf16, row stride ldx) * W[k][n]
// (bf16, row-major): the column-major product Y^T = W^T X^T.
mlkv_status gemm(rocblas_handle h, int rows, int n, int k, const void* X, int ldx, const void* W,
                 float* Y, int ldy) {
  const float one = 1.f, zero = 0.f;
  const rocblas_status st = rocblas_gemm_ex(
      h, rocblas_operation_none, rocblas_operation_none, n, rows, k, &one, W,
      rocblas_datatype_bf16_r, n, X, rocblas_datatype_bf16_r, ldx, &zero, Y,
      rocblas_datatype_f32_r, ldy, Y, rocblas_datatype_f32_r, ldy, rocblas_datatype_f32_r,
      rocblas_gemm_algo_standard, 0, 0);
  if (st != rocblas_status_success)
    return fail(MLKV_ERR_HIP, "rocblas_gemm_ex: %s", rocblas_status_to_string(st));
  return MLKV_OK;
}

mlkv_status hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(MLKV_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  return MLKV_OK;
}

// Copies every layer's matrices into the fused path's MFMA tiles (one device
// allocation; after all work already queued on the device, on the null
// stream, finished before returning).
mlkv_status pack_weights(mlkv_model* m) {
  const hipError_t e0 = hipDeviceSynchronize();  // the caller's writes of the weights
  if (e0 != hipSuccess) return fail(MLKV_ERR_HIP, "weight packing: %s", hipGetErrorString(e0));
  const mlkv_map* map = m->map;
  const int D = m->D, NT = D / 16, d = m->d, ff = m->d_ff, h = map->h, hD = h * D;
  const int KB = d / 32, ff_blocks = (ff + D - 1) / D;
  size_t total = 0;
  for (int n = 0; n < map->l; ++n) {
    const int owned = map->own_count[n];
    m->in_off.push_back(total);
    total += static_cast<size_t>(h + 2 * owned + ff_blocks) * NT * KB * mlkv::kPackTile;
    m->out_off.push_back(total);
    total += static_cast<size_t>(d) * (hD + ff);
  }
  void* mem = nullptr;
  if (hipMalloc(&mem, total * sizeof(uint16_t)) != hipSuccess)
    return fail(MLKV_ERR_HIP, "hipMalloc of %zu bytes of packed weights failed", total * 2);
  m->packed = static_cast<uint16_t*>(mem);
  auto u16 = [](const void* p) { return static_cast<const uint16_t*>(p); };
  auto pack = [&](const void* src, int k_rows, int n_cols, uint16_t* dst, int kb_total, int kb0,
                  int nt0, int nt_count) {
    const mlkv::PackParams pp{u16(src), dst, k_rows, n_cols, kb_total, kb0, nt0, nt_count};
    return hip_ok(mlkv::launch_pack(pp, nullptr), "weight packing");
  };
  mlkv_status s;
  for (int n = 0; n < map->l; ++n) {
    const mlkv_layer_weights& lw = m->layers[n];
    const int owned = map->own_count[n];
    uint16_t* win = m->packed + m->in_off[n];
    uint16_t* wout = m->packed + m->out_off[n];
    if ((s = pack(lw.w_q, d, hD, win, KB, 0, 0, h * NT)) != MLKV_OK) return s;
    if (owned > 0 &&
        ((s = pack(lw.w_k, d, owned * D, win, KB, 0, h * NT, owned * NT)) != MLKV_OK ||
         (s = pack(lw.w_v, d, owned * D, win, KB, 0, (h + owned) * NT, owned * NT)) != MLKV_OK))
      return s;
    if ((s = pack(lw.w_fc1, d, ff, win, KB, 0, (h + 2 * owned) * NT, ff_blocks * NT)) != MLKV_OK ||
        (s = pack(lw.w_o, hD, d, wout, (hD + ff) / 32, 0, 0, d / 16)) != MLKV_OK ||
        (s = pack(lw.w_fc2, ff, d, wout, (hD + ff) / 32, hD / 32, 0, d / 16)) != MLKV_OK)
      return s;
  }
  const hipError_t e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) return fail(MLKV_ERR_HIP, "weight packing: %s", hipGetErrorString(e));
  return MLKV_OK;
}

// The fused path serves every batch the decode path takes (its products
// read the weights once per 16 rows); MLKV_MODEL_GEMM=library forces the
// library GEMMs.
bool use_fused(const mlkv_model* m, int B) {
  if (!m->packed || B > mlkv::kFusedMaxBatch) return false;
  const char* env = std::getenv("MLKV_MODEL_GEMM");
  return !(env && std::strcmp(env, "library") == 0);
}

}  // namespace

mlkv_status mlkv_model_create(const mlkv_map* map, int d_model, int d_ff, int head_dim,
                              int rotary_dims, double rotary_base, double ln_eps,
                              const mlkv_layer_weights* layers, mlkv_model** out) {
  mlkv_status s;
  if (!out) return fail(MLKV_ERR_INVALID_ARG, "out must be non-NULL");
  *out = nullptr;
  if ((s = check_map(map)) != MLKV_OK) return s;
  if (head_dim != 64 && head_dim != 128)
    return fail(MLKV_ERR_UNSUPPORTED, "head_dim %d: 64 or 128 supported", head_dim);
  if (d_model != map->h * head_dim)
    return fail(MLKV_ERR_INVALID_ARG, "d_model %d must equal h * head_dim = %d", d_model,
                map->h * head_dim);
  if (d_ff <= 0) return fail(MLKV_ERR_INVALID_ARG, "d_ff must be positive");
  if (rotary_dims < 0 || rotary_dims > head_dim || rotary_dims % 2 != 0)
    return fail(MLKV_ERR_INVALID_ARG, "rotary_dims %d: even, in [0, head_dim]", rotary_dims);
  if (!(rotary_base > 0.0) || !std::isfinite(rotary_base) || !(ln_eps >= 0.0))
    return fail(MLKV_ERR_INVALID_ARG, "rotary_base must be positive, ln_eps non-negative");
  if (!layers) return fail(MLKV_ERR_INVALID_ARG, "layers must be non-NULL");
  for (int n = 0; n < map->l; ++n) {
    const mlkv_layer_weights& w = layers[n];
    if (!w.ln1_w || !w.ln1_b || !w.ln2_w || !w.ln2_b || !w.w_q || !w.b_q || !w.w_o || !w.b_o ||
        !w.w_fc1 || !w.b_fc1 || !w.w_fc2 || !w.b_fc2)
      return fail(MLKV_ERR_INVALID_ARG, "layer %d: a weight pointer is NULL", n);
    const bool owns = map->own_count[n] > 0;
    const bool has_kv = w.w_k && w.b_k && w.w_v && w.b_v;
    const bool no_kv = !w.w_k && !w.b_k && !w.w_v && !w.b_v;
    if (owns ? !has_kv : !no_kv)
      return fail(MLKV_ERR_INVALID_ARG,
                  "layer %d: key/value weights must be given exactly when it owns KV heads", n);
  }
  mlkv_model* m = new (std::nothrow) mlkv_model;
  if (!m) return fail(MLKV_ERR_INVALID_ARG, "out of host memory");
  m->map = map;
  m->d = d_model;
  m->d_ff = d_ff;
  m->D = head_dim;
  m->dims = rotary_dims;
  m->eps = static_cast<float>(ln_eps);
  for (int j = 0; j < rotary_dims / 2; ++j)
    m->inv_freq[j] = std::pow(rotary_base, -2.0 * j / rotary_dims);
  m->layers.assign(layers, layers + map->l);
  if (rocblas_create_handle(&m->blas) != rocblas_status_success) {
    delete m;
    return fail(MLKV_ERR_HIP, "rocblas_create_handle failed");
  }
  // The fused path reads the layer-norm vectors 16 bytes at a time.
  bool ln_aligned = true;
  for (const mlkv_layer_weights& w : m->layers)
    ln_aligned = ln_aligned && aligned16(w.ln1_w) && aligned16(w.ln1_b) && aligned16(w.ln2_w) &&
                 aligned16(w.ln2_b);
  if (d_ff % 32 == 0 && ln_aligned && (s = pack_weights(m)) != MLKV_OK) {
    mlkv_model_destroy(m);
    return s;
  }
  *out = m;
  return ok();
}

void mlkv_model_destroy(mlkv_model* model) {
  if (!model) return;
  if (model->blas) (void)rocblas_destroy_handle(model->blas);
  if (model->packed) (void)hipFree(model->packed);
  delete model;
}

int mlkv_model_fused_path(const mlkv_model* model, int batch) {
  return model && batch > 0 && use_fused(model, batch) ? 1 : 0;
}

size_t mlkv_model_workspace_bytes(const mlkv_model* model, int batch, int capacity) {
  if (!model || batch <= 0 || batch > mlkv::max_batch() || capacity <= 0) return 0;
  return model_ws(model, batch, capacity).total;
}

mlkv_status mlkv_model_decode_step(mlkv_model* model, float* x, const mlkv_cache* cache,
                                   const int32_t* ctx_lens, int max_len_hint, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  mlkv_status s;
  if (!model) return fail(MLKV_ERR_INVALID_ARG, "model must be non-NULL");
  const mlkv_map* map = model->map;
  if ((s = check_cache(cache, map)) != MLKV_OK) return s;
  if (cache->head_dim != model->D)
    return fail(MLKV_ERR_INVALID_ARG, "cache head_dim %d differs from the model's %d",
                cache->head_dim, model->D);
  for (int n = 0; n < map->l; ++n)
    if ((s = check_group_size(map, n)) != MLKV_OK) return s;
  if (!x || !ctx_lens) return fail(MLKV_ERR_INVALID_ARG, "x and ctx_lens must be non-NULL");
  if (!aligned16(x)) return fail(MLKV_ERR_ALIGNMENT, "x must be 16-byte aligned");
  if (!aligned4(ctx_lens)) return fail(MLKV_ERR_ALIGNMENT, "ctx_lens must be 4-byte aligned");
  if (max_len_hint > cache->capacity)
    return fail(MLKV_ERR_CAPACITY, "max_len_hint %d above capacity %d", max_len_hint,
                cache->capacity);
  const int B = cache->batch, D = model->D, n_kv = map->n_kv, h = map->h;
  const ModelWs w = model_ws(model, B, cache->capacity);
  if (!workspace || workspace_bytes < w.total)
    return fail(MLKV_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", w.total,
                workspace ? workspace_bytes : 0);
  if (!aligned16(workspace)) return fail(MLKV_ERR_ALIGNMENT, "workspace not 16-byte aligned");
  const int limit = max_len_hint <= 0 ? cache->capacity : max_len_hint;
  if ((s = check_lengths_if_requested(ctx_lens, B, 1, limit, stream)) != MLKV_OK) return s;
  if (rocblas_set_stream(model->blas, stream) != rocblas_status_success)
    return fail(MLKV_ERR_HIP, "rocblas_set_stream failed");

  char* base = static_cast<char*>(workspace);
  auto bf = [&](size_t off) { return reinterpret_cast<uint16_t*>(base + off); };
  auto f32 = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  const int hD = h * D, kvD = n_kv * D, d = model->d, ff = model->d_ff;
  auto u16 = [](const void* p) { return static_cast<const uint16_t*>(p); };
  // Attention of layer n with the owner's append (inside the attention launch
  // when the layer reads every head it owns).  The schedule is planned again
  // only when the plan's key changes.
  auto layer_attention = [&](int n, PlanKey& planned_key,
                             const mlkv::SideProduct* side = nullptr) -> mlkv_status {
    mlkv_status st;
    const int owned = map->own_count[n];
    const int own0 = owned ? map->own_begin[n] * D : 0;
    const bool fused_append = owned > 0 && map->own_begin[n] >= map->kv_begin[n] &&
                              map->own_begin[n] + owned <= map->kv_begin[n] + map->kv_count[n];
    if (owned > 0 && !fused_append &&
        (st = append_impl(n, map, cache, bf(w.k16) + own0, bf(w.v16) + own0, kvD, ctx_lens,
                          stream)) != MLKV_OK)
      return st;
    const Plan pl = plan(map, n, B, max_len_of(cache, max_len_hint), cache->head_dim);
    const bool records = plan_records(pl);
    const PlanKey key = plan_key(pl, map->kv_count[n]);
    const int mode = !records ? 0 : key == planned_key ? 2 : 1;
    if ((st = attention_impl(n, bf(w.q16), cache, map, ctx_lens, 1, bf(w.o16), MLKV_OUT_BF16,
                             max_len_hint, base + w.attn, w.attn_bytes, stream, mode,
                             fused_append ? bf(w.k16) : nullptr,
                             fused_append ? bf(w.v16) : nullptr, nullptr, 0, side)) != MLKV_OK)
      return st;
    if (records) planned_key = key;
    return MLKV_OK;
  };
  const bool fused = use_fused(model, B);
  PlanKey planned_key;
  for (int n = 0; n < map->l; ++n) {
    const mlkv_layer_weights& lw = model->layers[n];
    const int owned = map->own_count[n];
    const int own0 = owned ? map->own_begin[n] * D : 0;
    if (fused) {
      mlkv::LayerInParams ip{};
      ip.x = x;
      ip.ln1_w = u16(lw.ln1_w);
      ip.ln1_b = u16(lw.ln1_b);
      ip.ln2_w = u16(lw.ln2_w);
      ip.ln2_b = u16(lw.ln2_b);
      ip.w = model->packed + model->in_off[n];
      ip.b_q = u16(lw.b_q);
      ip.b_k = u16(lw.b_k);
      ip.b_v = u16(lw.b_v);
      ip.b_fc1 = u16(lw.b_fc1);
      ip.q16 = bf(w.q16);
      ip.k16 = bf(w.k16);
      ip.v16 = bf(w.v16);
      ip.f16 = bf(w.f16);
      ip.pos = ctx_lens;
      ip.rows = B;
      ip.d = d;
      ip.h = h;
      ip.owned = owned;
      ip.ff = ff;
      ip.kv_stride = kvD;
      ip.kv_offset = own0;
      ip.dims = model->dims;
      ip.eps = model->eps;
      std::memcpy(ip.inv_freq, model->inv_freq, sizeof ip.inv_freq);
      if ((s = hip_ok(mlkv::launch_layer_in(ip, D, stream), "layer-in product")) != MLKV_OK)
        return s;
      // The MLP's second product rides in the attention launch (its extra
      // workgroups), leaving layer-out the W_o product and the sum.
      mlkv::SideProduct sp{};
      sp.w = model->packed + model->out_off[n];
      sp.f16 = bf(w.f16);
      sp.b2 = u16(lw.b_fc2);
      sp.y = f32(w.m32);
      sp.rows = B;
      sp.d = d;
      sp.ff = ff;
      sp.ka = hD / 32;
      sp.kt = hD / 32 + ff / 32;
      sp.n_blocks = (d / 16) * ((B + 15) / 16);
      if ((s = layer_attention(n, planned_key, &sp)) != MLKV_OK) return s;
      const mlkv::LayerOutParams op{bf(w.o16), bf(w.f16), model->packed + model->out_off[n],
                                    u16(lw.b_o), u16(lw.b_fc2), x, B, d, hD, ff, f32(w.m32)};
      if ((s = hip_ok(mlkv::launch_layer_out(op, stream), "layer-out product")) != MLKV_OK)
        return s;
      continue;
    }
    mlkv::NormParams np{x, u16(lw.ln1_w), u16(lw.ln1_b), u16(lw.ln2_w), u16(lw.ln2_b),
                        bf(w.h1), bf(w.h2), B, d, model->eps};
    if ((s = hip_ok(mlkv::launch_norm2(np, stream), "layer norm")) != MLKV_OK) return s;
    if ((s = gemm(model->blas, B, hD, d, bf(w.h1), d, lw.w_q, f32(w.q32), hD)) != MLKV_OK)
      return s;
    if (owned) {
      if ((s = gemm(model->blas, B, owned * D, d, bf(w.h1), d, lw.w_k, f32(w.k32) + own0,
                    kvD)) != MLKV_OK ||
          (s = gemm(model->blas, B, owned * D, d, bf(w.h1), d, lw.w_v, f32(w.v32) + own0,
                    kvD)) != MLKV_OK)
        return s;
    }
    mlkv::QkvEpilogueParams qp{};
    qp.q32 = f32(w.q32);
    qp.b_q = u16(lw.b_q);
    qp.q16 = bf(w.q16);
    qp.k32 = f32(w.k32);
    qp.v32 = f32(w.v32);
    qp.b_k = u16(lw.b_k);
    qp.b_v = u16(lw.b_v);
    qp.k16 = bf(w.k16);
    qp.v16 = bf(w.v16);
    qp.pos = ctx_lens;
    qp.rows = B;
    qp.q_width = hD;
    qp.kv_width = owned * D;
    qp.kv_stride = kvD;
    qp.kv_offset = own0;
    qp.D = D;
    qp.dims = model->dims;
    std::memcpy(qp.inv_freq, model->inv_freq, sizeof qp.inv_freq);
    if ((s = hip_ok(mlkv::launch_qkv_epilogue(qp, stream), "q/k/v epilogue")) != MLKV_OK)
      return s;
    if ((s = layer_attention(n, planned_key)) != MLKV_OK) return s;
    if ((s = gemm(model->blas, B, d, hD, bf(w.o16), hD, lw.w_o, f32(w.a32), d)) != MLKV_OK ||
        (s = gemm(model->blas, B, ff, d, bf(w.h2), d, lw.w_fc1, f32(w.f32), ff)) != MLKV_OK)
      return s;
    mlkv::GeluParams gp{f32(w.f32), u16(lw.b_fc1), bf(w.f16), B, ff};
    if ((s = hip_ok(mlkv::launch_gelu(gp, stream), "GELU")) != MLKV_OK) return s;
    if ((s = gemm(model->blas, B, d, ff, bf(w.f16), ff, lw.w_fc2, f32(w.m32), d)) != MLKV_OK)
      return s;
    mlkv::ResidualParams rp{x, f32(w.a32), f32(w.m32), u16(lw.b_o), u16(lw.b_fc2), B, d};
    if ((s = hip_ok(mlkv::launch_residual(rp, stream), "residual")) != MLKV_OK) return s;
  }
  return ok();
}

mlkv_status mlkv_profile_enable(int max_launches) {
  if (max_launches <= 0) return fail(MLKV_ERR_INVALID_ARG, "max_launches must be positive");
  mlkv_profile_disable();
  Profile& prof = g_profile;
  prof.start.assign(max_launches, nullptr);
  prof.stop.assign(max_launches, nullptr);
  for (int i = 0; i < max_launches; ++i) {
    // Timing-only events: no system-scope fence (no cache writeback or
    // invalidate around the timed kernel, which would slow it and the next).
    if (hipEventCreateWithFlags(&prof.start[i], hipEventDisableSystemFence) != hipSuccess ||
        hipEventCreateWithFlags(&prof.stop[i], hipEventDisableSystemFence) != hipSuccess) {
      mlkv_profile_disable();
      return fail(MLKV_ERR_HIP, "hipEventCreate failed");
    }
  }
  prof.used = 0;
  prof.on = true;
  return ok();
}

mlkv_status mlkv_profile_read(int* launches, double* total_ms, double* min_ms, double* max_ms) {
  if (!launches || !total_ms || !min_ms || !max_ms)
    return fail(MLKV_ERR_INVALID_ARG, "output pointers must be non-NULL");
  Profile& prof = g_profile;
  double tot = 0.0, lo = 0.0, hi = 0.0;
  for (int i = 0; i < prof.used; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(prof.stop[i]) != hipSuccess ||
        hipEventElapsedTime(&ms, prof.start[i], prof.stop[i]) != hipSuccess)
      return fail(MLKV_ERR_HIP, "reading profile events failed");
    tot += ms;
    lo = i == 0 || ms < lo ? ms : lo;
    hi = i == 0 || ms > hi ? ms : hi;
  }
  *launches = prof.used;
  *total_ms = tot;
  *min_ms = lo;
  *max_ms = hi;
  return ok();
}

mlkv_status mlkv_profile_durations(double* ms, int capacity, int* count) {
  if (!count || (capacity > 0 && !ms)) return fail(MLKV_ERR_INVALID_ARG, "bad output arguments");
  Profile& prof = g_profile;
  const int n = prof.used < capacity ? prof.used : (capacity > 0 ? capacity : 0);
  for (int i = 0; i < n; ++i) {
    float t = 0.f;
    if (hipEventSynchronize(prof.stop[i]) != hipSuccess ||
        hipEventElapsedTime(&t, prof.start[i], prof.stop[i]) != hipSuccess)
      return fail(MLKV_ERR_HIP, "reading profile events failed");
    ms[i] = t;
  }
  *count = n;
  return ok();
}

mlkv_status mlkv_profile_launch_floor(int workgroups, int threads, int reps, hipStream_t stream,
                                      double* median_ms) {
  if (workgroups <= 0 || threads <= 0 || threads > 1024 || reps <= 0 || !median_ms)
    return fail(MLKV_ERR_INVALID_ARG, "workgroups, threads (<= 1024), reps must be positive");
  std::vector<hipEvent_t> ev(2 * static_cast<size_t>(reps), nullptr);
  mlkv_status s = MLKV_OK;
  for (auto& e : ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
      s = fail(MLKV_ERR_HIP, "hipEventCreate failed");
      break;
    }
  std::vector<double> ms;
  for (int i = 0; s == MLKV_OK && i < reps; ++i)
    if (mlkv::launch_empty_timed(workgroups, threads, stream, ev[2 * i], ev[2 * i + 1]) !=
        hipSuccess)
      s = fail(MLKV_ERR_HIP, "empty launch failed");
  for (int i = 0; s == MLKV_OK && i < reps; ++i) {
    float t = 0.f;
    if (hipEventSynchronize(ev[2 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&t, ev[2 * i], ev[2 * i + 1]) != hipSuccess)
      s = fail(MLKV_ERR_HIP, "reading floor events failed");
    ms.push_back(t);
  }
  for (hipEvent_t e : ev)
    if (e) (void)hipEventDestroy(e);
  if (s != MLKV_OK) return s;
  std::sort(ms.begin(), ms.end());
  *median_ms = ms[ms.size() / 2];
  return ok();
}

mlkv_status mlkv_profile_read_bandwidth(const void* buffer, size_t bytes, int reps,
                                        hipStream_t stream, double* median_gbs, double* best_gbs) {
  if (!buffer || bytes < 16 * 1024 || reps <= 0 || !median_gbs || !best_gbs)
    return fail(MLKV_ERR_INVALID_ARG, "buffer, bytes (>= 16 KiB), reps and outputs required");
  if (!aligned16(buffer)) return fail(MLKV_ERR_ALIGNMENT, "buffer must be 16-byte aligned");
  const size_t body = bytes / 16 * 16 - 16;  // the last 16 bytes hold the sink word
  uint32_t* sink = reinterpret_cast<uint32_t*>(static_cast<char*>(const_cast<void*>(buffer)) + body);
  const int workgroups = static_cast<int>(8 * compute_units_or_fallback());
  std::vector<hipEvent_t> ev(2 * static_cast<size_t>(reps), nullptr);
  mlkv_status s = MLKV_OK;
  for (auto& e : ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
      s = fail(MLKV_ERR_HIP, "hipEventCreate failed");
      break;
    }
  for (int i = 0; s == MLKV_OK && i < reps; ++i)
    if (mlkv::launch_stream_read_timed(buffer, body, sink, workgroups, stream, ev[2 * i],
                                       ev[2 * i + 1]) != hipSuccess)
      s = fail(MLKV_ERR_HIP, "stream read launch failed");
  std::vector<double> gbs;
  for (int i = 0; s == MLKV_OK && i < reps; ++i) {
    float t = 0.f;
    if (hipEventSynchronize(ev[2 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&t, ev[2 * i], ev[2 * i + 1]) != hipSuccess)
      s = fail(MLKV_ERR_HIP, "reading stream events failed");
    gbs.push_back(static_cast<double>(body) / (t * 1e-3) / 1e9);
  }
  for (hipEvent_t e : ev)
    if (e) (void)hipEventDestroy(e);
  if (s != MLKV_OK) return s;
  std::sort(gbs.begin(), gbs.end());
  *median_gbs = gbs[gbs.size() / 2];
  *best_gbs = gbs.back();
  return ok();
}

void mlkv_profile_disable(void) {
  Profile& prof = g_profile;
  for (hipEvent_t e : prof.start)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : prof.stop)
    if (e) (void)hipEventDestroy(e);
  prof.start.clear();
  prof.stop.clear();
  prof.used = 0;
  prof.on = false;
}

}  // extern "C"
