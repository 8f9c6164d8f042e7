// HIP kernels of MLKV decode attention for CDNA4 (gfx950, wave64, MFMA).
//
//   append_kernel     newest token's K/V rows -> cache slot (bit copy)
//   attention_kernel  split-K attention of one layer.  Each (sequence, KV
//                     head) unit is cut into runs of the same number of
//                     32-token tiles, the run length chosen on the device from
//                     the actual lengths so that the runs of all units fill
//                     the launched workgroups (ragged batches stay balanced);
//                     a workgroup takes one run and serves every query head
//                     mapped to the KV head from one pass over it.  A unit of
//                     one run is finished in place; otherwise each run leaves
//                     a partial (max, denominator, output), merged by the
//                     unit's last run to finish when the partials fit its
//                     staging area.  In a decode step the owning layer's
//                     launch also appends the newest token.
//   combine_kernel    log-sum-exp merge of a unit's partials, fixed order
//                     (when they were not merged in place)
//   fill_kernel       zero fill of a workspace
//
// Math (paper Section 2.1 Eqs. 1-3; MLKV head map Section 3 Eqs. 13-17):
//   o = sum_t softmax_t(q.k_t / sqrt(D)) v_t.  Scores are kept in the log2
//   domain (scale folded with log2(e)) so every exponential is one v_exp_f32.
//   The running-max form of softmax is an exact rewrite up to rounding.
//
// Register-level data flow of one wave and one 32-token tile (G <= 16 query
// heads of the KV head are padded to the 16 MFMA columns):
//   S^T[32 tok][16 heads] = K[32][D] * Q^T[D][16]      (2 x D/32 MFMA 16x16x32)
//   P = exp2(S - running max), rounded to bf16
//   O^T[D][16]          += V^T[D][32] * P^T[32][16]   (D/16 MFMA 16x16x32)
// MFMA operand rule used throughout: lane l supplies row/column (l % 16) and
// the 8 consecutive k-slots 8*(l/16) .. 8*(l/16)+7; the 16x16 fp32 result
// gives lane l column (l % 16), rows 4*(l/16) .. 4*(l/16)+3.
// K rows are therefore loaded 16 bytes per lane straight from the row-major
// key plane, V^T rows 16 bytes per lane straight from the value plane whose
// 32-token blocks are stored channel-major (see mlkv.h).  The score tile's
// row order is chosen so that the lane holding scores of tokens 8j..8j+7
// is exactly the lane that must supply them as P^T k-slots: no shuffles
// between the two products.  Each wave keeps the next tile's loads in flight
// while it computes the current one.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "kernels.h"
#include "tile.h"

namespace mlkv {

// Attended length of sequence b: lens[b] + len_offset, clamped to [0, max_len]
// (max_len <= capacity bounds the work list and the workspace).
__device__ __forceinline__ int attended_len(const AttnParams& p, int b) {
  int L = p.lens[b] + p.len_offset;
  L = L < 0 ? 0 : L;
  return L > p.max_len ? p.max_len : L;
}

// Tiles of L >= 0 positions.
__device__ __forceinline__ int tiles_of(int L) {
  return static_cast<int>((static_cast<unsigned>(L) + kTile - 1) / kTile);
}

// ---------------------------------------------------------------------------
// Rotary position embedding of the GPT-NeoX architecture (the paper's Pythia
// models, Section 4.2) for the newest token of each sequence.  Pair
// (j, j + half) of a head vector's first 2*half channels turns by the angle
// pos * base^(-2j/(2*half)):
//   y_j = x_j cos - x_{j+half} sin,   y_{j+half} = x_{j+half} cos + x_j sin.
// rope_table_kernel tabulates cos and sin in double once per step, one
// (sequence, pair) per thread; the attention and append kernels rotate the
// 8-channel chunks they load from that table.  Each product and the sum are
// rounded in double (no fused multiply-add) and the result once to bf16,
// nearest even.
// ---------------------------------------------------------------------------
constexpr int kRopeThreads = 256;

__global__ __launch_bounds__(kRopeThreads) void rope_table_kernel(RopeTableParams p) {
  const int i = blockIdx.x * kRopeThreads + threadIdx.x;
  if (i >= p.B * p.half) return;
  const int b = i / p.half, j = i - b * p.half;
  double s, c;
  sincos(static_cast<double>(p.pos[b]) * p.inv_freq[j], &s, &c);
  reinterpret_cast<double2*>(p.cs)[i] = make_double2(c, s);
}

__device__ __forceinline__ uint16_t f64_to_bf16_bits(double v) {
  // Round to odd into fp32 (24 bits: no double rounding), then to nearest
  // even into bf16.
  const float f = __double2float_rz(v);
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if (static_cast<double>(f) != v && v == v) u |= 1u;
  return f32_to_bf16_bits(__builtin_bit_cast(float, u));
}

__device__ __forceinline__ double bf16_to_f64(uint16_t x) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(x) << 16);
}

// y = own cos -/+ partner sin with both products and the sum rounded.
template <bool HI>
__device__ __forceinline__ double rotate_one(double own, double partner, double c, double s) {
#pragma clang fp contract(off)
  return HI ? own * c + partner * s : own * c - partner * s;
}

// The rotated chunk of channels c0 .. c0+7 (c0 a multiple of 8): `own` holds
// them, `partner` channels c0 + half (c0 < half) or c0 - half (half <= c0 <
// 2*half); cs = the table entries (cos, sin) of pairs c0 % half ... Chunks at
// or past 2*half are returned unchanged.
template <typename CS>
__device__ __forceinline__ u16x8 rotate_chunk(u16x8 own, u16x8 partner, int c0, int half, CS cs) {
  if (c0 >= 2 * half) return own;
  const bool hi = c0 >= half;
  const int j0 = hi ? c0 - half : c0;
  u16x8 y;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double2 t = cs(j0 + e);
    const double u = bf16_to_f64(own[e]), w = bf16_to_f64(partner[e]);
    y[e] = f64_to_bf16_bits(hi ? rotate_one<true>(u, w, t.x, t.y) : rotate_one<false>(u, w, t.x, t.y));
  }
  return y;
}

// Offset of the channel chunk paired with chunk c0 (see rotate_chunk).
__device__ __forceinline__ int partner_chunk(int c0, int half) {
  return c0 < half ? c0 + half : c0 - half;
}

// ---------------------------------------------------------------------------
// Cache append (Section 2.4): one workgroup per (sequence b, owned head c),
// one thread per 8 channels.  With a rotary table the key is rotated first.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(D / 8) void append_kernel(AppendParams p) {
  const int b = blockIdx.x;
  const int c = blockIdx.y;
  const int pos = p.positions[b];
  if (pos < 0 || pos >= p.S) return;
  const int d0 = threadIdx.x * 8;
  const size_t row = static_cast<size_t>(b) * p.row_stride + static_cast<size_t>(c) * D;
  u16x8 kv_k = load16(p.k_new + row + d0);
  const u16x8 kv_v = load16(p.v_new + row + d0);
  if (p.rope_cs && d0 < 2 * p.rope_half) {
    const u16x8 partner = load16(p.k_new + row + partner_chunk(d0, p.rope_half));
    const double2* cs = reinterpret_cast<const double2*>(p.rope_cs) + static_cast<size_t>(b) * p.rope_half;
    kv_k = rotate_chunk(kv_k, partner, d0, p.rope_half, [&](int j) { return cs[j]; });
  }
  const size_t seq = static_cast<size_t>(p.kv_begin + c) * p.B + b;
  *reinterpret_cast<u16x8*>(p.k + (seq * p.S + (pos & ~(kTile - 1))) * D +
                            kchunk<D>(pos & (kTile - 1), d0 / 8) * 8) = kv_k;
  uint16_t* vdst = p.v + (seq * p.S + (pos & ~(kTile - 1))) * D + (pos & (kTile - 1));
#pragma unroll
  for (int e = 0; e < 8; ++e) vdst[(d0 + e) * kTile] = kv_v[e];
}

// ---------------------------------------------------------------------------
// Cache planes <-> logical rows, one workgroup per 32-token block of one
// (KV head, sequence): the block's K rows move as 16-byte chunks to and from
// their places in the tile (kchunk); its V rows go through LDS, where the
// [32][D] tile is transposed to [D][32], so both the row side and the plane
// side move in 16-byte pieces.
// ---------------------------------------------------------------------------
constexpr int kRowsThreads = 256;

template <int D>
__global__ __launch_bounds__(kRowsThreads) void cache_rows_kernel(CacheRowsParams p) {
  constexpr int kChunks = kTile * D / 8;      // 16-byte pieces per block and plane
  constexpr int kPad = 8;                     // LDS row padding (elements)
  __shared__ alignas(16) uint16_t tile[kTile][D + kPad];
  const size_t blocks_per_seq = static_cast<size_t>(p.S / kTile);
  const size_t blk = blockIdx.x;              // (c, b, t-block), c-major
  const size_t seq = blk / blocks_per_seq;    // c * B + b
  const size_t tb = blk - seq * blocks_per_seq;
  const size_t row_off = (seq * p.S + tb * kTile) * D;  // in the rows
  const size_t plane_off = (static_cast<size_t>(p.kv_begin) * p.B * p.S) * D + row_off;
  for (int i = threadIdx.x; i < kChunks; i += kRowsThreads) {  // token i / (D/8), channels
    const size_t e = static_cast<size_t>(i) * 8;
    const size_t pe = static_cast<size_t>(kchunk<D>(i / (D / 8), i % (D / 8))) * 8;
    if (p.to_cache)
      *reinterpret_cast<u16x8*>(p.k_plane + plane_off + pe) = load16(p.k_rows + row_off + e);
    else
      *reinterpret_cast<u16x8*>(p.k_rows + row_off + e) = load16(p.k_plane + plane_off + pe);
  }
  if (p.to_cache) {
    for (int i = threadIdx.x; i < kChunks; i += kRowsThreads) {  // token i / (D/8), channels
      const int t = i / (D / 8), c = (i - t * (D / 8)) * 8;
      *reinterpret_cast<u16x8*>(&tile[t][c]) = load16(p.v_rows + row_off + t * D + c);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kChunks; i += kRowsThreads) {  // channel i / 4, tokens
      const int d = i / (kTile / 8), t0 = (i - d * (kTile / 8)) * 8;
      u16x8 v;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = tile[t0 + e][d];
      *reinterpret_cast<u16x8*>(p.v_plane + plane_off + d * kTile + t0) = v;
    }
  } else {
    for (int i = threadIdx.x; i < kChunks; i += kRowsThreads) {
      const int d = i / (kTile / 8), t0 = (i - d * (kTile / 8)) * 8;
      const u16x8 v = load16(p.v_plane + plane_off + d * kTile + t0);
#pragma unroll
      for (int e = 0; e < 8; ++e) tile[t0 + e][d] = v[e];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kChunks; i += kRowsThreads) {
      const int t = i / (D / 8), c = (i - t * (D / 8)) * 8;
      *reinterpret_cast<u16x8*>(p.v_rows + row_off + t * D + c) =
          *reinterpret_cast<const u16x8*>(&tile[t][c]);
    }
  }
}

// acc / den with one reciprocal (within one ulp) for the four channels; zeros
// for an empty row (den = 0).  A row with any attended position has den >= 1
// (its largest weight is at least one), and den = 1 leaves acc exact;
// non-finite inputs give a non-finite den, which propagates as in the
// definition rather than being taken for an empty row.
__device__ __forceinline__ f32x4 normalize4(f32x4 acc, float den) {
  return den != 0.f ? acc * __builtin_amdgcn_rcpf(den) : f32x4{0.f, 0.f, 0.f, 0.f};
}

// ---------------------------------------------------------------------------
// Split-K attention over a balanced flat tile list.
// ---------------------------------------------------------------------------
// Four consecutive channels d..d+3 of output row `row` (d a multiple of 4).
template <int D>
__device__ __forceinline__ void store_out4(const AttnParams& p, size_t row, int d, f32x4 v) {
  if (p.out_bf16) {
    typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
    const u16x4 bits = {f32_to_bf16_bits(v[0]), f32_to_bf16_bits(v[1]), f32_to_bf16_bits(v[2]),
                        f32_to_bf16_bits(v[3])};
    *reinterpret_cast<u16x4*>(static_cast<uint16_t*>(p.out) + row * D + d) = bits;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + row * D + d) = v;
  }
}

constexpr int kMaxWaves = 16;  // waves of the widest attention workgroup the schedule serves

struct SchedShared {
  int len[kMaxBatch];         // attended lengths (each thread's own sequences)
  int wsum[2][kMaxWaves][4];  // per-wave totals of the two scans
};

// A run of the plan: sequence b, KV group r, run j of nb of that unit,
// attended length L, tiles [k0, k1).  b < 0 marks a workgroup with no run.
// z >= 0: sequence z attends to nothing and this workgroup writes its zero
// output (a launch has at least as many workgroups as sequences).
struct alignas(16) RunItem {
  int b, r, j, nb;
  int L, k0, k1, z;
};

// Partial outputs the last run of a unit can stage in LDS to merge in place.
constexpr int kStageFloats = 8192;
constexpr int kStageMl = 512;

template <int D, int W>
struct alignas(16) AttnShared {
  union {  // phases: schedule, then the waves' merge, then (last run only) staging
    SchedShared sc;
    struct {
      float acc[W][16][D + 4];
      float m[W][16];
      float l[W][16];
    };
    float stage[kStageFloats];
  };
  float stage_ml[kStageMl];
  RunItem run;                          // this workgroup's run, from the schedule
  alignas(16) uint16_t new_row[2 * D];  // newest token's key and value (fused append)
  double2 rope[kMaxRopePairs];          // the sequence's rotary (cos, sin) pairs
  int last;
};

// Inclusive prefix sum over the 64 lanes of a wave: within each row of 16
// lanes by shifted adds (1, 2, 4, 8), then the last lane of row 0 into row 1
// and of row 2 into row 3, then the last lane of row 1 into rows 2 and 3
// (row broadcasts).  Lane 63 ends with the wave's total.
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

__device__ __forceinline__ int wave_total(int incl) { return __builtin_amdgcn_readlane(incl, 63); }

// floor(x) as an integer (the convert rounds toward minus infinity).
__device__ __forceinline__ int floor_int(float x) { return static_cast<int>(__builtin_floorf(x)); }

// ceil(t / R) for integers 0 <= t < 2^21 and R >= 1, from th = t - 1/2 and
// rR = the float reciprocal of R (within one ulp): th / R lies at least
// 1 / (2R) from every integer, farther than the product's rounding error
// (below th * 2^-22 / R), so floor(th * rR) = ceil(t / R) - 1 exactly (also
// for t = 0, where it is -1).
__device__ __forceinline__ int ceil_div_half(float th, float rR) { return floor_int(th * rR) + 1; }

// The run schedule every workgroup derives identically from the lengths,
// computed by all NT threads together (the sequences split evenly over them)
// between barriers: tiles t_b = ceil(L_b / 32); run length R is the least of
// R0 = ceil(T / W), R0 + 1, R0 + 2 (T = all tiles, W = workgroups, never
// below min_tiles) whose run count N(R) = n_groups * sum_b ceil(t_b / R) fits
// W, else RF = ceil(T / (W - U)) (U = non-empty units), which always fits.
// One scan (per wave, then across the waves' totals) gives T and U, and the
// uniform arithmetic on them runs on the scalar unit.  A second scan covers
// the four candidates' per-thread run counts at once, two to a 32-bit word:
// every count and prefix is at most N(R) / n_groups <= W + U <= 2W <= 2^15
// (the host schedules at most 2^14 workgroups), so the 16-bit halves never
// carry.  Each thread's first run under the chosen R is its prefix less its
// own count.  The thread whose sequence holds run g writes that run to `run`
// (b stays -1 when no sequence does), the thread of sequence g marks it for
// zeroing when it attends to nothing, and workgroup 0 writes the runs per
// sequence to p.runs (the merge kernel's input).  Ends with a barrier.
template <int NT>
__device__ void schedule(const AttnParams& p, SchedShared& sm, RunItem& run, int g) {
  constexpr int NW = NT / 64;
  static_assert(NW <= kMaxWaves, "schedule: too many waves");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (p.B + NT - 1) / NT;  // sequences per thread
  const int b0 = tid * per;
  const int b1 = b0 + per < p.B ? b0 + per : p.B;
  if (tid == 0) run = RunItem{-1, 0, 0, 0, 0, 0, 0, -1};
  int tot = 0, nonempty = 0;
  for (int b = b0; b < b1; ++b) {
    const int L = attended_len(p, b);
    sm.len[b] = L;
    const int t = tiles_of(L);
    tot += t;
    nonempty += t > 0 ? 1 : 0;
  }
  tot = wave_incl_scan(tot);
  nonempty = wave_incl_scan(nonempty);
  if (lane == 63) {
    sm.wsum[0][wave][0] = tot;
    sm.wsum[0][wave][1] = nonempty;
  }
  __syncthreads();
  unsigned all_tot = 0, all_nonempty = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    all_tot += __builtin_amdgcn_readfirstlane(sm.wsum[0][w][0]);
    all_nonempty += __builtin_amdgcn_readfirstlane(sm.wsum[0][w][1]);
  }
  const unsigned T = all_tot * static_cast<unsigned>(p.n_groups);  // below 2^30
  const unsigned U = all_nonempty * static_cast<unsigned>(p.n_groups);
  const unsigned W = static_cast<unsigned>(p.n_blocks);  // at least the units, so U <= W
  const unsigned mt = static_cast<unsigned>(p.min_tiles);
  unsigned R0 = (T + W - 1) / W;
  R0 = R0 < mt ? mt : R0;
  unsigned RF = U < W ? (T + (W - U) - 1) / (W - U) : static_cast<unsigned>(p.max_len);
  RF = RF < mt ? mt : RF;
  const int Rc[4] = {static_cast<int>(R0), static_cast<int>(R0 + 1), static_cast<int>(R0 + 2),
                     static_cast<int>(RF)};
  float rc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) rc[c] = __builtin_amdgcn_rcpf(static_cast<float>(Rc[c]));
  int own[4] = {0, 0, 0, 0};
  for (int b = b0; b < b1; ++b) {
    const float th = static_cast<float>(tiles_of(sm.len[b])) - 0.5f;
#pragma unroll
    for (int c = 0; c < 4; ++c) own[c] += floor_int(th * rc[c]);
  }
  const int nseq = b1 > b0 ? b1 - b0 : 0;  // the +1 of each ceil_div_half
  const int own01 = (own[0] + nseq) | ((own[1] + nseq) << 16);
  const int own23 = (own[2] + nseq) | ((own[3] + nseq) << 16);
  const int incl01 = wave_incl_scan(own01);
  const int incl23 = wave_incl_scan(own23);
  if (lane == 63) {
    sm.wsum[1][wave][0] = incl01;
    sm.wsum[1][wave][1] = incl23;
  }
  __syncthreads();
  unsigned tot01 = 0, tot23 = 0;
  int before01 = 0, before23 = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int v01 = __builtin_amdgcn_readfirstlane(sm.wsum[1][w][0]);
    const int v23 = __builtin_amdgcn_readfirstlane(sm.wsum[1][w][1]);
    tot01 += static_cast<unsigned>(v01);
    tot23 += static_cast<unsigned>(v23);
    before01 += w < wave ? v01 : 0;
    before23 += w < wave ? v23 : 0;
  }
  const unsigned total[4] = {tot01 & 0xffffu, tot01 >> 16, tot23 & 0xffffu, tot23 >> 16};
  int pick = 3;
#pragma unroll
  for (int c = 2; c >= 0; --c)
    if (total[c] * static_cast<unsigned>(p.n_groups) <= W) pick = c;
  int R = Rc[3];
  float rR = rc[3];
#pragma unroll
  for (int c = 2; c >= 0; --c)
    if (pick == c) {
      R = Rc[c];
      rR = rc[c];
    }
  // This thread's exclusive prefix under the chosen candidate (packed halves
  // subtract without borrow: each half of incl is at least that of own).
  const int pre2 = pick < 2 ? before01 + incl01 - own01 : before23 + incl23 - own23;
  int excl = ((pre2 >> ((pick & 1) * 16)) & 0xffff) * p.n_groups;  // runs before this thread's
  for (int b = b0; b < b1; ++b) {
    const int L = sm.len[b];
    const int t = tiles_of(L);
    const int nb = ceil_div_half(static_cast<float>(t) - 0.5f, rR);  // runs of each unit of b
    const int runs = p.n_groups * nb;
    if (g == 0 && p.runs) p.runs[b] = nb;
    if (excl <= g && g < excl + runs) {  // exactly one sequence holds run g
      const int rem = g - excl;
      // floor(rem / nb): (rem + 1/2) / nb lies at least 1 / (2 nb) from an integer.
      const int r = floor_int((static_cast<float>(rem) + 0.5f) *
                              __builtin_amdgcn_rcpf(static_cast<float>(nb)));
      const int j = rem - r * nb;
      const int k0 = j * R;
      run.b = b;
      run.r = r;
      run.j = j;
      run.nb = nb;
      run.L = L;
      run.k0 = k0;
      run.k1 = k0 + R < t ? k0 + R : t;
    }
    if (b == g && L == 0) run.z = g;
    excl += runs;
  }
  __syncthreads();
}

// Register budget: at least 3 waves per SIMD for D = 64 and 2 for D = 128
// with four-wave workgroups (12 / 8 waves per compute unit in flight).
// One workgroup of a SideProduct: the W waves stand for the eight waves of a
// layer-out workgroup (wave w for virtual waves w, w + W, ...), so every
// output is the same sum in the same order; part: 8 x 64 tiles of LDS.
template <int W>
__device__ void side_product(const SideProduct& s, int id, f32x4* part) {
  constexpr int PRE = 12;  // k-blocks whose loads are issued before their products
  const int nb = s.d / 16;
  const int blk = id % nb, b0 = (id / nb) * 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, grp = lane >> 4;
  const bool live = b0 + r < s.rows;
  const uint16_t* wblk = s.w + static_cast<size_t>(blk) * s.kt * kPackTile + lane * 8;
  const uint16_t* frow = s.f16 + static_cast<size_t>(b0 + (live ? r : 0)) * s.ff + 8 * grp;
  const u16x8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int v = wave; v < 8; v += W) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    // the first W_2 k-block of virtual wave v: the least kb >= ka with kb % 8 == v
    for (int base = s.ka + (v - s.ka % 8 + 8) % 8; base < s.kt; base += PRE * 8) {
      u16x8 a[PRE], f[PRE];
#pragma unroll
      for (int i = 0; i < PRE; ++i) {
        const int kb = base + i * 8;
        if (kb < s.kt) {
          a[i] = load16(wblk + static_cast<size_t>(kb) * kPackTile);
          f[i] = live ? load16(frow + (kb - s.ka) * 32) : zero;
        }
      }
#pragma unroll
      for (int i = 0; i < PRE; ++i)
        if (base + i * 8 < s.kt) acc = mfma_bf16(as_bf16(a[i]), as_bf16(f[i]), acc);
    }
    part[v * 64 + lane] = acc;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    f32x4 sm = part[l];
#pragma unroll
    for (int v = 1; v < 8; ++v) sm += part[v * 64 + l];
    // Result lane l: row b0 + l % 16, outputs 16 blk + 4 ((l / 16) % 4) + i.
    const int b = b0 + (l & 15), n0 = blk * 16 + 4 * ((l >> 4) & 3);
    if (b < s.rows) {
      float4 y;
      y.x = sm[0] + __builtin_bit_cast(float, static_cast<uint32_t>(s.b2[n0]) << 16);
      y.y = sm[1] + __builtin_bit_cast(float, static_cast<uint32_t>(s.b2[n0 + 1]) << 16);
      y.z = sm[2] + __builtin_bit_cast(float, static_cast<uint32_t>(s.b2[n0 + 2]) << 16);
      y.w = sm[3] + __builtin_bit_cast(float, static_cast<uint32_t>(s.b2[n0 + 3]) << 16);
      *reinterpret_cast<float4*>(s.y + static_cast<size_t>(b) * s.d + n0) = y;
    }
  }
}

// SIDE: the launch also carries a SideProduct in its workgroups from
// n_blocks on (AttnSideParams); launches without one keep AttnParams and the
// code without the test.
template <int D, int W, bool SIDE = false>
__global__ __launch_bounds__(W * 64) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2)))
void attention_kernel(std::conditional_t<SIDE, AttnSideParams, AttnParams> p) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  constexpr int NT = W * 64;  // threads
  constexpr int D4 = D / 4;    // four-channel groups of a head
  __shared__ AttnShared<D, W> sm;
  if constexpr (SIDE) {
    if (static_cast<int>(blockIdx.x) >= p.n_blocks) {  // a workgroup of the carried product
      static_assert(sizeof(sm.stage) >= 8 * 64 * sizeof(f32x4), "staging area too small");
      side_product<W>(p.side, static_cast<int>(blockIdx.x) - p.n_blocks,
                      reinterpret_cast<f32x4*>(sm.stage));
      return;
    }
  }
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;  // query head inside the group / MFMA row
  const int grp = lane >> 4;  // k-slot group: tokens 8*grp .. 8*grp+7 of a tile
  const int g = blockIdx.x;

  int b, r, j, nb, L, k0, k1;
  const bool single = !p.plan && p.n_blocks == 1 && p.B == 1 && p.n_groups == 1;
  if (p.direct) {
    // One workgroup per (sequence, KV group) unit, in unit order: the run is
    // the whole unit, so no schedule, plan or partials (any batch size).
    b = static_cast<int>(static_cast<unsigned>(g) / static_cast<unsigned>(p.n_groups));
    r = g - b * p.n_groups;
    j = 0;
    nb = 1;
    L = attended_len(p, b);
    k0 = 0;
    k1 = tiles_of(L);
  } else if (p.plan) {  // the step's plan, written by the step's first attention launch
    const RunItem item = reinterpret_cast<const RunItem*>(p.plan)[g];
    if (item.z >= 0)
      for (int i = threadIdx.x; i < p.h * D4; i += NT)
        store_out4<D>(p, static_cast<size_t>(item.z) * p.h, i * 4, f32x4{0.f, 0.f, 0.f, 0.f});
    if (item.b < 0 || item.b >= p.B) return;
    b = item.b;
    r = item.r;
    j = item.j;
    nb = item.nb;
    L = item.L;
    k0 = item.k0;
    k1 = item.k1;
  } else if (single) {
    // One workgroup for one short unit: its run is the whole sequence.  The
    // first tiles are requested for the longest allowed length before the
    // length itself arrives; the length is read below.
    b = r = j = k0 = 0;
    nb = 1;
    L = p.max_len;
    k1 = tiles_of(L);
  } else {
    schedule<NT>(p, sm.sc, sm.run, g);
    // The run item lies outside the schedule's LDS tables, so the waves'
    // merge may overwrite those while other waves still read it.
    const RunItem item = sm.run;
    const int ib = __builtin_amdgcn_readfirstlane(item.b);
    const int iz = __builtin_amdgcn_readfirstlane(item.z);
    if (p.plan_out && threadIdx.x == 0) reinterpret_cast<RunItem*>(p.plan_out)[g] = item;
    if (iz >= 0)
      for (int i = threadIdx.x; i < p.h * D4; i += NT)
        store_out4<D>(p, static_cast<size_t>(iz) * p.h, i * 4, f32x4{0.f, 0.f, 0.f, 0.f});
    if (ib < 0 || ib >= p.B) return;  // no run for this workgroup
    b = ib;
    r = __builtin_amdgcn_readfirstlane(item.r);
    j = __builtin_amdgcn_readfirstlane(item.j);
    nb = __builtin_amdgcn_readfirstlane(item.nb);
    L = __builtin_amdgcn_readfirstlane(item.L);
    k0 = __builtin_amdgcn_readfirstlane(item.k0);
    k1 = __builtin_amdgcn_readfirstlane(item.k1);
  }

  const int kv = p.kv_begin + r;
  const int head0 = r * p.G;
  const size_t seq = static_cast<size_t>(kv) * p.B + b;
  const uint16_t* kbase = p.k + seq * p.S * D;
  const uint16_t* vbase = p.v + seq * p.S * D;

  // This lane's query chunks (channels grp*8 + kk*32 .. +7 of its head; a
  // padded head reads the group's last one and scores zero).  With rotation,
  // also the partner chunks and this sequence's table entries, all in flight
  // together with the first tile.
  const int rope_half = p.rope_cs ? p.rope_half : 0;
  const bool valid = col < p.G;
  const uint16_t* qrow = p.q + (static_cast<size_t>(b) * p.h + head0 + (valid ? col : p.G - 1)) * D;
  u16x8 qraw[KK], qpart[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const int c0 = grp * 8 + kk * 32;
    qraw[kk] = load16(qrow + c0);
    qpart[kk] = c0 < 2 * rope_half ? load16(qrow + partner_chunk(c0, rope_half)) : qraw[kk];
  }
  double2 cs_mine = make_double2(0.0, 0.0);
  if (threadIdx.x < rope_half)
    cs_mine = reinterpret_cast<const double2*>(p.rope_cs)[static_cast<size_t>(b) * rope_half + threadIdx.x];

  Tile<D> ta, tb;
  int it = k0 + wave;
  WaveState<D> st;
  st.den = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int db = 0; db < DB; ++db) st.acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (it < k1) load_tile<D>(ta, kbase, vbase, it * kTile, col, grp);
  if (single) {  // the actual length (the tile above may go unused)
    L = attended_len(p, 0);
    k1 = tiles_of(L);
    if (L == 0) {
      for (int i = threadIdx.x; i < p.h * D4; i += NT)
        store_out4<D>(p, 0, i * 4, f32x4{0.f, 0.f, 0.f, 0.f});
      return;
    }
  }
  auto cs_lds = [&](int jj) { return sm.rope[jj]; };
  if (rope_half) {  // the table to LDS, then the queries rotated in registers
    if (threadIdx.x < rope_half) sm.rope[threadIdx.x] = cs_mine;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qraw[kk] = rotate_chunk(qraw[kk], qpart[kk], grp * 8 + kk * 32, rope_half, cs_lds);
  }
  bf16x8 qf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const u16x8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
    qf[kk] = as_bf16(valid ? qraw[kk] : zero);  // padded heads score zero
  }
  const bool has_tiles = it < k1;

  // Fused append of the owning layer (Section 2.4): the last run of each
  // owned unit writes the newest token's K/V row into slot lens[b] +
  // len_offset - 1 and, when that slot is the last attended position, takes
  // the row from LDS (this kernel's tile loads may not see the write).
  int pos_new = -1;
  if (p.k_new && j == nb - 1 && kv >= p.own_begin && kv < p.own_begin + p.own_count) {
    const int pos = p.lens[b] + p.len_offset - 1;
    if (pos >= 0 && pos < p.S) {
      if (threadIdx.x < D / 8) {
        const int d0 = threadIdx.x * 8;
        const size_t src = static_cast<size_t>(b) * p.new_stride + static_cast<size_t>(kv) * D + d0;
        u16x8 nk = load16(p.k_new + src);
        const u16x8 nv = load16(p.v_new + src);
        if (d0 < 2 * rope_half)
          nk = rotate_chunk(nk, load16(p.k_new + src - d0 + partner_chunk(d0, rope_half)), d0,
                            rope_half, cs_lds);
        uint16_t* kc = const_cast<uint16_t*>(kbase);  // the caller's cache, written here only
        uint16_t* vc = const_cast<uint16_t*>(vbase);
        *reinterpret_cast<u16x8*>(kc + static_cast<size_t>(pos & ~(kTile - 1)) * D +
                                  kchunk<D>(pos & (kTile - 1), d0 / 8) * 8) = nk;
        uint16_t* vdst = vc + static_cast<size_t>(pos & ~(kTile - 1)) * D + (pos & (kTile - 1));
#pragma unroll
        for (int e = 0; e < 8; ++e) vdst[(d0 + e) * kTile] = nv[e];
        *reinterpret_cast<u16x8*>(&sm.new_row[d0]) = nk;
        *reinterpret_cast<u16x8*>(&sm.new_row[D + d0]) = nv;
      }
      if (pos == L - 1) {
        pos_new = pos;
        __syncthreads();  // the staged row is visible to every wave
      }
    }
  }

  // The loads of tile it+W are issued before tile it is consumed (two
  // register buffers); the wave's last tile is processed after the loop,
  // with the ragged-end mask and the newest token.
  if (has_tiles) {
    for (;;) {
      const int nxt = it + W;
      if (nxt >= k1) break;  // ta holds the last tile
      load_tile<D>(tb, kbase, vbase, nxt * kTile, col, grp);
      process_tile<D, false>(st, ta, qf, it * kTile, L, col, grp, p.scale_log2, -1, nullptr);
      it = nxt;
      const int nx2 = it + W;
      if (nx2 >= k1) {  // tb holds the last tile
        ta = tb;
        break;
      }
      load_tile<D>(ta, kbase, vbase, nx2 * kTile, col, grp);
      process_tile<D, false>(st, tb, qf, it * kTile, L, col, grp, p.scale_log2, -1, nullptr);
      it = nx2;
    }
    process_tile<D, true>(st, ta, qf, it * kTile, L, col, grp, p.scale_log2, pos_new,
                          sm.new_row);
  }

  // Merge the four waves through LDS.
  if (grp == 0) {
    sm.m[wave][col] = st.m;
    sm.l[wave][col] = st.den[0];
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
    *reinterpret_cast<f32x4*>(&sm.acc[wave][col][db * 16 + grp * 4]) = st.acc[db];
  __syncthreads();

  const int GD = p.G * D;
  const size_t out_row0 = static_cast<size_t>(b) * p.h + head0;
  const size_t unit = static_cast<size_t>(b) * p.n_groups + r;
  const size_t slot = unit * p.max_parts + j;
  const bool fuse = nb > 1 && p.fused && nb * GD <= kStageFloats && nb * p.G * 2 <= kStageMl;
  // The unit's partial outputs ([run][head][channel], nb * GD floats), for
  // the in-place merge.
  float* const unit_acc = fuse ? p.part_acc + unit * p.max_parts * GD : p.part_acc;
  const __amdgpu_buffer_rsrc_t rsrc_acc =
      device_rsrc(unit_acc, fuse ? static_cast<uint32_t>(nb * GD * 4) : 0u);
  // Each thread merges four channels of one head over the waves.
  for (int idx = threadIdx.x; idx < p.G * D4; idx += NT) {
    const int hh = idx / D4;
    const int d = (idx - hh * D4) * 4;
    float mw[W];
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      mw[w] = sm.m[w][hh];
      M = fmaxf(M, mw[w]);
    }
    float wsum = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const float f = fast_exp2(mw[w] - M);
        wsum += f * sm.l[w][hh];
        o += f * *reinterpret_cast<const f32x4*>(&sm.acc[w][hh][d]);
      }
    }
    if (nb == 1) {
      store_out4<D>(p, out_row0 + hh, d, normalize4(o, wsum));
    } else if (fuse) {
      store4_device(rsrc_acc, (j * GD + hh * D + d) * 4, o);
      if (d == 0) {
        store_device(&p.part_ml[(slot * p.G + hh) * 2 + 0], M);
        store_device(&p.part_ml[(slot * p.G + hh) * 2 + 1], wsum);
      }
    } else {
      *reinterpret_cast<f32x4*>(&p.part_acc[slot * GD + hh * D + d]) = o;
      if (d == 0) {
        p.part_ml[(slot * p.G + hh) * 2 + 0] = M;
        p.part_ml[(slot * p.G + hh) * 2 + 1] = wsum;
      }
    }
  }
  if (!fuse) return;

  // ---- the last run of the unit to finish merges its runs in place ----
  wait_stores_complete();  // this thread's partials are visible device-wide
  __syncthreads();         // ... and those of every thread; LDS merge data is dead
  if (threadIdx.x == 0)
    sm.last = __hip_atomic_fetch_add(&p.counters[unit], 1, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == nb - 1;
  __syncthreads();
  if (!sm.last) return;
  // Every other run bumped the counter after its partials completed, so the
  // device-scope loads below see them.  The unit's partials are contiguous
  // ([run][head][channel]); stage them with all loads in flight, then merge
  // in ascending run order (deterministic).
  {
    // One round trip: every 16-byte piece of the unit's partials is in
    // flight at once (kStageFloats / 4 / NT pieces per thread at most).
    constexpr int kPieces = (kStageFloats / 4 + NT - 1) / NT;
    const int n4 = nb * GD / 4;
    f32x4 v[kPieces];
#pragma unroll
    for (int u = 0; u < kPieces; ++u) {
      const int i4 = threadIdx.x + u * NT;
      v[u] = i4 < n4 ? load4_device(rsrc_acc, i4 * 16) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int n_ml = nb * p.G * 2;
    float* src_ml = p.part_ml + unit * p.max_parts * p.G * 2;
    float ml[(kStageMl + NT - 1) / NT];
#pragma unroll
    for (int u = 0; u < (kStageMl + NT - 1) / NT; ++u) {
      const int jj = threadIdx.x + u * NT;
      ml[u] = jj < n_ml ? load_device(src_ml + jj) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kPieces; ++u) {
      const int i4 = threadIdx.x + u * NT;
      if (i4 < n4) *reinterpret_cast<f32x4*>(&sm.stage[i4 * 4]) = v[u];
    }
#pragma unroll
    for (int u = 0; u < (kStageMl + NT - 1) / NT; ++u) {
      const int jj = threadIdx.x + u * NT;
      if (jj < n_ml) sm.stage_ml[jj] = ml[u];
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < p.G * D4; idx += NT) {
    const int hh = idx / D4;
    const int d = (idx - hh * D4) * 4;
    float M = -INFINITY;
    for (int s2 = 0; s2 < nb; ++s2) M = fmaxf(M, sm.stage_ml[(s2 * p.G + hh) * 2]);
    float den = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    if (M != -INFINITY) {
      for (int s2 = 0; s2 < nb; ++s2) {
        const float f = fast_exp2(sm.stage_ml[(s2 * p.G + hh) * 2] - M);
        den += f * sm.stage_ml[(s2 * p.G + hh) * 2 + 1];
        o += f * *reinterpret_cast<const f32x4*>(&sm.stage[s2 * GD + hh * D + d]);
      }
    }
    store_out4<D>(p, out_row0 + hh, d, normalize4(o, den));
  }
  if (threadIdx.x == 0)  // ready for the next call on this workspace
    __hip_atomic_store(&p.counters[unit], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge of the partials of units cut into several runs (and zero
// output for empty sequences).  A (sequence, query head) row is merged by
// p.merge_waves waves (1 or 4).  Inside a wave, lane (sub, c) reads channels
// 4c..4c+3 of partials sub, sub + SP, ... (SP = 256 / D partials side by side),
// 16 partials per wave per round trip; the first round is issued before the
// run count arrives (slots past it are ignored).  Sub-streams are merged with
// shuffles, waves through LDS, always in the same order (deterministic).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void combine_kernel(AttnParams p) {
  constexpr int CL = D / 4;   // lanes covering one partial (a float4 each)
  constexpr int SP = 64 / CL;  // partials a wave reads side by side
  constexpr int U = 16 / SP;   // partials per lane per round trip
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wpr = p.merge_waves;  // waves per row: 1 or kWaves
  const int rows_per_block = kWaves / wpr;
  const int wr = wave % wpr;      // wave index inside its row
  const size_t row = static_cast<size_t>(blockIdx.x) * rows_per_block + wave / wpr;
  const bool row_ok = row < static_cast<size_t>(p.B) * p.h;
  const size_t rrow = row_ok ? row : 0;
  const int b = static_cast<int>(rrow / p.h);
  const int i = static_cast<int>(rrow - static_cast<size_t>(b) * p.h);
  const int r = i / p.G;
  const int hh = i - r * p.G;
  const int sub = lane / CL;
  const int c = (lane - sub * CL) * 4;
  const int GD = p.G * D;
  const size_t base = (static_cast<size_t>(b) * p.n_groups + r) * p.max_parts;
  const int stride = wpr * SP;  // partial index step between a lane's consecutive reads
  const int first = wr * SP + sub;

  float m[U], w[U];
  f32x4 a[U];
  auto load_round = [&](int s0, int ns) {  // lanes past ns load nothing
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + first + u * stride;
      m[u] = -INFINITY;
      w[u] = 0.f;
      a[u] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (s < ns) {
        const size_t slot = base + s;
        m[u] = p.part_ml[(slot * p.G + hh) * 2];
        w[u] = p.part_ml[(slot * p.G + hh) * 2 + 1];
        a[u] = *reinterpret_cast<const f32x4*>(&p.part_acc[slot * GD + hh * D + c]);
      }
    }
  };
  // First round before the run count is known, over the slots the launch
  // expects to be used (p.merge_first <= max_parts: inside the workspace).
  load_round(0, p.merge_first);
  const int ns = row_ok ? p.runs[b] : 0;  // runs of each unit of sequence b
  const bool merged_in_place =
      ns == 1 || (p.fused && ns * p.G * D <= kStageFloats && ns * p.G * 2 <= kStageMl);
  if (!row_ok || merged_in_place) return;  // uniform per row: all its waves leave
  if (ns == 0) {                           // nothing to attend: zero output
    if (wr == 0 && sub == 0) store_out4<D>(p, rrow, c, f32x4{0.f, 0.f, 0.f, 0.f});
    return;
  }

  float run_m = -INFINITY, run_den = 0.f;
  f32x4 run_o = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0;;) {
#pragma unroll
    for (int u = 0; u < U; ++u) {  // drop speculative slots at or past ns
      const bool ok = s0 + first + u * stride < ns;
      m[u] = ok ? m[u] : -INFINITY;
      w[u] = ok ? w[u] : 0.f;
      a[u] = ok ? a[u] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float bm = run_m;
#pragma unroll
    for (int u = 0; u < U; ++u) bm = fmaxf(bm, m[u]);
    if (bm != -INFINITY) {
      const float sc = fast_exp2(run_m - bm);  // 0 while nothing is accumulated
      run_den *= sc;
      run_o *= sc;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float f = fast_exp2(m[u] - bm);
        run_den += f * w[u];
        run_o += f * a[u];
      }
      run_m = bm;
    }
    s0 += U * stride;
    if (s0 >= ns) break;
    load_round(s0, ns);
  }

  // Merge the SP sub-streams of the wave (lanes CL apart).
  float M = run_m;
#pragma unroll
  for (int off = CL; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
  const float f = run_m == -INFINITY ? 0.f : fast_exp2(run_m - M);
  float den = f * run_den;
  f32x4 o = f * run_o;
#pragma unroll
  for (int off = CL; off < 64; off <<= 1) {
    den += __shfl_xor(den, off);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] += __shfl_xor(o[e], off);
  }
  if (wpr == 1) {
    if (sub == 0) store_out4<D>(p, rrow, c, normalize4(o, den));
    return;
  }
  // Several waves per row (one row per workgroup): merge through LDS.
  __shared__ float sm_m[kWaves], sm_den[kWaves];
  __shared__ f32x4 sm_o[kWaves][CL];
  if (lane == 0) {
    sm_m[wave] = M;
    sm_den[wave] = den;
  }
  if (sub == 0) sm_o[wave][lane] = o;
  __syncthreads();
  if (wave == 0 && sub == 0) {
    float MM = -INFINITY;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) MM = fmaxf(MM, sm_m[v]);
    float dd = 0.f;
    f32x4 oo = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      const float fv = sm_m[v] == -INFINITY ? 0.f : fast_exp2(sm_m[v] - MM);
      dd += fv * sm_den[v];
      oo += fv * sm_o[v][lane];
    }
    store_out4<D>(p, rrow, c, dd != 0.f ? oo / dd : f32x4{0.f, 0.f, 0.f, 0.f});
  }
}

__global__ void fill_kernel(uint32_t* dst, size_t n, uint32_t value) {
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    dst[i] = value;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_append(const AppendParams& p, int head_dim, int owned_count,
                         hipStream_t stream) {
  const dim3 grid(p.B, owned_count);
  if (head_dim == 64)
    hipLaunchKernelGGL(append_kernel<64>, grid, dim3(64 / 8), 0, stream, p);
  else
    hipLaunchKernelGGL(append_kernel<128>, grid, dim3(128 / 8), 0, stream, p);
  return hipGetLastError();
}

template <int D, int W>
static void launch_attention_t(const AttnParams& p, const SideProduct* side, hipStream_t stream,
                               hipEvent_t start, hipEvent_t stop) {
  const dim3 block(W * 64);
  if (side && side->n_blocks > 0) {
    AttnSideParams ps;
    static_cast<AttnParams&>(ps) = p;
    ps.side = *side;
    const dim3 grid(p.n_blocks + side->n_blocks);
    auto kernel = attention_kernel<D, W, true>;
    if (start)
      hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, start, stop, 0, ps);
    else
      hipLaunchKernelGGL(kernel, grid, block, 0, stream, ps);
    return;
  }
  const dim3 grid(p.n_blocks);
  auto kernel = attention_kernel<D, W>;
  if (start)  // timed: events recorded with the dispatch itself
    hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, start, stop, 0, p);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, p);
}

hipError_t launch_attention_main(const AttnParams& p, int head_dim, hipStream_t stream,
                                 hipEvent_t start, hipEvent_t stop, const SideProduct* side) {
  const bool wide = p.waves == kWideWaves;
  if (head_dim == 64) {
    if (wide)
      launch_attention_t<64, kWideWaves>(p, side, stream, start, stop);
    else
      launch_attention_t<64, kWaves>(p, side, stream, start, stop);
  } else {
    if (wide)
      launch_attention_t<128, kWideWaves>(p, side, stream, start, stop);
    else
      launch_attention_t<128, kWaves>(p, side, stream, start, stop);
  }
  return hipGetLastError();
}

hipError_t launch_attention_merge(const AttnParams& p, int head_dim, hipStream_t stream,
                                  hipEvent_t stop) {
  if (p.n_blocks == 1) return hipSuccess;  // every unit is finished in place
  const int rows_per_block = kWaves / p.merge_waves;
  const dim3 cgrid((p.B * p.h + rows_per_block - 1) / rows_per_block);
  auto kernel = head_dim == 64 ? combine_kernel<64> : combine_kernel<128>;
  if (stop)
    hipExtLaunchKernelGGL(kernel, cgrid, dim3(kThreads), 0, stream, nullptr, stop, 0, p);
  else
    hipLaunchKernelGGL(kernel, cgrid, dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

int max_batch() { return kMaxBatch; }
int stage_floats() { return kStageFloats; }

int compute_units() {
  static std::atomic<int> cached{-1};
  int v = cached.load(std::memory_order_relaxed);
  if (v >= 0) return v;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  cached.store(cus, std::memory_order_relaxed);
  return cus;
}

int wide_waves() { return kWideWaves; }
int default_waves() { return kWaves; }

int resident_workgroups(int head_dim) {
  static std::atomic<int> cached[2] = {{-1}, {-1}};
  std::atomic<int>& slot = cached[head_dim == 64 ? 0 : 1];
  int v = slot.load(std::memory_order_relaxed);
  if (v >= 0) return v;
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const hipError_t err =
      head_dim == 64
          ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attention_kernel<64, kWaves>, kThreads, 0)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attention_kernel<128, kWaves>, kThreads, 0);
  if (err != hipSuccess) return 0;
  v = cus * per_cu;
  slot.store(v, std::memory_order_relaxed);
  return v;
}

hipError_t launch_rope_table(const RopeTableParams& p, hipStream_t stream) {
  const int items = p.B * p.half;
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3((items + kRopeThreads - 1) / kRopeThreads),
                     dim3(kRopeThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_cache_rows(const CacheRowsParams& p, int head_dim, hipStream_t stream) {
  const size_t blocks = static_cast<size_t>(p.kv_count) * p.B * (p.S / kTile);
  if (blocks == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(blocks));
  if (head_dim == 64)
    hipLaunchKernelGGL(cache_rows_kernel<64>, grid, dim3(kRowsThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(cache_rows_kernel<128>, grid, dim3(kRowsThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_fill(uint32_t* dst, size_t n_words, uint32_t value, hipStream_t stream) {
  if (n_words == 0) return hipSuccess;
  size_t blocks = (n_words + 255) / 256;
  blocks = blocks > 1024 ? 1024 : blocks;
  hipLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, dst,
                     n_words, value);
  return hipGetLastError();
}

}  // namespace mlkv
