// HIP kernels of MLKV decode attention for CDNA4 (gfx950, wave64, MFMA).
//
//   append_kernel     newest token's K/V rows -> cache slot (bit copy)
//   attention_kernel  split-K attention of one layer: each workgroup owns one
//                     (sequence, KV head, token range) and serves every query
//                     head mapped to that KV head from one pass over the range;
//                     the last workgroup of a sequence to finish merges the
//                     split partials (log-sum-exp) and writes the output
//   fill_kernel       zeroes the workspace's split counters
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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace mlkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 32;     // tokens per wave iteration
constexpr int kWaves = 4;     // waves per workgroup
constexpr int kThreads = kWaves * 64;
constexpr int kMaxSplits = 256;  // most splits one sequence may have (host plans within it)
// The last workgroup of a sequence merges the splits itself when their partial
// outputs fit in LDS (kFusedPartialFloats floats); otherwise combine_kernel runs.
constexpr int kFusedPartialFloats = 8192;
constexpr int kStageBatch = 32;  // partial loads in flight per thread while staging
template <int D>
constexpr int kLdsFloats = (kWaves * 16 * (D + 4)) > kFusedPartialFloats ? (kWaves * 16 * (D + 4))
                                                                         : kFusedPartialFloats;

__device__ __forceinline__ u16x8 load16(const uint16_t* p) {
  return *reinterpret_cast<const u16x8*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16(u16x8 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Device-scope (all XCDs) stores and loads of the split partials.  On CDNA3/4
// the scope travels with each access (SC bits), so partials written and read
// this way need no L2 writeback or invalidate, only completion of the stores
// before the split counter is bumped.
__device__ __forceinline__ void store_device(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_device(float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wait_stores_complete() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t u) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(u) << 16);
}

// Attended length of sequence b (clamped to the cache and to the split grid).
__device__ __forceinline__ int attended_len(const AttnParams& p, int b) {
  int L = p.lens[b] + p.len_offset;
  L = L < 0 ? 0 : L;
  L = L > p.S ? p.S : L;
  const int cap = p.n_split * p.tiles_per_split * kTile;
  return L > cap ? cap : L;
}

// ---------------------------------------------------------------------------
// Cache append (Section 2.4): one workgroup per (sequence b, owned head c),
// one thread per 8 channels.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(D / 8) void append_kernel(AppendParams p) {
  const int b = blockIdx.x;
  const int c = blockIdx.y;
  const int pos = p.positions[b];
  if (pos < 0 || pos >= p.S) return;
  const int d0 = threadIdx.x * 8;
  const size_t src = static_cast<size_t>(b) * p.row_stride + static_cast<size_t>(c) * D + d0;
  const u16x8 kv_k = load16(p.k_new + src);
  const u16x8 kv_v = load16(p.v_new + src);
  const size_t seq = static_cast<size_t>(p.kv_begin + c) * p.B + b;
  *reinterpret_cast<u16x8*>(p.k + (seq * p.S + pos) * D + d0) = kv_k;
  uint16_t* vdst = p.v + (seq * p.S + (pos & ~(kTile - 1))) * D + (pos & (kTile - 1));
#pragma unroll
  for (int e = 0; e < 8; ++e) vdst[(d0 + e) * kTile] = kv_v[e];
}

// ---------------------------------------------------------------------------
// Split-K attention with in-kernel combine.
// Grid: x = split, y = sequence * n_groups + group.
// ---------------------------------------------------------------------------
template <int D>
struct Tile {
  static constexpr int KK = D / 32;  // k-steps of the q.K product
  static constexpr int DB = D / 16;  // 16-channel blocks of the output
  u16x8 k[2][KK];                    // key rows of the two 16-token score blocks
  u16x8 v[DB];                       // value rows of V^T
};

// Score block sb, MFMA row rr holds token 8*(rr/4) + 4*sb + rr%4, so the result
// lane (col, grp) ends up with tokens 8*grp + 4*sb + i: the P^T k-slots it owns.
template <int D>
__device__ __forceinline__ void load_tile(Tile<D>& t, const uint16_t* kbase,
                                          const uint16_t* vbase, int t0, int col, int grp) {
#pragma unroll
  for (int sb = 0; sb < 2; ++sb) {
    const int tok = t0 + (col >> 2) * 8 + sb * 4 + (col & 3);
    const uint16_t* krow = kbase + static_cast<size_t>(tok) * D + grp * 8;
#pragma unroll
    for (int kk = 0; kk < Tile<D>::KK; ++kk) t.k[sb][kk] = load16(krow + kk * 32);
  }
  const uint16_t* vblk = vbase + static_cast<size_t>(t0) * D + grp * 8;
#pragma unroll
  for (int db = 0; db < Tile<D>::DB; ++db) t.v[db] = load16(vblk + (db * 16 + col) * kTile);
}

template <int D>
struct WaveState {
  float m = -INFINITY;  // running max of this lane's head (log2 domain)
  float l = 0.f;        // this lane's share of the running denominator
  f32x4 acc[Tile<D>::DB];
};

template <int D>
__device__ __forceinline__ void process_tile(WaveState<D>& st, Tile<D>& t, const bf16x8* qf,
                                             int t0, int L, int grp, float scale_log2) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  f32x4 s[2];
#pragma unroll
  for (int sb = 0; sb < 2; ++sb) {
    s[sb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) s[sb] = mfma_bf16(as_bf16(t.k[sb][kk]), qf[kk], s[sb]);
  }
  float x[8];
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int i = 0; i < 4; ++i) x[sb * 4 + i] = s[sb][i] * scale_log2;

  if (t0 + kTile > L) {  // ragged tail: positions >= L take no weight and no value
    const int first = t0 + grp * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (first + e >= L) {
        x[e] = -INFINITY;
#pragma unroll
        for (int db = 0; db < DB; ++db) t.v[db][e] = 0;
      }
    }
  }

  float tmax = x[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) tmax = fmaxf(tmax, x[e]);
  tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
  tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
  const float m_new = fmaxf(st.m, tmax);
  const float alpha = fast_exp2(st.m - m_new);

  u16x8 pbits;
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint16_t pb = f32_to_bf16_bits(fast_exp2(x[e] - m_new));
    pbits[e] = pb;
    psum += bf16_bits_to_f32(pb);  // denominator from the rounded weights
  }
  st.l = st.l * alpha + psum;
  st.m = m_new;
  const bf16x8 pf = as_bf16(pbits);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    st.acc[db] *= alpha;
    st.acc[db] = mfma_bf16(as_bf16(t.v[db]), pf, st.acc[db]);
  }
}

template <int D>
__device__ __forceinline__ void store_out(const AttnParams& p, size_t row, int d, float val) {
  if (p.out_bf16)
    static_cast<uint16_t*>(p.out)[row * D + d] = f32_to_bf16_bits(val);
  else
    static_cast<float*>(p.out)[row * D + d] = val;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

template <int D>
__global__ __launch_bounds__(kThreads) void attention_kernel(AttnParams p) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  constexpr int LDS_STRIDE = D + 4;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;  // query head inside the group / MFMA row
  const int grp = lane >> 4;  // k-slot group: tokens 8*grp .. 8*grp+7 of a tile

  // Grid x runs over (sequence, KV head) units and y over splits, so the
  // dispatcher hands out every sequence's first splits before any later
  // split: workgroups of splits past a sequence's end come last and leave at
  // once.  Consecutive units land on different XCDs, and all splits of one
  // unit share an XCD (workgroup id modulo 8), keeping its partials in one L2.
  const int unit = blockIdx.x;
  const int split = blockIdx.y;
  const int b = unit / p.n_groups;
  const int r = unit - b * p.n_groups;
  const int kv = p.kv_begin + r;
  const int head0 = r * p.G;
  const int chunk = p.tiles_per_split * kTile;
  const int t_begin = split * chunk;

  const size_t seq = static_cast<size_t>(kv) * p.B + b;
  const uint16_t* kbase = p.k + seq * p.S * D;
  const uint16_t* vbase = p.v + seq * p.S * D;

  // The query loads go out before the sequence length is known.
  Tile<D> ta, tb;
  bf16x8 qf[KK];
  {
    const bool valid = col < p.G;
    const uint16_t* qrow =
        p.q + (static_cast<size_t>(b) * p.h + head0 + (valid ? col : p.G - 1)) * D + grp * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      u16x8 v = load16(qrow + kk * 32);
      const u16x8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
      qf[kk] = as_bf16(valid ? v : zero);  // padded heads score zero
    }
  }

  const int L = attended_len(p, b);
  int ns = (L + chunk - 1) / chunk;  // active splits of this sequence
  ns = ns < 1 ? 1 : ns;
  if (split >= ns) return;  // empty split: nothing to contribute
  int n_tiles = (L - t_begin + kTile - 1) / kTile;
  n_tiles = n_tiles < 0 ? 0 : (n_tiles > p.tiles_per_split ? p.tiles_per_split : n_tiles);

  WaveState<D> st;
#pragma unroll
  for (int db = 0; db < DB; ++db) st.acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Two tile buffers: the loads of tile it+kWaves are issued before tile it
  // is consumed.  The prefetch is never skipped (past the last tile it re-reads
  // the current, cache-resident tile) so that the wait before each tile only
  // covers that tile's own loads.
  int it = wave;
  if (it < n_tiles) {
    load_tile(ta, kbase, vbase, t_begin + it * kTile, col, grp);
    for (;;) {
      int nxt = it + kWaves;
      load_tile(tb, kbase, vbase, t_begin + (nxt < n_tiles ? nxt : it) * kTile, col, grp);
      process_tile(st, ta, qf, t_begin + it * kTile, L, grp, p.scale_log2);
      it = nxt;
      if (it >= n_tiles) break;
      nxt = it + kWaves;
      load_tile(ta, kbase, vbase, t_begin + (nxt < n_tiles ? nxt : it) * kTile, col, grp);
      process_tile(st, tb, qf, t_begin + it * kTile, L, grp, p.scale_log2);
      it = nxt;
      if (it >= n_tiles) break;
    }
  }

  // ---- merge the four waves of the workgroup through LDS ----
  // sm_buf first holds the four waves' accumulators, later (last workgroup of
  // a sequence only) the staged partials of every split.
  __shared__ float sm_buf[kLdsFloats<D>];
  __shared__ float sm_m[kWaves][16];
  __shared__ float sm_l[kWaves][16];
  __shared__ float sm_ml[kFusedPartialFloats / 8];
  __shared__ int sm_last;
  float(*sm_acc)[16][LDS_STRIDE] = reinterpret_cast<float(*)[16][LDS_STRIDE]>(sm_buf);
  float l_tot = st.l + __shfl_xor(st.l, 16);
  l_tot += __shfl_xor(l_tot, 32);
  if (grp == 0) {
    sm_m[wave][col] = st.m;
    sm_l[wave][col] = l_tot;
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
    *reinterpret_cast<f32x4*>(&sm_acc[wave][col][db * 16 + grp * 4]) = st.acc[db];
  __syncthreads();

  const int GD = p.G * D;
  const size_t out_row0 = static_cast<size_t>(b) * p.h + head0;
  const size_t slot = static_cast<size_t>(unit) * p.n_split + split;
  for (int idx = threadIdx.x; idx < GD; idx += kThreads) {
    const int hh = idx / D;
    const int d = idx - hh * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm_m[w][hh]);
    float wsum = 0.f, o = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float f = fast_exp2(sm_m[w][hh] - M);
        wsum += f * sm_l[w][hh];
        o += f * sm_acc[w][hh][d];
      }
    }
    if (ns == 1) {
      store_out<D>(p, out_row0 + hh, d, wsum > 0.f ? o / wsum : 0.f);
    } else {
      store_device(&p.part_acc[slot * GD + idx], o);
      if (d == 0) {
        store_device(&p.part_ml[(slot * p.G + hh) * 2 + 0], M);
        store_device(&p.part_ml[(slot * p.G + hh) * 2 + 1], wsum);
      }
    }
  }
  if (ns == 1 || !p.fused_combine) return;

  // ---- split-K combine by the last workgroup of this sequence to finish ----
  wait_stores_complete();  // this thread's partials are visible device-wide
  __syncthreads();         // ... and so are those of every thread of the workgroup
  if (threadIdx.x == 0)
    sm_last = __hip_atomic_fetch_add(&p.counters[unit], 1, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT) == ns - 1;
  __syncthreads();
  if (!sm_last) return;
  // Every other split bumped the counter after its partials completed, so the
  // device-scope loads below see them.  The sequence's partials are one
  // contiguous range [split][head][channel]: stage them in LDS with all loads
  // in flight at once, then merge in ascending split order (deterministic).
  const size_t base = static_cast<size_t>(unit) * p.n_split;
  {
    const int n_acc = ns * GD;
    const int n_ml = ns * p.G * 2;
    float* src_acc = p.part_acc + base * GD;
    float* src_ml = p.part_ml + base * p.G * 2;
    for (int j0 = threadIdx.x; j0 < n_acc; j0 += kThreads * kStageBatch) {
      float v[kStageBatch];
#pragma unroll
      for (int u = 0; u < kStageBatch; ++u) {
        const int j = j0 + u * kThreads;
        v[u] = j < n_acc ? load_device(src_acc + j) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kStageBatch; ++u) {
        const int j = j0 + u * kThreads;
        if (j < n_acc) sm_buf[j] = v[u];
      }
    }
    for (int j = threadIdx.x; j < n_ml; j += kThreads) sm_ml[j] = load_device(src_ml + j);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < GD; idx += kThreads) {
    const int hh = idx / D;
    float M = -INFINITY;
    for (int s = 0; s < ns; ++s) M = fmaxf(M, sm_ml[(s * p.G + hh) * 2]);
    float den = 0.f, o = 0.f;
    if (M != -INFINITY) {
      for (int s = 0; s < ns; ++s) {
        const float f = fast_exp2(sm_ml[(s * p.G + hh) * 2] - M);
        den += f * sm_ml[(s * p.G + hh) * 2 + 1];
        o += f * sm_buf[s * GD + idx];
      }
    }
    store_out<D>(p, out_row0 + hh, idx - hh * D, den > 0.f ? o / den : 0.f);
  }
  if (threadIdx.x == 0)  // ready for the next call on this workspace
    __hip_atomic_store(&p.counters[unit], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Separate log-sum-exp combine for sequences with many splits: one workgroup
// of four waves per (sequence, query head).  Wave w reads splits w, w+4, ...
// eight at a time (max, denominator and channels in one round trip) and keeps
// a running merge; the four waves then merge through LDS.  Fixed order.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void combine_kernel(AttnParams p) {
  constexpr int C = D / 64;  // channels per lane
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const size_t row = blockIdx.x;  // b * h + i
  const int b = static_cast<int>(row / p.h);
  const int i = static_cast<int>(row - static_cast<size_t>(b) * p.h);
  const int r = i / p.G;
  const int hh = i - r * p.G;
  const int unit = b * p.n_groups + r;
  const int L = attended_len(p, b);
  const int chunk = p.tiles_per_split * kTile;
  const int ns = (L + chunk - 1) / chunk;
  if (ns <= 1) return;  // one split: the attention kernel wrote the output itself
  const size_t base = static_cast<size_t>(unit) * p.n_split;
  const int GD = p.G * D;

  float run_m = -INFINITY, run_den = 0.f, run_o[C];
#pragma unroll
  for (int k = 0; k < C; ++k) run_o[k] = 0.f;
  for (int s0 = wave; s0 < ns; s0 += kWaves * 8) {
    float m[8], w[8], a[8][C];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int s = s0 + u * kWaves;
      const bool ok = s < ns;
      const size_t slot = base + (ok ? s : 0);
      m[u] = ok ? p.part_ml[(slot * p.G + hh) * 2] : -INFINITY;
      w[u] = ok ? p.part_ml[(slot * p.G + hh) * 2 + 1] : 0.f;
#pragma unroll
      for (int k = 0; k < C; ++k) a[u][k] = ok ? p.part_acc[slot * GD + hh * D + lane + 64 * k] : 0.f;
    }
    float bm = run_m;
#pragma unroll
    for (int u = 0; u < 8; ++u) bm = fmaxf(bm, m[u]);
    if (bm == -INFINITY) continue;
    const float sc = fast_exp2(run_m - bm);
    run_den *= sc;
#pragma unroll
    for (int k = 0; k < C; ++k) run_o[k] *= sc;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float f = fast_exp2(m[u] - bm);
      run_den += f * w[u];
#pragma unroll
      for (int k = 0; k < C; ++k) run_o[k] += f * a[u][k];
    }
    run_m = bm;
  }
  __shared__ float sm_m[kWaves], sm_den[kWaves], sm_o[kWaves][D];
  if (lane == 0) {
    sm_m[wave] = run_m;
    sm_den[wave] = run_den;
  }
#pragma unroll
  for (int k = 0; k < C; ++k) sm_o[wave][lane + 64 * k] = run_o[k];
  __syncthreads();
  if (wave == 0) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm_m[w]);
    float f[kWaves], den = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      f[w] = M == -INFINITY ? 0.f : fast_exp2(sm_m[w] - M);
      den += f[w] * sm_den[w];
    }
#pragma unroll
    for (int k = 0; k < C; ++k) {
      const int d = lane + 64 * k;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += f[w] * sm_o[w][d];
      store_out<D>(p, row, d, den > 0.f ? v / den : 0.f);
    }
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

int fused_partial_capacity() { return kFusedPartialFloats; }

hipError_t launch_attention(const AttnParams& p, int head_dim, hipStream_t stream) {
  const dim3 grid(p.B * p.n_groups, p.n_split);
  if (head_dim == 64)
    hipLaunchKernelGGL(attention_kernel<64>, grid, dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(attention_kernel<128>, grid, dim3(kThreads), 0, stream, p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.n_split == 1 || p.fused_combine) return err;
  const dim3 cgrid(p.B * p.h);
  if (head_dim == 64)
    hipLaunchKernelGGL(combine_kernel<64>, cgrid, dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(combine_kernel<128>, cgrid, dim3(kThreads), 0, stream, p);
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
