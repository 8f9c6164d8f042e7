// Device helpers shared by the decode and prefill kernels (gfx950, wave64):
// vector types, MFMA and conversion wrappers, and the wave-level tile
// arithmetic of attention (one 32-token tile of keys/values against 16 query
// columns).  Included by kernels.hip, prefill.hip and model.hip only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace mlkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 32;     // tokens per wave iteration
constexpr int kWaves = 4;      // waves per workgroup (split runs, merge kernel)
constexpr int kThreads = kWaves * 64;
constexpr int kWideWaves = 8;  // waves per workgroup when each unit is one run
constexpr int kMaxBatch = 2048;  // sequences one call may hold (schedule tables in LDS)

__device__ __forceinline__ u16x8 load16(const uint16_t* p) {
  return *reinterpret_cast<const u16x8*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16(u16x8 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Device-scope (all XCDs) stores and loads for partials merged inside the
// attention kernel: on CDNA3/4 the scope travels with each access (SC bits),
// so no L2 writeback or invalidate is needed, only completion of the stores
// before the unit's counter is bumped.
__device__ __forceinline__ void store_device(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_device(float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wait_stores_complete() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// 16-byte device-scope (sc1) accesses through a buffer resource over `bytes`
// bytes at `base` (offsets are 32-bit; out-of-range accesses are dropped).
constexpr int kCpolDevice = 16;  // sc1: coherent across XCDs
__device__ __forceinline__ __amdgpu_buffer_rsrc_t device_rsrc(float* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, bytes, 0x00020000);
}
__device__ __forceinline__ void store4_device(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, kCpolDevice);
}
__device__ __forceinline__ f32x4 load4_device(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCpolDevice));
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// ---------------------------------------------------------------------------
// One 32-token tile of keys/values against 16 query columns (a wave).
// ---------------------------------------------------------------------------
// Key plane: each 32-token tile keeps, for each of its two 16-token score
// blocks and each 32-channel k-step, the 64 lanes' MFMA operands contiguous
// (1 KB per block and k-step; lane 16 g + r holds channels 8 g .. 8 g + 7 of
// the step for the block's row r).  The 16-byte chunk of tile token u (0 ..
// 31) with channels 8c .. 8c + 7, so that one load instruction of a wave
// reads 1 KB in one piece:
template <int D>
__device__ __forceinline__ int kchunk(int u, int c) {
  return ((((u >> 2) & 1) * (D / 32) + (c >> 2)) * 64) + (c & 3) * 16 + ((u >> 3) << 2) + (u & 3);
}
template <int D>
struct Tile {
  static constexpr int KK = D / 32;  // k-steps of the q.K product
  static constexpr int DB = D / 16;  // 16-channel blocks of the output
  u16x8 k[2][KK];                    // key rows of the two 16-token score blocks
  u16x8 v[DB];                       // value rows of V^T
};

// Score block sb, MFMA row rr holds token 8*(rr/4) + 4*sb + rr%4, so the result
// lane (col, grp) ends up with tokens 8*grp + 4*sb + i: the P^T k-slots it owns.
//
template <int D>
__device__ __forceinline__ void load_tile(Tile<D>& t, const uint16_t* kbase,
                                          const uint16_t* vbase, int t0, int col, int grp) {
  // The key operands: one contiguous 1 KB piece per score block and k-step.
  const uint16_t* kt = kbase + static_cast<size_t>(t0) * D + (grp * 16 + col) * 8;
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int kk = 0; kk < Tile<D>::KK; ++kk) t.k[sb][kk] = load16(kt + (sb * Tile<D>::KK + kk) * 512);
  const uint16_t* vblk = vbase + static_cast<size_t>(t0) * D + grp * 8;
#pragma unroll
  for (int db = 0; db < Tile<D>::DB; ++db) t.v[db] = load16(vblk + (db * 16 + col) * kTile);
}

template <int D>
struct WaveState {
  float m = -INFINITY;  // reference max of this lane's head (log2 domain)
  f32x4 den;            // softmax denominator of this lane's head (all four equal)
  f32x4 acc[Tile<D>::DB];
};

// The reference max is only moved when a tile's max exceeds it by more than
// kLazyRescale (log2 units): weights stay <= 2^kLazyRescale, and most tiles
// skip rescaling the accumulators.  Any reference gives the same softmax.
constexpr float kLazyRescale = 8.f;

// LAST: the wave's last tile of its run, the only one that can hold the
// ragged end of a sequence or the newest token.  pos_new >= 0: position of
// the newest token, whose key and value are taken from new_row (LDS: key
// then value, D each) instead of the loaded tile.
template <int D, bool LAST>
__device__ __forceinline__ void process_tile(WaveState<D>& st, Tile<D>& t, const bf16x8* qf,
                                             int t0, int L, int col, int grp, float scale_log2,
                                             int pos_new, const uint16_t* new_row) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  if (LAST && pos_new >= t0 && pos_new < t0 + kTile) {
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      if (t0 + (col >> 2) * 8 + sb * 4 + (col & 3) == pos_new) {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          t.k[sb][kk] = *reinterpret_cast<const u16x8*>(new_row + grp * 8 + kk * 32);
      }
    }
    const int e_new = pos_new - t0 - grp * 8;  // in [0, 8) for the lanes holding it
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint16_t vn = new_row[D + db * 16 + col];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (e == e_new) t.v[db][e] = vn;
    }
  }
  float x[8];  // raw scores q.k of tokens 8*grp + e
  {
    f32x4 s[2];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      s[sb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) s[sb] = mfma_bf16(as_bf16(t.k[sb][kk]), qf[kk], s[sb]);
    }
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int i = 0; i < 4; ++i) x[sb * 4 + i] = s[sb][i];
  }

  if (LAST && t0 + kTile > L) {  // ragged tail: positions >= L take no weight and no value
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

  float tmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                     fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
  tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
  tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
  tmax *= scale_log2;
  const bool raise = tmax > st.m + kLazyRescale;
  if (__ballot(raise)) {  // some head of this wave needs a new reference max
    const float m_new = raise ? tmax : st.m;
    const float alpha = fast_exp2(st.m - m_new);  // 0 on the first tile, 1 if unchanged
    st.m = m_new;
    st.den *= alpha;
#pragma unroll
    for (int db = 0; db < DB; ++db) st.acc[db] *= alpha;
  }

  u16x8 pbits;
  const float neg_m = -st.m;
#pragma unroll
  for (int e = 0; e < 8; ++e) pbits[e] = f32_to_bf16_bits(fast_exp2(fmaf(x[e], scale_log2, neg_m)));
  const bf16x8 pf = as_bf16(pbits);
  // Denominator from the same rounded weights, on the matrix core: a row of
  // ones times P^T sums the 32 weights of each head.
  const u16x8 ones = {0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80};
  st.den = mfma_bf16(as_bf16(ones), pf, st.den);
#pragma unroll
  for (int db = 0; db < DB; ++db) st.acc[db] = mfma_bf16(as_bf16(t.v[db]), pf, st.acc[db]);
}

}  // namespace mlkv
