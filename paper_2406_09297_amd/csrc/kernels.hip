// HIP kernels of MLKV decode attention for CDNA4 (gfx950, wave64, MFMA).
//
//   append_kernel        newest token's K/V rows -> cache slot (bit copy)
//   attn_partial_kernel  split-K attention of one layer: each workgroup owns one
//                        (sequence, KV head, token range) and serves every
//                        query head mapped to that KV head from one pass
//   attn_combine_kernel  log-sum-exp merge of the split partials
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
// between the two products.
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

__device__ __forceinline__ u16x8 load16(const uint16_t* p) {
  return *reinterpret_cast<const u16x8*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16(u16x8 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t u) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(u) << 16);
}

// Attended length of sequence b as seen by both the partial and the combine
// kernels (identical clamping keeps their split counts consistent).
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
// Split-K partial attention.  Grid: x = split, y = sequence * n_groups + group.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void attn_partial_kernel(AttnParams p) {
  constexpr int KK = D / 32;  // k-steps of the q.K product
  constexpr int DB = D / 16;  // 16-channel blocks of the output
  constexpr int LDS_STRIDE = D + 4;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;  // query head inside the group / MFMA row
  const int grp = lane >> 4;  // k-slot group: tokens 8*grp .. 8*grp+7 of a tile

  const int split = blockIdx.x;
  const int unit = blockIdx.y;
  const int b = unit / p.n_groups;
  const int r = unit - b * p.n_groups;
  const int kv = p.kv_begin + r;
  const int head0 = r * p.G;

  const int L = attended_len(p, b);
  const int t_begin = split * p.tiles_per_split * kTile;
  if (split > 0 && t_begin >= L) return;  // empty split: nothing to contribute
  int n_tiles = (L - t_begin + kTile - 1) / kTile;
  n_tiles = n_tiles < 0 ? 0 : (n_tiles > p.tiles_per_split ? p.tiles_per_split : n_tiles);

  // Q^T fragments: column = query head, k = channels.  Padded heads are zero.
  bf16x8 qf[KK];
  {
    const bool valid = col < p.G;
    const uint16_t* qrow = p.q + (static_cast<size_t>(b) * p.h + head0 + (valid ? col : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      u16x8 v = valid ? load16(qrow + kk * 32 + grp * 8) : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
      qf[kk] = as_bf16(v);
    }
  }

  const size_t seq = static_cast<size_t>(kv) * p.B + b;
  const uint16_t* kbase = p.k + seq * p.S * D;
  const uint16_t* vbase = p.v + seq * p.S * D;

  float m_run = -INFINITY;  // running max of this lane's head (log2 domain)
  float l_run = 0.f;        // this lane's share of the running denominator
  f32x4 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int it = wave; it < n_tiles; it += kWaves) {
    const int t0 = t_begin + it * kTile;
    // Key rows.  Score sub-block sb, MFMA row rr holds token 8*(rr/4) + 4*sb + rr%4,
    // so the result lane (col, grp) ends up with tokens 8*grp + 4*sb + i.
    u16x8 kf[2][KK];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      const int tok = t0 + (col >> 2) * 8 + sb * 4 + (col & 3);
      const uint16_t* krow = kbase + static_cast<size_t>(tok) * D + grp * 8;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) kf[sb][kk] = load16(krow + kk * 32);
    }
    // V^T rows: channel db*16+col, tokens 8*grp .. 8*grp+7 of the tile.
    u16x8 vf[DB];
    const uint16_t* vblk = vbase + static_cast<size_t>(t0) * D + grp * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) vf[db] = load16(vblk + (db * 16 + col) * kTile);

    f32x4 s[2];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      s[sb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) s[sb] = mfma_bf16(as_bf16(kf[sb][kk]), qf[kk], s[sb]);
    }
    float x[8];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int i = 0; i < 4; ++i) x[sb * 4 + i] = s[sb][i] * p.scale_log2;

    if (t0 + kTile > L) {  // ragged tail: positions >= L take no weight and no value
      const int first = t0 + grp * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (first + e >= L) {
          x[e] = -INFINITY;
#pragma unroll
          for (int db = 0; db < DB; ++db) vf[db][e] = 0;
        }
      }
    }

    float tmax = x[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) tmax = fmaxf(tmax, x[e]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = fast_exp2(m_run - m_new);

    u16x8 pbits;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint16_t pb = f32_to_bf16_bits(fast_exp2(x[e] - m_new));
      pbits[e] = pb;
      psum += bf16_bits_to_f32(pb);  // denominator from the rounded weights
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    const bf16x8 pf = as_bf16(pbits);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      acc[db] *= alpha;
      acc[db] = mfma_bf16(as_bf16(vf[db]), pf, acc[db]);
    }
  }

  // ---- merge the four waves of the workgroup through LDS ----
  __shared__ float sm_acc[kWaves][16][LDS_STRIDE];
  __shared__ float sm_m[kWaves][16];
  __shared__ float sm_l[kWaves][16];
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  if (grp == 0) {
    sm_m[wave][col] = m_run;
    sm_l[wave][col] = l_tot;
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
    *reinterpret_cast<f32x4*>(&sm_acc[wave][col][db * 16 + grp * 4]) = acc[db];
  __syncthreads();

  for (int idx = threadIdx.x; idx < 16 * D; idx += kThreads) {
    const int hh = idx / D;
    const int d = idx - hh * D;
    if (hh >= p.G) break;  // idx grows with hh: every later index is padding too
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
    const size_t row = static_cast<size_t>(b) * p.h + head0 + hh;
    if (p.n_split == 1) {
      const float val = wsum > 0.f ? o / wsum : 0.f;
      if (p.out_bf16)
        static_cast<uint16_t*>(p.out)[row * D + d] = f32_to_bf16_bits(val);
      else
        static_cast<float*>(p.out)[row * D + d] = val;
    } else {
      const size_t slot = row * p.n_split + split;
      p.part_acc[slot * D + d] = o;
      if (d == 0) {
        p.part_ml[slot * 2 + 0] = M;
        p.part_ml[slot * 2 + 1] = wsum;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Log-sum-exp combine: one workgroup of D threads per (sequence, query head),
// splits merged in ascending order (deterministic).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(D) void attn_combine_kernel(AttnParams p) {
  const size_t row = blockIdx.x;  // b * h + i
  const int b = static_cast<int>(row / p.h);
  const int d = threadIdx.x;
  const int L = attended_len(p, b);
  const int chunk = p.tiles_per_split * kTile;
  int ns = (L + chunk - 1) / chunk;
  ns = ns < 1 ? 1 : ns;
  const float* ml = p.part_ml + row * p.n_split * 2;
  const float* acc = p.part_acc + row * p.n_split * D + d;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, ml[2 * s]);
  float wsum = 0.f, o = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < ns; ++s) {
      const float f = fast_exp2(ml[2 * s] - M);
      wsum += f * ml[2 * s + 1];
      o += f * acc[static_cast<size_t>(s) * D];
    }
  }
  const float val = wsum > 0.f ? o / wsum : 0.f;
  if (p.out_bf16)
    static_cast<uint16_t*>(p.out)[row * D + d] = f32_to_bf16_bits(val);
  else
    static_cast<float*>(p.out)[row * D + d] = val;
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

hipError_t launch_attention(const AttnParams& p, int head_dim, hipStream_t stream) {
  const dim3 grid(p.n_split, p.B * p.n_groups);
  if (head_dim == 64)
    hipLaunchKernelGGL(attn_partial_kernel<64>, grid, dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(attn_partial_kernel<128>, grid, dim3(kThreads), 0, stream, p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.n_split == 1) return err;
  const dim3 cgrid(p.B * p.h);
  if (head_dim == 64)
    hipLaunchKernelGGL(attn_combine_kernel<64>, cgrid, dim3(64), 0, stream, p);
  else
    hipLaunchKernelGGL(attn_combine_kernel<128>, cgrid, dim3(128), 0, stream, p);
  return hipGetLastError();
}

}  // namespace mlkv
