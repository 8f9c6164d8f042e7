// HIP kernels around attention in a GPT-NeoX decode step (the architecture of
// the paper's Pythia models, Section 4.2), for CDNA4 (gfx950).
//
// Fused path (any batch, in tiles of 16 rows; two launches around each
// layer's attention):
//   pack_kernel         once, at model creation: weights into MFMA A-operand
//                       tiles (layout in kernels.h)
//   layer_in_kernel     both layer norms of the residual stream x computed in
//                       the prologue, then [q | k | v | fc1] = LN(x) W on the
//                       matrix cores; epilogue: bias, rotary embedding at the
//                       token's position, exact GELU for fc1, bf16 rounding
//   layer_out_kernel    x += (o W_o + b_o) + (f W_2 + b_2) on the matrix cores
//
// Library path (d_ff not a multiple of 32, layer-norm vectors not 16-byte
// aligned, or MLKV_MODEL_GEMM=library): plain library GEMMs between
//   norm2_kernel        both layer norms of x (fp32) -> h1, h2 (bf16)
//   qkv_epilogue_kernel bias, rotary embedding at the token's position and
//                       bf16 rounding of the query (every head) and the
//                       owner's key; bias and rounding of the owner's value
//   gelu_kernel         bias + exact GELU of the first MLP product, bf16
//   residual_kernel     x += (o W_o + b_o) + (MLP out + b_2)
//
// Both paths round at the same points: the layer-norm outputs, the rotated
// q and k, v, the attention output and the GELU output are bf16; products
// accumulate in fp32; the residual stream is fp32.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
#include "tile.h"

namespace mlkv {
namespace {

constexpr int kModelThreads = 256;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// Nearest bf16 (ties to even) of a double: round to odd into fp32 (24 bits,
// no double rounding), then to nearest even into bf16.
__device__ __forceinline__ uint16_t f64_to_bf16_rne(double v) {
  const float f = __double2float_rz(v);
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if (static_cast<double>(f) != v && v == v) u |= 1u;
  return f32_to_bf16_rne(__builtin_bit_cast(float, u));
}

// Sum over the workgroup (256 threads) through wave shuffles and LDS.
__device__ __forceinline__ float block_sum(float v, float* lds4) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) lds4[wave] = v;
  __syncthreads();
  const float s = lds4[0] + lds4[1] + lds4[2] + lds4[3];
  __syncthreads();
  return s;
}

__global__ __launch_bounds__(kModelThreads) void norm2_kernel(NormParams p) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  const float* x = p.x + static_cast<size_t>(b) * p.d;
  float s = 0.f;
  for (int i = threadIdx.x; i < p.d; i += kModelThreads) s += x[i];
  const float mean = block_sum(s, red) / p.d;
  float s2 = 0.f;
  for (int i = threadIdx.x; i < p.d; i += kModelThreads) {
    const float c = x[i] - mean;
    s2 += c * c;
  }
  const float var = block_sum(s2, red) / p.d;
  const float rstd = 1.f / sqrtf(var + p.eps);
  uint16_t* h1 = p.h1 + static_cast<size_t>(b) * p.d;
  uint16_t* h2 = p.h2 + static_cast<size_t>(b) * p.d;
  for (int i = threadIdx.x; i < p.d; i += kModelThreads) {
    const float z = (x[i] - mean) * rstd;
    h1[i] = f32_to_bf16_rne(z * bf16_to_f32(p.w1[i]) + bf16_to_f32(p.b1[i]));
    h2[i] = f32_to_bf16_rne(z * bf16_to_f32(p.w2[i]) + bf16_to_f32(p.b2[i]));
  }
}

// One workgroup per sequence b.  Element c of a head vector: value
// y32[c] + bias[c] in double; channels c < dims are rotated with their
// partner (rotate-half pairs (j, j + dims/2)) by pos * inv_freq[j], sine and
// cosine in double from an LDS table; rounded once to bf16.
__global__ __launch_bounds__(kModelThreads) void qkv_epilogue_kernel(QkvEpilogueParams p) {
  __shared__ double cos_t[kMaxRopePairs], sin_t[kMaxRopePairs];
  const int b = blockIdx.x;
  const int half = p.dims / 2;
  const double pos = static_cast<double>(p.pos[b]);
  for (int j = threadIdx.x; j < half; j += kModelThreads)
    sincos(pos * p.inv_freq[j], &sin_t[j], &cos_t[j]);
  __syncthreads();
  const int D = p.D;
  auto rotated = [&](const float* y, const uint16_t* bias, int c) -> uint16_t {
    const int e = c % D;  // channel inside the head
    const double u = static_cast<double>(y[c]) + static_cast<double>(bf16_to_f32(bias[c]));
    if (e >= p.dims) return f64_to_bf16_rne(u);
    const int partner = e < half ? c + half : c - half;
    const double w =
        static_cast<double>(y[partner]) + static_cast<double>(bf16_to_f32(bias[partner]));
    const int j = e < half ? e : e - half;
    return f64_to_bf16_rne(e < half ? u * cos_t[j] - w * sin_t[j] : u * cos_t[j] + w * sin_t[j]);
  };
  const float* q32 = p.q32 + static_cast<size_t>(b) * p.q_width;
  uint16_t* q16 = p.q16 + static_cast<size_t>(b) * p.q_width;
  for (int c = threadIdx.x; c < p.q_width; c += kModelThreads) q16[c] = rotated(q32, p.b_q, c);
  if (p.kv_width > 0) {
    const float* k32 = p.k32 + static_cast<size_t>(b) * p.kv_stride + p.kv_offset;
    const float* v32 = p.v32 + static_cast<size_t>(b) * p.kv_stride + p.kv_offset;
    uint16_t* k16 = p.k16 + static_cast<size_t>(b) * p.kv_stride + p.kv_offset;
    uint16_t* v16 = p.v16 + static_cast<size_t>(b) * p.kv_stride + p.kv_offset;
    for (int c = threadIdx.x; c < p.kv_width; c += kModelThreads) {
      k16[c] = rotated(k32, p.b_k, c);
      v16[c] = f64_to_bf16_rne(static_cast<double>(v32[c]) +
                               static_cast<double>(bf16_to_f32(p.b_v[c])));
    }
  }
}

__global__ __launch_bounds__(kModelThreads) void gelu_kernel(GeluParams p) {
  const size_t n = static_cast<size_t>(p.rows) * p.width;
  for (size_t i = blockIdx.x * static_cast<size_t>(kModelThreads) + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * kModelThreads) {
    const int c = static_cast<int>(i % p.width);
    const double z = static_cast<double>(p.y32[i]) + static_cast<double>(bf16_to_f32(p.bias[c]));
    p.out16[i] = f64_to_bf16_rne(0.5 * z * (1.0 + erf(z * 0.70710678118654752440)));
  }
}

__global__ __launch_bounds__(kModelThreads) void residual_kernel(ResidualParams p) {
  const size_t n = static_cast<size_t>(p.rows) * p.d;
  for (size_t i = blockIdx.x * static_cast<size_t>(kModelThreads) + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * kModelThreads) {
    const int c = static_cast<int>(i % p.d);
    p.x[i] += (p.a32[i] + bf16_to_f32(p.b_o[c])) + (p.m32[i] + bf16_to_f32(p.b_2[c]));
  }
}

// ---------------------------------------------------------------------------
// Fused path.  B operand of every product: batch rows b0 .. b0+15 (lane l
// supplies row b0 + l % 16, inputs 8 (l / 16) .. +7 of the k-block); rows at
// or beyond `rows` supply zeros and their results are never stored.  Eight
// waves split the k-blocks (wave w takes w, w + 8, ...) and their partial
// tiles are summed in LDS in wave order, so a launch is deterministic.
// ---------------------------------------------------------------------------
constexpr int kFusedWaves = 8;
constexpr int kFusedThreads = kFusedWaves * 64;

__global__ __launch_bounds__(256) void pack_kernel(PackParams p) {
  const int kbs = p.k_rows / 32;
  const size_t chunks = static_cast<size_t>(p.nt_count) * kbs * 64;
  for (size_t i = blockIdx.x * 256ull + threadIdx.x; i < chunks;
       i += static_cast<size_t>(gridDim.x) * 256) {
    const int lane = static_cast<int>(i % 64);
    const size_t rest = i / 64;
    const int kb = static_cast<int>(rest % kbs);
    const int nt = static_cast<int>(rest / kbs);
    const int n = nt * 16 + lane % 16;
    const int k = kb * 32 + 8 * (lane / 16);
    u16x8 v;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = n < p.n_cols ? p.src[static_cast<size_t>(k + j) * p.n_cols + n] : uint16_t(0);
    *reinterpret_cast<u16x8*>(
        p.dst + (static_cast<size_t>(p.nt0 + nt) * p.kb_total + p.kb0 + kb) * kPackTile +
        lane * 8) = v;
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Column block blk of the layer-in product: q head blk (blk < h), then the
// owned key heads, the owned value heads and the fc1 blocks, each D wide.
// Each wave takes its k-blocks in chunks of PRE and issues every load of a
// chunk (weights, the x rows, the layer-norm scale and shift) before the
// first product, so a chunk costs one memory round trip; the first chunk's
// loads are in flight while the layer-norm statistics are taken.
template <int D>
__global__ __launch_bounds__(kFusedThreads) void layer_in_kernel(LayerInParams p) {
  constexpr int NT = D / 16;
  constexpr int PRE = 16 / NT;  // k-blocks per chunk: 4 (D = 64) or 2 (D = 128)
  __shared__ f32x4 part[kFusedWaves][NT][64];
  __shared__ float y[16][D + 1];
  __shared__ float stats[16][2];
  __shared__ double sc[16][kMaxRopePairs][2];
  const int blk = blockIdx.x, b0 = blockIdx.y * 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool mlp = blk >= p.h + 2 * p.owned;
  const uint16_t* lnw = mlp ? p.ln2_w : p.ln1_w;
  const uint16_t* lnb = mlp ? p.ln2_b : p.ln1_b;
  const int d = p.d, KB = d / 32;
  const int r = lane & 15, grp = lane >> 4;
  const bool live = b0 + r < p.rows;
  const float* xr = p.x + static_cast<size_t>(b0 + (live ? r : 0)) * d + 8 * grp;
  const uint16_t* wblk = p.w + static_cast<size_t>(blk) * NT * KB * kPackTile + lane * 8;

  u16x8 a[PRE][NT], gw[PRE], gb[PRE];
  float4 x0[PRE], x1[PRE];
  auto issue = [&](int base) {
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      const int kb = base + i * kFusedWaves;
      if (kb < KB) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          a[i][nt] = load16(wblk + (static_cast<size_t>(nt) * KB + kb) * kPackTile);
        if (live) {
          x0[i] = *reinterpret_cast<const float4*>(xr + kb * 32);
          x1[i] = *reinterpret_cast<const float4*>(xr + kb * 32 + 4);
          gw[i] = load16(lnw + kb * 32 + 8 * grp);
          gb[i] = load16(lnb + kb * 32 + 8 * grp);
        }
      }
    }
  };
  issue(wave);

  const int half = p.dims / 2;
  const int role = blk < p.h ? 0 : blk < p.h + p.owned ? 1 : blk < p.h + 2 * p.owned ? 2 : 3;
  // The epilogue's biases (element e = threadIdx.x + k * kFusedThreads of the
  // 16 x D tile: its own and, for rotated channels, its partner's), requested
  // now so that their latency hides under the products.
  constexpr int kEpi = 16 * D / kFusedThreads;
  const uint16_t* const bias = role == 0 ? p.b_q : role == 1 ? p.b_k : role == 2 ? p.b_v : p.b_fc1;
  const int jb = role == 0 ? blk : role == 1 ? blk - p.h : role == 2 ? blk - p.h - p.owned
                                                                     : blk - p.h - 2 * p.owned;
  float bias_own[kEpi], bias_partner[kEpi];
#pragma unroll
  for (int k = 0; k < kEpi; ++k) {
    const int e = threadIdx.x + k * kFusedThreads, rr = e / D, c = e % D;
    bias_own[k] = bias_partner[k] = 0.f;
    if (b0 + rr >= p.rows) continue;
    if (role == 3) {
      if (jb * D + c < p.ff) bias_own[k] = bf16_to_f32(bias[jb * D + c]);
      continue;
    }
    bias_own[k] = bf16_to_f32(bias[jb * D + c]);
    if (role < 2 && c < p.dims) {
      const int partner = c < half ? c + half : c - half;
      bias_partner[k] = bf16_to_f32(bias[jb * D + partner]);
    }
  }

  // Rotation angles of the tile's rows (q and k blocks), in double, while the
  // loads are in flight: sc[row][j] = (sin, cos) of pos[row] * inv_freq[j].
  if (role < 2) {
    for (int e = threadIdx.x; e < 16 * half; e += kFusedThreads) {
      const int row = e / half, jj = e % half;
      if (b0 + row < p.rows)
        sincos(static_cast<double>(p.pos[b0 + row]) * p.inv_freq[jj], &sc[row][jj][0],
               &sc[row][jj][1]);
    }
  }

  // Layer-norm statistics: 32 threads per row, each holding up to kStatRegs
  // float4 of it, so the centred second pass reads registers (wider rows
  // read the rest again, from cache).
  {
    constexpr int kStatRegs = 8;
    const int row = threadIdx.x >> 5, j = threadIdx.x & 31;
    float mean = 0.f, rstd = 0.f;
    if (b0 + row < p.rows) {
      const float* xs = p.x + static_cast<size_t>(b0 + row) * d;
      float4 xv[kStatRegs];
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < kStatRegs; ++i) {
        const int c = 4 * j + 128 * i;
        xv[i] = c < d ? *reinterpret_cast<const float4*>(xs + c) : float4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int i = 0; i < kStatRegs; ++i) s += (xv[i].x + xv[i].y) + (xv[i].z + xv[i].w);
      for (int c = 4 * j + 128 * kStatRegs; c < d; c += 128) {
        const float4 v = *reinterpret_cast<const float4*>(xs + c);
        s += (v.x + v.y) + (v.z + v.w);
      }
#pragma unroll
      for (int off = 16; off >= 1; off >>= 1) s += __shfl_xor(s, off);
      mean = s / d;
      float s2 = 0.f;
#pragma unroll
      for (int i = 0; i < kStatRegs; ++i) {
        if (4 * j + 128 * i < d) {
          const float c0 = xv[i].x - mean, c1 = xv[i].y - mean, c2 = xv[i].z - mean,
                      c3 = xv[i].w - mean;
          s2 += (c0 * c0 + c1 * c1) + (c2 * c2 + c3 * c3);
        }
      }
      for (int c = 4 * j + 128 * kStatRegs; c < d; c += 128) {
        const float4 v = *reinterpret_cast<const float4*>(xs + c);
        const float c0 = v.x - mean, c1 = v.y - mean, c2 = v.z - mean, c3 = v.w - mean;
        s2 += (c0 * c0 + c1 * c1) + (c2 * c2 + c3 * c3);
      }
#pragma unroll
      for (int off = 16; off >= 1; off >>= 1) s2 += __shfl_xor(s2, off);
      rstd = 1.f / sqrtf(s2 / d + p.eps);
    }
    if (j == 0) {
      stats[row][0] = mean;
      stats[row][1] = rstd;
    }
  }
  __syncthreads();
  const float mean = stats[r][0], rstd = stats[r][1];

  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int base = wave;;) {
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      if (base + i * kFusedWaves < KB) {
        // LN(x) for 8 consecutive inputs of row b0 + r, rounded to bf16.
        u16x8 hb = {0, 0, 0, 0, 0, 0, 0, 0};
        if (live) {
          const float xv[8] = {x0[i].x, x0[i].y, x0[i].z, x0[i].w,
                               x1[i].x, x1[i].y, x1[i].z, x1[i].w};
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const float z = (xv[jj] - mean) * rstd;
            hb[jj] = f32_to_bf16_rne(z * bf16_to_f32(gw[i][jj]) + bf16_to_f32(gb[i][jj]));
          }
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nt] = mfma_bf16(as_bf16(a[i][nt]), as_bf16(hb), acc[nt]);
      }
    }
    base += PRE * kFusedWaves;
    if (base >= KB) break;
    issue(base);
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) part[wave][nt][lane] = acc[nt];
  __syncthreads();
  // Result lane l of tile nt: column b = l % 16, outputs 16 nt + 4 (l / 16) + i.
  if (threadIdx.x < NT * 64) {
    const int nt = threadIdx.x >> 6, l = threadIdx.x & 63;
    f32x4 s = part[0][nt][l];
#pragma unroll
    for (int w = 1; w < kFusedWaves; ++w) s += part[w][nt][l];
#pragma unroll
    for (int i = 0; i < 4; ++i) y[l & 15][nt * 16 + 4 * (l >> 4) + i] = s[i];
  }
  __syncthreads();

  // Epilogue, in double as the library path's: bias, rotation (q and k),
  // GELU (fc1), one rounding to bf16.
#pragma unroll
  for (int k = 0; k < kEpi; ++k) {
    const int e = threadIdx.x + k * kFusedThreads;
    const int rr = e / D, c = e % D, b = b0 + rr;
    if (b >= p.rows) continue;
    const double u = y[rr][c];
    if (role == 3) {
      const int col = jb * D + c;
      if (col >= p.ff) continue;
      const double z = u + static_cast<double>(bias_own[k]);
      p.f16[static_cast<size_t>(b) * p.ff + col] =
          f64_to_bf16_rne(0.5 * z * (1.0 + erf(z * 0.70710678118654752440)));
      continue;
    }
    const double ub = u + static_cast<double>(bias_own[k]);
    uint16_t out;
    if (role == 2 || c >= p.dims) {
      out = f64_to_bf16_rne(ub);
    } else {
      const int partner = c < half ? c + half : c - half;
      const double w = static_cast<double>(y[rr][partner]) + static_cast<double>(bias_partner[k]);
      const int jj = c < half ? c : c - half;
      const double sn = sc[rr][jj][0], cs = sc[rr][jj][1];
      out = f64_to_bf16_rne(c < half ? ub * cs - w * sn : ub * cs + w * sn);
    }
    if (role == 0)
      p.q16[static_cast<size_t>(b) * p.h * D + jb * D + c] = out;
    else
      (role == 1 ? p.k16 : p.v16)[static_cast<size_t>(b) * p.kv_stride + p.kv_offset + jb * D + c] = out;
  }
}

// Column block blk (16 outputs) of x += (o W_o + b_o) + (f W_2 + b_2); the two
// products keep separate accumulators, as the library path's two GEMMs do.
// K-blocks 0 .. KA-1 are W_o's (input o), KA .. KA+KM-1 W_2's (input f); each
// wave takes every eighth one, in chunks of PRE whose loads are all issued
// before the chunk's products.  With y_mlp given, f W_2 + b_2 was computed
// beside the attention (with the same sums) and only W_o's k-blocks are read.
__global__ __launch_bounds__(kFusedThreads) void layer_out_kernel(LayerOutParams p) {
  constexpr int PRE = 16;
  __shared__ f32x4 part[kFusedWaves][2][64];
  const int blk = blockIdx.x, b0 = blockIdx.y * 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 15, grp = lane >> 4;
  const bool live = b0 + r < p.rows;
  const int KA = p.hD / 32, KM = p.ff / 32, KT = KA + KM;
  const int KU = p.y_mlp ? KA : KT;  // k-blocks multiplied here
  const uint16_t* wblk = p.w + static_cast<size_t>(blk) * KT * kPackTile + lane * 8;
  const uint16_t* orow = p.o16 + static_cast<size_t>(b0 + (live ? r : 0)) * p.hD + 8 * grp;
  const uint16_t* frow = p.f16 + static_cast<size_t>(b0 + (live ? r : 0)) * p.ff + 8 * grp;
  const u16x8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
  // The epilogue's inputs (lane l < 64 finishes four outputs of one row: the
  // residual and both biases), requested now so that their latency hides
  // under the products.
  const int b_out = b0 + (threadIdx.x & 15);
  const int n0 = blk * 16 + 4 * ((threadIdx.x >> 4) & 3);
  const bool writer = threadIdx.x < 64 && b_out < p.rows;
  float4 x_old = {0.f, 0.f, 0.f, 0.f}, y_mlp = {0.f, 0.f, 0.f, 0.f};
  float bo[4] = {0.f, 0.f, 0.f, 0.f}, b2[4] = {0.f, 0.f, 0.f, 0.f};
  if (writer) {
    x_old = *reinterpret_cast<const float4*>(p.x + static_cast<size_t>(b_out) * p.d + n0);
    if (p.y_mlp)
      y_mlp = *reinterpret_cast<const float4*>(p.y_mlp + static_cast<size_t>(b_out) * p.d + n0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bo[i] = bf16_to_f32(p.b_o[n0 + i]);
      if (!p.y_mlp) b2[i] = bf16_to_f32(p.b_2[n0 + i]);
    }
  }
  f32x4 acc_a = {0.f, 0.f, 0.f, 0.f}, acc_m = {0.f, 0.f, 0.f, 0.f};
  for (int base = wave; base < KU; base += PRE * kFusedWaves) {
    u16x8 a[PRE], v[PRE];
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      const int kb = base + i * kFusedWaves;
      if (kb < KU) {
        a[i] = load16(wblk + static_cast<size_t>(kb) * kPackTile);
        v[i] = !live ? zero : kb < KA ? load16(orow + kb * 32) : load16(frow + (kb - KA) * 32);
      }
    }
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      const int kb = base + i * kFusedWaves;
      if (kb < KA)
        acc_a = mfma_bf16(as_bf16(a[i]), as_bf16(v[i]), acc_a);
      else if (kb < KU)
        acc_m = mfma_bf16(as_bf16(a[i]), as_bf16(v[i]), acc_m);
    }
  }
  part[wave][0][lane] = acc_a;
  part[wave][1][lane] = acc_m;
  __syncthreads();
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    f32x4 sa = part[0][0][l], sm = part[0][1][l];
#pragma unroll
    for (int w = 1; w < kFusedWaves; ++w) {
      sa += part[w][0][l];
      sm += part[w][1][l];
    }
    if (writer) {
      if (!p.y_mlp) {
        y_mlp.x = sm[0] + b2[0];
        y_mlp.y = sm[1] + b2[1];
        y_mlp.z = sm[2] + b2[2];
        y_mlp.w = sm[3] + b2[3];
      }
      float4 x_new;
      x_new.x = x_old.x + ((sa[0] + bo[0]) + y_mlp.x);
      x_new.y = x_old.y + ((sa[1] + bo[1]) + y_mlp.y);
      x_new.z = x_old.z + ((sa[2] + bo[2]) + y_mlp.z);
      x_new.w = x_old.w + ((sa[3] + bo[3]) + y_mlp.w);
      *reinterpret_cast<float4*>(p.x + static_cast<size_t>(b_out) * p.d + n0) = x_new;
    }
  }
}

unsigned grid_for(size_t n) {
  const size_t blocks = (n + kModelThreads - 1) / kModelThreads;
  return static_cast<unsigned>(blocks < 2048 ? (blocks > 0 ? blocks : 1) : 2048);
}

}  // namespace

hipError_t launch_pack(const PackParams& p, hipStream_t stream) {
  const size_t chunks = static_cast<size_t>(p.nt_count) * (p.k_rows / 32) * 64;
  hipLaunchKernelGGL(pack_kernel, dim3(grid_for(chunks)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_layer_in(const LayerInParams& p, int head_dim, hipStream_t stream) {
  const dim3 grid(p.h + 2 * p.owned + (p.ff + head_dim - 1) / head_dim, (p.rows + 15) / 16);
  if (head_dim == 64)
    hipLaunchKernelGGL(layer_in_kernel<64>, grid, dim3(kFusedThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(layer_in_kernel<128>, grid, dim3(kFusedThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_layer_out(const LayerOutParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(layer_out_kernel, dim3(p.d / 16, (p.rows + 15) / 16), dim3(kFusedThreads), 0,
                     stream, p);
  return hipGetLastError();
}

hipError_t launch_norm2(const NormParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(norm2_kernel, dim3(p.rows), dim3(kModelThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_qkv_epilogue(const QkvEpilogueParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(qkv_epilogue_kernel, dim3(p.rows), dim3(kModelThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_gelu(const GeluParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(gelu_kernel, dim3(grid_for(static_cast<size_t>(p.rows) * p.width)),
                     dim3(kModelThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_residual(const ResidualParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(residual_kernel, dim3(grid_for(static_cast<size_t>(p.rows) * p.d)),
                     dim3(kModelThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace mlkv
