// HIP kernels around attention in a GPT-NeoX decode step (the architecture of
// the paper's Pythia models, Section 4.2), for CDNA4 (gfx950):
//
//   norm2_kernel        both layer norms of the residual stream x (fp32) ->
//                       h1, h2 (bf16); one workgroup per row
//   qkv_epilogue_kernel bias, rotary embedding at the token's position and
//                       bf16 rounding of the query (every head) and the
//                       owner's key; bias and rounding of the owner's value
//   gelu_kernel         bias + exact GELU of the first MLP product, bf16
//   residual_kernel     x += (o W_o + b_o) + (MLP out + b_2)
//
// The matrix products between them are plain library GEMMs (bf16 operands,
// fp32 results); these kernels carry the elementwise work and the rounding
// points.  Small, bandwidth-light passes over [batch][width] rows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

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

unsigned grid_for(size_t n) {
  const size_t blocks = (n + kModelThreads - 1) / kModelThreads;
  return static_cast<unsigned>(blocks < 2048 ? (blocks > 0 ? blocks : 1) : 2048);
}

}  // namespace

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
