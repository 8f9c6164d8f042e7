// HIP kernels of MLKV prefill for CDNA4 (gfx950, wave64, MFMA).
//
//   append_rows_kernel  the owners' new rows of a prompt -> cache slots
//                       ctx_b .. ctx_b + T - 1 (bit copy)
//   prefill_kernel      causal attention of one layer over the cache: token
//                       t of sequence b attends positions 0 .. ctx_b + t
//
// The query rows of a KV head (T tokens x G heads of its group) are the MFMA
// columns, 16 per wave; the tile arithmetic is the decode path's (tile.h).
// A separate translation unit, so that the decode kernels are compiled
// exactly as on their own.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
#include "tile.h"

namespace mlkv {

// ---------------------------------------------------------------------------
// Prefill (Section 2.4's cache filled from a prompt, causal): T new tokens per
// sequence.  Unit (b, r) has T*G query rows, row rho = t*G + hh (token t,
// query head hh of KV group r).  A workgroup takes 64 consecutive rows, 16 per
// wave as the MFMA columns; each wave streams the key/value tiles from
// position 0 to its last row's limit with its own online softmax (the same
// tile arithmetic as decode: S^T = K Q^T, O^T += V^T P^T), so there is no
// split over tokens and nothing to merge.  Token t attends positions
// 0 .. ctx_b + t; only the tiles from the wave's smallest limit on are masked.
// Grid: x = unit, y = block of 64 rows, heaviest blocks (latest tokens) first.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void prefill_kernel(PrefillParams p) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int unit = blockIdx.x;
  const int b = unit / p.n_groups;
  const int r = unit - b * p.n_groups;
  const int rows = p.T * p.G;
  const int blk = gridDim.y - 1 - blockIdx.y;
  const int row0 = blk * kPrefillRows + wave * 16;
  if (row0 >= rows) return;  // no barrier below: a wave past the end leaves alone
  const int rho = row0 + col;
  const bool valid = rho < rows;
  const int t = valid ? rho / p.G : 0;
  const int hh = valid ? rho - t * p.G : 0;
  const int c0 = max(p.ctx[b], 0);
  const int L = min(c0 + p.T, p.S);          // filled positions of the sequence
  const int lim = min(c0 + t, p.S - 1);       // last position this column attends
  const int last_row = min(row0 + 15, rows - 1);
  const int lim_max = min(c0 + last_row / p.G, p.S - 1);
  const int lim_min = min(c0 + row0 / p.G, p.S - 1);
  const int n_tiles = lim_max / kTile + 1;
  const int first_masked = (lim_min + 1) / kTile;  // tiles before it lie under every limit

  const int kv = p.kv_begin + r;
  const size_t seq = static_cast<size_t>(kv) * p.B + b;
  const uint16_t* kbase = p.k + seq * p.S * D;
  const uint16_t* vbase = p.v + seq * p.S * D;

  Tile<D> ta, tb;
  load_tile<D, false>(ta, kbase, vbase, 0, col, grp);
  bf16x8 qf[KK];
  {
    const uint16_t* qrow =
        p.q + ((static_cast<size_t>(b) * p.T + t) * p.h + r * p.G + hh) * D + grp * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const u16x8 v = load16(qrow + kk * 32);
      const u16x8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
      qf[kk] = as_bf16(valid ? v : zero);  // rows past the end: scores 0, output unused
    }
  }
  WaveState<D> st;
  st.den = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int db = 0; db < DB; ++db) st.acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto process = [&](Tile<D>& tile, int it) {
    if (it >= first_masked)
      process_tile<D, true, false, true>(st, tile, qf, it * kTile, L, col, grp, p.scale_log2, -1,
                                         nullptr, nullptr, nullptr, 16, lim);
    else
      process_tile<D, false, false, true>(st, tile, qf, it * kTile, L, col, grp, p.scale_log2,
                                          -1, nullptr, nullptr, nullptr, 16, lim);
  };
  int it = 0;
  for (;;) {  // tile it is in ta; the next one's loads go out before it is used
    if (it + 1 < n_tiles) load_tile<D, false>(tb, kbase, vbase, (it + 1) * kTile, col, grp);
    process(ta, it);
    if (++it >= n_tiles) break;
    if (it + 1 < n_tiles) load_tile<D, false>(ta, kbase, vbase, (it + 1) * kTile, col, grp);
    process(tb, it);
    if (++it >= n_tiles) break;
  }

  if (!valid) return;
  // Lane (col, grp) holds channels db*16 + 4*grp .. +3 of its row.
  const float inv = 1.f / st.den[0];
  const size_t orow = ((static_cast<size_t>(b) * p.T + t) * p.h + r * p.G + hh) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const f32x4 o = st.acc[db] * inv;
    const size_t off = orow + db * 16 + grp * 4;
    if (p.out_bf16) {
      uint16_t* dst = static_cast<uint16_t*>(p.out) + off;
      const uint32_t lo = f32_to_bf16_bits(o[0]) | (static_cast<uint32_t>(f32_to_bf16_bits(o[1])) << 16);
      const uint32_t hi = f32_to_bf16_bits(o[2]) | (static_cast<uint32_t>(f32_to_bf16_bits(o[3])) << 16);
      *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + off) = o;
    }
  }
}

// Owners store the T new rows of each sequence at slots ctx_b .. ctx_b+T-1:
// workgroup (x, b, c) covers 256 (token, 8-channel chunk) pairs of owned head c.
template <int D>
__global__ __launch_bounds__(256) void append_rows_kernel(AppendRowsParams p) {
  constexpr int C8 = D / 8;
  const int b = blockIdx.y;
  const int c = blockIdx.z;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= p.T * C8) return;
  const int t = idx / C8;
  const int d0 = (idx - t * C8) * 8;
  const long pos = static_cast<long>(p.ctx[b]) + t;
  if (pos < 0 || pos >= p.S) return;
  const size_t src = (static_cast<size_t>(b) * p.T + t) * p.row_stride + static_cast<size_t>(c) * D + d0;
  const u16x8 kv_k = load16(p.k_new + src);
  const u16x8 kv_v = load16(p.v_new + src);
  const size_t seq = static_cast<size_t>(p.kv_begin + c) * p.B + b;
  *reinterpret_cast<u16x8*>(p.k + (seq * p.S + pos) * D + d0) = kv_k;
  uint16_t* vdst = p.v + (seq * p.S + (pos & ~static_cast<long>(kTile - 1))) * D + (pos & (kTile - 1));
#pragma unroll
  for (int e = 0; e < 8; ++e) vdst[(d0 + e) * kTile] = kv_v[e];
}

hipError_t launch_prefill(const PrefillParams& p, int head_dim, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop) {
  const int blocks = (p.T * p.G + kPrefillRows - 1) / kPrefillRows;
  const dim3 grid(p.B * p.n_groups, blocks);
  auto kernel = head_dim == 64 ? prefill_kernel<64> : prefill_kernel<128>;
  if (start || stop) {
    hipExtLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, start, stop, 0, p);
  } else {
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_append_rows(const AppendRowsParams& p, int head_dim, int owned_count,
                              hipStream_t stream) {
  const int chunks = p.T * (head_dim / 8);
  const dim3 grid((chunks + 255) / 256, p.B, owned_count);
  auto kernel = head_dim == 64 ? append_rows_kernel<64> : append_rows_kernel<128>;
  hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace mlkv
