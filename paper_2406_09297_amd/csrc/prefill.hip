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
// query head hh of KV group r).  A wave takes NB blocks of 16 consecutive
// rows (the MFMA columns) and streams the key/value tiles from position 0 to
// its last row's limit with one online softmax per block (the tile
// arithmetic of decode: S^T = K Q^T, O^T += V^T P^T); each tile's key and
// value registers serve all NB blocks, so a loaded byte feeds NB times the
// matrix work.  Nothing is split over tokens, nothing is merged.  Token t
// attends positions 0 .. ctx_b + t; only the tiles from the wave's smallest
// limit on are masked.  A workgroup is four waves (64*NB consecutive rows).
// Grid: x = unit, y = row block, heaviest blocks (latest tokens) first.
// ---------------------------------------------------------------------------
// One 32-token tile against the wave's NB column blocks.  The tile's key and
// value registers serve every block.  Phases: the scores of all blocks
// (MFMA); the causal mask (MASK: the tile may cross some column's limit);
// the weights' exponents y = scaled score - column reference (FIRST: the
// wave's first tile sets each reference to its column's maximum); one
// wave-wide vote on whether any y exceeds kLazyRescale (each lane tests its
// own eight, so the common case needs no cross-lane traffic); on a yes, the
// column maxima through the wave and the rescale of the blocks that need it;
// then the weights and the value products of all blocks.
// Maximum of a lane's eight values.  Over multiply-add results (canonical
// floats) the compiler forms three-input maxima with no canonicalising maxes;
// being compiler-visible, the reads of matrix-core results also get the wait
// states the hardware requires after a matrix-core write.
__device__ __forceinline__ float max8(const float (&x)[8]) {
  return fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
               fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
}

template <int D, int NB, bool MASK, bool FIRST>
__device__ __forceinline__ void prefill_tile(WaveState<D> (&st)[NB], Tile<D>& t,
                                             const bf16x8 (&qf)[NB][Tile<D>::KK], int t0, int L,
                                             const int (&lim)[NB], int grp, float scale_log2) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  float x[NB][8];
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      s0 = mfma_bf16(as_bf16(t.k[0][kk]), qf[c][kk], s0);
      s1 = mfma_bf16(as_bf16(t.k[1][kk]), qf[c][kk], s1);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[c][i] = s0[i];
      x[c][4 + i] = s1[i];
    }
  }
  if (MASK) {  // positions past a column's limit take no weight, positions >= L no value
    const int first = t0 + grp * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int c = 0; c < NB; ++c)
        if (first + e > lim[c]) x[c][e] = -INFINITY;
      if (first + e >= L) {
#pragma unroll
        for (int db = 0; db < DB; ++db) t.v[db][e] = 0;
      }
    }
  }
  if (FIRST) {
    // The wave's first tile (positions 0..31, which every column attends at
    // position 0): each column's reference is its maximum scaled score.
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const float lmax = max8(x[c]);
      const float cm = fmaxf(lmax, __shfl_xor(lmax, 16));
      st[c].m = fmaxf(cm, __shfl_xor(cm, 32)) * scale_log2;
    }
  }
  // y = scaled score - reference (log2 units): the weights' exponents.
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const float neg_m = -st[c].m;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[c][e] = fmaf(x[c][e], scale_log2, neg_m);
  }
  if (!FIRST) {
    float ymax[NB];
    bool up = false;
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      ymax[c] = max8(x[c]);
      up = up || ymax[c] > kLazyRescale;
    }
    if (__ballot(up)) {  // some column needs a new reference
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        float cm = fmaxf(ymax[c], __shfl_xor(ymax[c], 16));
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        const bool raise = cm > kLazyRescale;  // uniform over the column's lanes
        if (__ballot(raise)) {
          // The reference moves up by the column's excess d: weights and the
          // running sums are scaled by 2^-d.
          const float d = raise ? cm : 0.f;
          const float alpha = fast_exp2(-d);
          st[c].m += d;
          st[c].den *= alpha;
#pragma unroll
          for (int db = 0; db < DB; ++db) st[c].acc[db] *= alpha;
#pragma unroll
          for (int e = 0; e < 8; ++e) x[c][e] -= d;
        }
      }
    }
  }
  const u16x8 ones = {0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80};
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    u16x8 pbits;
#pragma unroll
    for (int e = 0; e < 8; ++e) pbits[e] = f32_to_bf16_bits(fast_exp2(x[c][e]));
    const bf16x8 pf = as_bf16(pbits);
    st[c].den = mfma_bf16(as_bf16(ones), pf, st[c].den);
#pragma unroll
    for (int db = 0; db < DB; ++db) st[c].acc[db] = mfma_bf16(as_bf16(t.v[db]), pf, st[c].acc[db]);
  }
}

// Key/value tiles staged in LDS by direct global-to-LDS loads
// (global_load_lds_dwordx4: lane l of a wave writes its 16 bytes at the
// wave-uniform LDS address + 16 l), double-buffered and shared by the
// workgroup's four waves; no registers hold a tile in transit and no LDS
// store instructions are issued.  Key chunks keep the plane's order, in
// which a wave's operand reads are lane-contiguous; the value chunk
// of channel c and 8-token part p sits at slot 4 c + (p ^ vswz(c)), so that
// the sixteen lanes reading channels c .. c + 15 at one part hit distinct
// banks (for both 32- and 64-bank phase groupings).
constexpr int kRing = 2;
__device__ __forceinline__ int vswz(int c) { return ((c >> 1) ^ (c >> 3)) & 3; }

template <int D>
struct PrefillRing {
  alignas(16) uint16_t k[kRing][kTile * D];
  alignas(16) uint16_t v[kRing][kTile * D];
};

// Wait until this wave's vector memory loads, the direct loads included,
// have landed (vmcnt(0); the other counters are left alone).
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

// A shared-memory pointer as the LDS address the direct loads take.
__device__ __forceinline__ __attribute__((address_space(3))) void* lds_address(uint16_t* p) {
  return (__attribute__((address_space(3))) void*)p;
}

// Requests the tile at position t0 into buffer s: each thread issues D/64
// key and D/64 value chunk loads, 2 D/64 instructions per wave.
template <int D>
__device__ __forceinline__ void ring_issue(PrefillRing<D>& rg, int s, const uint16_t* kbase,
                                           const uint16_t* vbase, int t0) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int u = 0; u < D / 64; ++u) {
    const int slot0 = u * 256 + wave * 64;  // this wave's 64 slots (1 KB) of the buffer
    const int q = slot0 + lane;
    __builtin_amdgcn_global_load_lds(
        static_cast<const void*>(kbase + static_cast<size_t>(t0) * D + q * 8),
        lds_address(&rg.k[s][slot0 * 8]), 16, 0, 0);
    const int c = q >> 2, part = (q & 3) ^ vswz(c);
    __builtin_amdgcn_global_load_lds(
        static_cast<const void*>(vbase + static_cast<size_t>(t0) * D + (c * 4 + part) * 8),
        lds_address(&rg.v[s][slot0 * 8]), 16, 0, 0);
  }
}

// A wave's MFMA operands of one tile from buffer s (the register layout of
// load_tile: permuted key rows, V^T rows).
template <int D>
__device__ __forceinline__ void tile_from_ring(Tile<D>& t, const PrefillRing<D>& rg, int s, int col,
                                               int grp) {
  const int lane = grp * 16 + col;
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int kk = 0; kk < Tile<D>::KK; ++kk)
      t.k[sb][kk] = *reinterpret_cast<const u16x8*>(
          &rg.k[s][((sb * Tile<D>::KK + kk) * 64 + lane) * 8]);
#pragma unroll
  for (int db = 0; db < Tile<D>::DB; ++db) {
    const int c = db * 16 + col;
    t.v[db] = *reinterpret_cast<const u16x8*>(&rg.v[s][(c * 4 + (grp ^ vswz(c))) * 8]);
  }
}

template <int D, int NB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 2)))
void prefill_kernel(PrefillParams p) {
  constexpr int KK = Tile<D>::KK, DB = Tile<D>::DB;
  constexpr int WAVE_ROWS = 16 * NB;
  __shared__ PrefillRing<D> rg;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int unit = blockIdx.x;
  const int b = unit / p.n_groups;
  const int r = unit - b * p.n_groups;
  const int rows = p.T * p.G;
  const int blk = gridDim.y - 1 - blockIdx.y;
  const int wg_row0 = blk * 4 * WAVE_ROWS;  // < rows: the grid has no empty workgroup
  const int row0 = wg_row0 + wave * WAVE_ROWS;
  const bool active = row0 < rows;  // a wave past the end still stages tiles and syncs
  const int c0 = max(p.ctx[b], 0);
  const int L = min(c0 + p.T, p.S);  // filled positions of the sequence
  // Tiles of the workgroup (its last row's limit) and of this wave.
  const int wg_last = min(wg_row0 + 4 * WAVE_ROWS - 1, rows - 1);
  const int n_tiles_wg = min(c0 + wg_last / p.G, p.S - 1) / kTile + 1;
  const int last_row = min(row0 + WAVE_ROWS - 1, rows - 1);
  const int lim_max = min(c0 + last_row / p.G, p.S - 1);
  const int lim_min = min(c0 + min(row0, rows - 1) / p.G, p.S - 1);
  const int n_tiles = active ? lim_max / kTile + 1 : 0;
  const int first_masked = (lim_min + 1) / kTile;  // tiles before it lie under every limit

  const int kv = p.kv_begin + r;
  const size_t seq = static_cast<size_t>(kv) * p.B + b;
  const uint16_t* kbase = p.k + seq * p.S * D;
  const uint16_t* vbase = p.v + seq * p.S * D;
  ring_issue<D>(rg, 0, kbase, vbase, 0);  // every workgroup has at least one tile

  // Column block c: row row0 + 16c + col, its token, head and causal limit
  // (rows past the end: token 0, zero query, output not stored).
  int lim[NB];
  bf16x8 qf[NB][KK];
  WaveState<D> st[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const int rho = row0 + 16 * c + col;
    const bool valid = rho < rows;
    const int tok = valid ? rho / p.G : 0;
    const int head = valid ? rho - tok * p.G : 0;
    lim[c] = min(c0 + tok, p.S - 1);
    const uint16_t* qrow =
        p.q + ((static_cast<size_t>(b) * p.T + tok) * p.h + r * p.G + head) * D + grp * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const u16x8 v = load16(qrow + kk * 32);
      const u16x8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
      qf[c][kk] = as_bf16(valid ? v : zero);
    }
    st[c].den = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < DB; ++db) st[c].acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // Tile it sits in buffer it & 1.  At the barrier this wave's direct loads
  // have landed (waited for explicitly; the barrier's release fence would
  // wait for them too, as they count as writes to LDS), so every wave's part
  // of tile it is there, and every wave is done with tile it - 1, whose
  // buffer then takes tile it + 1 while tile it is used.
  for (int it = 0; it < n_tiles_wg; ++it) {
    wait_loads();
    __syncthreads();
    if (it + 1 < n_tiles_wg) ring_issue<D>(rg, (it + 1) & 1, kbase, vbase, (it + 1) * kTile);
    if (it < n_tiles) {
      Tile<D> t;
      tile_from_ring<D>(t, rg, it & 1, col, grp);
      if (it == 0)
        prefill_tile<D, NB, true, true>(st, t, qf, 0, L, lim, grp, p.scale_log2);
      else if (it >= first_masked)
        prefill_tile<D, NB, true, false>(st, t, qf, it * kTile, L, lim, grp, p.scale_log2);
      else
        prefill_tile<D, NB, false, false>(st, t, qf, it * kTile, L, lim, grp, p.scale_log2);
    }
  }

  // Lane (col, grp) holds channels db*16 + 4*grp .. +3 of its row in each block.
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const int rho = row0 + 16 * c + col;
    if (rho >= rows) continue;
    const int tok = rho / p.G;
    const int head = rho - tok * p.G;
    const float inv = 1.f / st[c].den[0];
    const size_t orow = ((static_cast<size_t>(b) * p.T + tok) * p.h + r * p.G + head) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const f32x4 o = st[c].acc[db] * inv;
      const size_t off = orow + db * 16 + grp * 4;
      if (p.out_bf16) {
        uint16_t* dst = static_cast<uint16_t*>(p.out) + off;
        const uint32_t lo =
            f32_to_bf16_bits(o[0]) | (static_cast<uint32_t>(f32_to_bf16_bits(o[1])) << 16);
        const uint32_t hi =
            f32_to_bf16_bits(o[2]) | (static_cast<uint32_t>(f32_to_bf16_bits(o[3])) << 16);
        *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
      } else {
        *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + off) = o;
      }
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
  *reinterpret_cast<u16x8*>(p.k + (seq * p.S + (pos & ~(kTile - 1))) * D +
                            kchunk<D>(pos & (kTile - 1), d0 / 8) * 8) = kv_k;
  uint16_t* vdst = p.v + (seq * p.S + (pos & ~static_cast<long>(kTile - 1))) * D + (pos & (kTile - 1));
#pragma unroll
  for (int e = 0; e < 8; ++e) vdst[(d0 + e) * kTile] = kv_v[e];
}

hipError_t launch_prefill(const PrefillParams& p, int head_dim, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop) {
  const int per_wg = prefill_rows_per_workgroup(head_dim);
  const int blocks = (p.T * p.G + per_wg - 1) / per_wg;
  const dim3 grid(p.B * p.n_groups, blocks);
  auto kernel = head_dim == 64 ? prefill_kernel<64, prefill_wave_blocks(64)>
                               : prefill_kernel<128, prefill_wave_blocks(128)>;
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
