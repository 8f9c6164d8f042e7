/*
 * Seeded synthetic inputs shared by the oracle side and the GPU side.
 *
 * This file holds no attention arithmetic: it only turns (seed, stream,
 * element index) into numbers.  Every element is a pure function of its
 * index, so any slice of any tensor can be regenerated on its own (that is
 * how full-size parity samples rows without copying anything back from the
 * device).
 *
 * Generator (counter-based SplitMix64, Steele/Lea/Flood 2014, with the
 * output mixer of Vigna's public-domain reference):
 *   mix(z)      : z ^= z>>30; z *= 0xBF58476D1CE4E5B9;
 *                 z ^= z>>27; z *= 0x94D049BB133111EB; z ^= z>>31
 *   key(s, k)   : mix(s + (k+1)*0x9E3779B97F4A7C15)      (k-th draw of seed s)
 *   U(s, st, n) : (mix(key(s, st) + (n+1)*0x9E3779B97F4A7C15) >> 11) * 2^-53
 * Normal deviates use the Box-Muller transform on the uniform pair
 * (U(2p), U(2p+1)) of pair p = n/2:
 *   r = sqrt(-2 ln(1 - U(2p))),  z(2p) = r cos(2 pi U(2p+1)),
 *                                z(2p+1) = r sin(2 pi U(2p+1)),
 * evaluated in double, scaled, rounded to float, then to bf16 with
 * round-to-nearest-even.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return mix64(seed + (stream + 1) * GOLDEN);
}

static inline double uniform01(uint64_t key, uint64_t n) {
  return (double)(mix64(key + (n + 1) * GOLDEN) >> 11) * 0x1.0p-53;
}

static inline double normal_at(uint64_t key, uint64_t n) {
  uint64_t p = n >> 1;
  double u1 = uniform01(key, 2 * p);
  double u2 = uniform01(key, 2 * p + 1);
  double r = sqrt(-2.0 * log(1.0 - u1));
  double a = 6.283185307179586476925286766559 * u2;
  return (n & 1) ? r * sin(a) : r * cos(a);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* Raw uniform doubles in [0, 1): out[i] = U(seed, stream, first + i). */
void synth_uniform(uint64_t seed, uint64_t stream, uint64_t first, int64_t count,
                   double* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) out[i] = uniform01(key, first + (uint64_t)i);
}

/* Integers uniform in [lo, hi]: lo + floor(U * (hi - lo + 1)). */
void synth_uniform_int(uint64_t seed, uint64_t stream, uint64_t first, int64_t count,
                       int64_t lo, int64_t hi, int32_t* out) {
  uint64_t key = stream_key(seed, stream);
  double span = (double)(hi - lo + 1);
  for (int64_t i = 0; i < count; ++i) {
    int64_t v = lo + (int64_t)floor(uniform01(key, first + (uint64_t)i) * span);
    if (v > hi) v = hi;
    out[i] = (int32_t)v;
  }
}

/* bf16 normals: out[i] = bf16(float(scale * z(first + i))). */
void synth_normal_bf16(uint64_t seed, uint64_t stream, uint64_t first, int64_t count,
                       double scale, uint16_t* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i)
    out[i] = f32_to_bf16_rne((float)(scale * normal_at(key, first + (uint64_t)i)));
}

/*
 * Rows of a [n_rows][S][D] bf16 tensor (one row per (kv, b) sequence).
 * Row r, token t, channel d takes the deviate of index
 *   ((row0 + r) * 2^26 + t) * D + d,
 * so a token's value does not depend on the buffer's capacity S or on the
 * valid length.  Tokens t >= len[r] (len may be NULL: all valid) get
 * `fill` (e.g. 0x0000 or the bf16 quiet NaN 0x7FC0).
 */
void synth_rows_bf16(uint64_t seed, uint64_t stream, int64_t row0, int64_t n_rows,
                     int64_t S, int64_t D, const int32_t* len, double scale,
                     uint16_t fill, uint16_t* out) {
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t r = 0; r < n_rows; ++r) {
    for (int64_t t = 0; t < S; ++t) {
      uint16_t* dst = out + (r * S + t) * D;
      int64_t valid = len ? len[r] : S;
      if (t >= valid) {
        for (int64_t d = 0; d < D; ++d) dst[d] = fill;
        continue;
      }
      uint64_t base = ((uint64_t)(row0 + r) * (1ULL << 26) + (uint64_t)t) * (uint64_t)D;
      for (int64_t d = 0; d < D; ++d)
        dst[d] = f32_to_bf16_rne((float)(scale * normal_at(key, base + (uint64_t)d)));
    }
  }
}
