/* Host implementation of the counter-based weight generator.
 *
 * Seeded inputs only: this file holds no step of the decoding method.  It is
 * the host half of a generator that the GPU library implements a second time
 * on its own (the weight-init kernel); the two share no code.
 *
 * Definition (every element of every weight tensor is independent):
 *   mix(z)   = SplitMix64 finaliser (Steele, Lea, Flood 2014):
 *              z ^= z >> 30; z *= 0xBF58476D1CE4E5B9;
 *              z ^= z >> 27; z *= 0x94D049BB133111EB; z ^= z >> 31
 *   key      = mix(seed)
 *   ctr      = (tensor_id << 40) | element_index        (row-major [out, in])
 *   h1, h2   = mix(key + (2 ctr + 1) G), mix(key + (2 ctr + 2) G),
 *              G = 0x9E3779B97F4A7C15  -- outputs 2ctr+1 and 2ctr+2 of the
 *              SplitMix64 stream started at `key`
 *   u1       = ((h1 >> 11) + 1) 2^-53  in (0, 1]
 *   u2       =  (h2 >> 11)      2^-53  in [0, 1)
 *   n        = sqrt(-2 ln u1) cos(2 pi u2)                (Box-Muller, fp64)
 *   w        = bf16_rne(float_rne(std * n))
 */
#include <math.h>
#include <stdint.h>

static inline uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ULL;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBULL;
  z ^= z >> 31;
  return z;
}

static inline uint16_t f32_to_bf16_rne(float f) {
  union { float f; uint32_t u; } v;
  v.f = f;
  uint32_t u = v.u;
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u); /* NaN */
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

static const uint64_t GOLDEN = 0x9E3779B97F4A7C15ULL;
static const double TWO_PI = 6.283185307179586476925286766559;

/* out[i] = weight element (start + i) of tensor `tensor_id`, as bf16 bits. */
void sgen_normal_bf16(uint64_t seed, uint64_t tensor_id, uint64_t start, uint64_t count,
                      double std_dev, uint16_t* out) {
  const uint64_t key = mix64(seed);
  const uint64_t base = tensor_id << 40;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)count; ++i) {
    uint64_t ctr = base | (start + (uint64_t)i);
    uint64_t h1 = mix64(key + (2 * ctr + 1) * GOLDEN);
    uint64_t h2 = mix64(key + (2 * ctr + 2) * GOLDEN);
    double u1 = (double)((h1 >> 11) + 1) * 0x1.0p-53;
    double u2 = (double)(h2 >> 11) * 0x1.0p-53;
    double n = sqrt(-2.0 * log(u1)) * cos(TWO_PI * u2);
    out[i] = f32_to_bf16_rne((float)(std_dev * n));
  }
}

/* Raw SplitMix64 stream, for checking against the published test vectors. */
void sgen_splitmix64_stream(uint64_t state, uint64_t count, uint64_t* out) {
  for (uint64_t i = 0; i < count; ++i) {
    state += GOLDEN;
    out[i] = mix64(state);
  }
}

/* Gather: out[r, :] = row rows[r] of a [n_rows_total, row_len] tensor. */
void sgen_normal_bf16_rows(uint64_t seed, uint64_t tensor_id, const int64_t* rows, int64_t n,
                           uint64_t row_len, double std_dev, uint16_t* out) {
  for (int64_t r = 0; r < n; ++r)
    sgen_normal_bf16(seed, tensor_id, (uint64_t)rows[r] * row_len, row_len, std_dev,
                     out + (uint64_t)r * row_len);
}
