/*
 * Seeded synthetic-input generator, host side.
 *
 * This file holds no part of the verification method: it only turns
 * (key, element index) into a bf16 value, so that the HIP path and the
 * oracle can be fed identical bytes for weights and KV context without
 * materialising tens of GB through Python.
 *
 * Definition (shared, bit for bit, with synth_dev.hip):
 *   mix64(z)      = SplitMix64 output function (Steele, Lea & Flood,
 *                   "Fast Splittable Pseudorandom Number Generators",
 *                   OOPSLA 2014):
 *                     z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9
 *                     z = (z ^ (z >> 27)) * 0x94D049BB133111EB
 *                     z =  z ^ (z >> 31)
 *   h_j(i)        = mix64(key + (2 i + j + 1) * 0x9E3779B97F4A7C15), j = 0, 1
 *   S(i)          = sum of the eight 16-bit fields of h_0(i) and h_1(i)
 *                   (an Irwin-Hall sum of 8 discrete uniforms on [0, 65535])
 *   value(i)      = bf16_rne( (float)(2 S(i) - 524280) * scale )
 * `scale` is an fp32 number chosen by the caller (std / (2 sigma_S));
 * the product is a single IEEE fp32 multiply of two exactly representable
 * operands, so every conforming implementation produces the same bits.
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>

static inline uint64_t sy_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint16_t sy_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline uint16_t sy_value(uint64_t key, uint64_t i, float scale) {
  const uint64_t g = 0x9E3779B97F4A7C15ULL;
  uint64_t a = sy_mix64(key + (2 * i + 1) * g);
  uint64_t b = sy_mix64(key + (2 * i + 2) * g);
  int32_t s = 0;
  for (int k = 0; k < 4; ++k) {
    s += (int32_t)((a >> (16 * k)) & 0xFFFFu);
    s += (int32_t)((b >> (16 * k)) & 0xFFFFu);
  }
  float v = (float)(2 * s - 524280) * scale;
  return sy_bf16_rne(v);
}

/* out[t] = value(base + t) for t in [0, n). */
void sy_fill_linear(uint16_t* out, uint64_t key, uint64_t base, int64_t n, float scale) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t) out[t] = sy_value(key, base + (uint64_t)t, scale);
}

/*
 * KV-context fill for one sequence and one layer.
 * out is [n_heads][n_pos][head_dim] (contiguous); element (h, p, j) takes
 * value(((seq * n_heads + h) << 20 | p) * head_dim + j), so the numbers do
 * not depend on any cache capacity or layout.
 */
void sy_fill_ctx(uint16_t* out, uint64_t key, int32_t seq, int32_t n_heads, int32_t n_pos,
                 int32_t head_dim, float scale) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int32_t h = 0; h < n_heads; ++h)
    for (int32_t p = 0; p < n_pos; ++p) {
      uint64_t row = ((((uint64_t)seq * (uint64_t)n_heads + (uint64_t)h) << 20) | (uint64_t)p) *
                     (uint64_t)head_dim;
      uint16_t* dst = out + ((size_t)h * n_pos + p) * head_dim;
      for (int32_t j = 0; j < head_dim; ++j) dst[j] = sy_value(key, row + (uint64_t)j, scale);
    }
}
