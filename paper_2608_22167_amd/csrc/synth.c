/*
 * Seeded synthetic-input generator (host side).
 *
 * This file draws random numbers only; it holds none of the decoder layer's
 * arithmetic. Both the GPU path and the CPU reference receive the arrays it
 * writes, so it is the one piece of code the two sides share.
 *
 * Definition (counter based, so any slice can be regenerated on its own):
 *   mix(x)   = the splitmix64 output function applied to x
 *              (Steele, Lea, Flood, "Fast splittable pseudorandom number
 *              generators", OOPSLA 2014).
 *   key      = mix(mix(seed) ^ tensor_id)
 *   h(i)     = mix(key + (i + 1) * 0x9E3779B97F4A7C15)
 *   S(i)     = sum of the eight bytes of h(i)            (integer, 0..2040)
 *   z(i)     = (S(i) - 1020) / sqrt(43690)
 * z is an Irwin-Hall(8) variate: mean 0, variance exactly 1, tails bounded at
 * about 4.9 sigma. The stored value is fp32((float)(S - 1020) * c) + bias with
 * c = fp32(std / sqrt(43690)), i.e. one correctly rounded multiply and one
 * correctly rounded add, so any IEEE-754 implementation reproduces it bit for
 * bit. bfloat16 outputs are that fp32 value rounded to nearest-even.
 */
#include <stdint.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_stream_key(uint64_t seed, uint64_t tensor_id) {
  return mix64(mix64(seed) ^ tensor_id);
}

static inline int byte_sum(uint64_t h) {
  uint64_t a = (h & 0x00FF00FF00FF00FFULL) + ((h >> 8) & 0x00FF00FF00FF00FFULL);
  a = (a & 0x0000FFFF0000FFFFULL) + ((a >> 16) & 0x0000FFFF0000FFFFULL);
  a = (a & 0x00000000FFFFFFFFULL) + (a >> 32);
  return (int)a;
}

static inline float draw(uint64_t key, uint64_t i, float c, float bias) {
  uint64_t h = mix64(key + (i + 1) * 0x9E3779B97F4A7C15ULL);
  float z = (float)(byte_sum(h) - 1020) * c;
  return z + bias;
}

static inline uint16_t to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* out[j] = draw(offset + j) for j < n, as fp32. c is the fp32 multiplier. */
void synth_fill_f32(uint64_t seed, uint64_t tensor_id, uint64_t offset, int64_t n,
                    float c, float bias, float* out) {
  uint64_t key = synth_stream_key(seed, tensor_id);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = draw(key, offset + (uint64_t)j, c, bias);
}

/* Same values rounded to bfloat16 (raw 16-bit patterns). */
void synth_fill_bf16(uint64_t seed, uint64_t tensor_id, uint64_t offset, int64_t n,
                     float c, float bias, uint16_t* out) {
  uint64_t key = synth_stream_key(seed, tensor_id);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = to_bf16_rne(draw(key, offset + (uint64_t)j, c, bias));
}

/*
 * Bulk variant for very large KV pools (indices below 2^32):
 *   g(i) = fmix32(key32 + i * 0x9E3779B9)   (murmur3 32-bit finaliser, a bijection)
 *   S(i) = sum of the four bytes of g(i)     (0..1020), Irwin-Hall(4)
 *   value = fp32(fp32((float)(S - 510) * c) + bias) -> bfloat16, c = fp32(std / sqrt(21845))
 * with key32 = low 32 bits of mix(mix(seed) ^ tensor_id).
 */
static inline uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

void synth_fill_fast_bf16(uint64_t seed, uint64_t tensor_id, uint32_t offset, int64_t n, float c, float bias,
                          uint16_t* out) {
  uint32_t key = (uint32_t)synth_stream_key(seed, tensor_id);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    uint32_t g = fmix32(key + (offset + (uint32_t)j) * 0x9E3779B9u);
    int s = (int)(g & 0xFF) + (int)((g >> 8) & 0xFF) + (int)((g >> 16) & 0xFF) + (int)(g >> 24);
    float z = (float)(s - 510) * c;
    out[j] = to_bf16_rne(z + bias);
  }
}

/* Uniform bytes: out[j] = low byte of h(offset + j). Used for MXFP4 codes and scales. */
void synth_fill_u8(uint64_t seed, uint64_t tensor_id, uint64_t offset, int64_t n, uint8_t* out) {
  uint64_t key = synth_stream_key(seed, tensor_id);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j)
    out[j] = (uint8_t)(mix64(key + (offset + (uint64_t)j + 1) * 0x9E3779B97F4A7C15ULL) & 0xFF);
}
