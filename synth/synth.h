/* Seeded synthetic inputs shared by the CPU oracle's drivers and the GPU tests.
 *
 * This header holds no arithmetic of the method: only a counter-based random
 * generator, a fixed-point approximate normal, and bf16 rounding.  The GPU fill
 * kernel in synth_gpu.hip implements the same definitions independently; a
 * GPU test checks the two bit for bit.
 *
 * Generator.  SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
 * number generators", OOPSLA 2014): a stream seeded with state s emits
 * mix(s + i*GAMMA) for i = 1, 2, ...  with GAMMA = 0x9E3779B97F4A7C15 and the
 * variant-13 finalizer mix(z) = z ^ (z>>31) after the multiply-xorshift steps
 * (z ^ (z>>30)) * 0xBF58476D1CE4E5B9 and (z ^ (z>>27)) * 0x94D049BB133111EB.
 *
 *   key(seed, tensor) = output (tensor+1) of the stream seeded with mix(seed + GAMMA)
 *   u(key, index)     = output (index+1)  of the stream seeded with key
 *
 * so each element is addressed by its logical index alone and any subset of a
 * tensor can be generated in any order.
 *
 * Approximate normal.  Irwin-Hall sum of the four 16-bit fields of u: the sum
 * S lies in [0, 262140] with mean 131070 and standard deviation 65536/sqrt(3),
 * so z = float(S - 131070) * c with c = float(sigma*sqrt(3)/65536) has standard
 * deviation sigma.  The integer is exact in fp32 and the product is one fp32
 * rounding, hence bit-identical on any IEEE machine.  value = offset + z in fp32,
 * then optionally rounded to bf16 (round to nearest, ties to even).
 *
 * Uniform integer in [0, n): ((u >> 32) * n) >> 32 (Lemire's multiply-shift).
 *
 * 4-bit weights (MXFP4 storage): element code = u >> 60, uniform over the 16 codes;
 * block scale byte = 119 + uniform{0, 1, 2}.  Codes are stored two per byte, element
 * 2j in the low nibble of byte j.  (Only the raw bytes are generated here; what they
 * encode is decided by their consumers.)
 */
#ifndef SYNTH_H
#define SYNTH_H

#include <stdint.h>
#include <string.h>

#define SYNTH_GAMMA 0x9E3779B97F4A7C15ull

static inline uint64_t synth_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline uint64_t synth_key(uint64_t seed, uint64_t tensor) {
  uint64_t s = synth_mix64(seed + SYNTH_GAMMA);
  return synth_mix64(s + (tensor + 1) * SYNTH_GAMMA);
}

static inline uint64_t synth_u64(uint64_t key, uint64_t index) {
  return synth_mix64(key + (index + 1) * SYNTH_GAMMA);
}

static inline float synth_scale(double sigma) {
  return (float)(sigma * 1.7320508075688772 / 65536.0);
}

static inline float synth_normal(uint64_t u, float c) {
  int32_t s = (int32_t)(u & 0xFFFFu) + (int32_t)((u >> 16) & 0xFFFFu) +
              (int32_t)((u >> 32) & 0xFFFFu) + (int32_t)(u >> 48);
  return (float)(s - 131070) * c;
}

static inline uint16_t synth_bf16_bits(float f) {
  uint32_t b;
  memcpy(&b, &f, 4);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (uint16_t)((b >> 16) | 0x40u);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

static inline float synth_bf16_value(uint16_t h) {
  uint32_t b = (uint32_t)h << 16;
  float f;
  memcpy(&f, &b, 4);
  return f;
}

static inline uint32_t synth_uniform(uint64_t u, uint32_t n) {
  return (uint32_t)(((u >> 32) * (uint64_t)n) >> 32);
}

/* value of element `index` of tensor `tensor` */
static inline float synth_value(uint64_t key, uint64_t index, float c, float offset, int round_bf16) {
  float v = offset + synth_normal(synth_u64(key, index), c);
  return round_bf16 ? synth_bf16_value(synth_bf16_bits(v)) : v;
}

static inline uint8_t synth_fp4_code(uint64_t u) { return (uint8_t)(u >> 60); }

static inline uint8_t synth_e8m0_byte(uint64_t u) { return (uint8_t)(119u + synth_uniform(u, 3)); }

/* Bulk CPU fills (synth_cpu.c).  out[i] is element (lbase + i) of the tensor. */
void synth_fill_f32(float* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase,
                    double sigma, float offset, int round_bf16);
void synth_fill_bf16(uint16_t* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase,
                     double sigma, float offset);
void synth_fill_tokens(int32_t* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase,
                       uint32_t vocab);
/* out[j] = code(2 (lbase + j)) | code(2 (lbase + j) + 1) << 4 */
void synth_fill_fp4(uint8_t* out, int64_t nbytes, uint64_t seed, uint64_t tensor, int64_t lbase);
void synth_fill_e8m0(uint8_t* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase);

#endif
