/* CPU bulk fills for the seeded synthetic inputs; definitions in synth.h. */
#include "synth.h"

void synth_fill_f32(float* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase,
                    double sigma, float offset, int round_bf16) {
  const uint64_t key = synth_key(seed, tensor);
  const float c = synth_scale(sigma);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    out[i] = synth_value(key, (uint64_t)(lbase + i), c, offset, round_bf16);
}

void synth_fill_bf16(uint16_t* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase,
                     double sigma, float offset) {
  const uint64_t key = synth_key(seed, tensor);
  const float c = synth_scale(sigma);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    out[i] = synth_bf16_bits(offset + synth_normal(synth_u64(key, (uint64_t)(lbase + i)), c));
}

void synth_fill_tokens(int32_t* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase,
                       uint32_t vocab) {
  const uint64_t key = synth_key(seed, tensor);
  for (int64_t i = 0; i < n; ++i)
    out[i] = (int32_t)synth_uniform(synth_u64(key, (uint64_t)(lbase + i)), vocab);
}

void synth_fill_fp4(uint8_t* out, int64_t nbytes, uint64_t seed, uint64_t tensor, int64_t lbase) {
  const uint64_t key = synth_key(seed, tensor);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < nbytes; ++j) {
    const uint64_t e = 2 * (uint64_t)(lbase + j);
    out[j] = (uint8_t)(synth_fp4_code(synth_u64(key, e)) | (synth_fp4_code(synth_u64(key, e + 1)) << 4));
  }
}

void synth_fill_e8m0(uint8_t* out, int64_t n, uint64_t seed, uint64_t tensor, int64_t lbase) {
  const uint64_t key = synth_key(seed, tensor);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = synth_e8m0_byte(synth_u64(key, (uint64_t)(lbase + i)));
}

/* Raw generator output (for the published SplitMix64 test vectors). */
uint64_t synth_raw(uint64_t key, uint64_t index) { return synth_u64(key, index); }
uint64_t synth_tensor_key(uint64_t seed, uint64_t tensor) { return synth_key(seed, tensor); }
