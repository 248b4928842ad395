// GPU fill of the seeded synthetic inputs: an independent implementation of
// the SplitMix64 counter generator, the Irwin-Hall approximate normal and the
// bf16 round-to-nearest-even defined in synth.h.  It writes a logical 3-D box
// (D0, D1, D2) whose element (i0, i1, i2) is tensor element
//   lbase + i0*L0 + i1*L1 + i2*L2
// to physical offset i0*S0 + i1*S1 + i2*S2 (elements) of `out`, so a tensor can
// be generated straight into any strided device layout.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__host__ __device__ inline uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ inline uint16_t to_bf16(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (uint16_t)((b >> 16) | 0x40u);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

struct Box {
  int64_t d0, d1, d2;
  int64_t l0, l1, l2, lbase;
  int64_t s0, s1, s2;
};

template <bool kBf16>
__global__ void fill_box(void* out, Box b, uint64_t key, float c, float offset) {
  const int64_t total = b.d0 * b.d1 * b.d2;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i2 = t % b.d2;
    const int64_t r = t / b.d2;
    const int64_t i1 = r % b.d1;
    const int64_t i0 = r / b.d1;
    const uint64_t idx = (uint64_t)(b.lbase + i0 * b.l0 + i1 * b.l1 + i2 * b.l2);
    const uint64_t u = mix(key + (idx + 1) * kGamma);
    const int32_t s = (int32_t)(u & 0xFFFFu) + (int32_t)((u >> 16) & 0xFFFFu) +
                      (int32_t)((u >> 32) & 0xFFFFu) + (int32_t)(u >> 48);
    // one rounding for the product, one for the sum, as on the CPU (no fused multiply-add)
    float v;
    {
#pragma clang fp contract(off)
      const float z = (float)(s - 131070) * c;
      v = offset + z;
    }
    const int64_t p = i0 * b.s0 + i1 * b.s1 + i2 * b.s2;
    if (kBf16)
      static_cast<uint16_t*>(out)[p] = to_bf16(v);
    else
      static_cast<float*>(out)[p] = v;
  }
}

// 4-bit weight bytes: byte j = code(2 (lbase + j)) | code(2 (lbase + j) + 1) << 4, code =
// the top 4 bits of the generator output; and scale bytes 119 + uniform{0, 1, 2}.
__global__ void fill_fp4(uint8_t* out, int64_t n, uint64_t key, int64_t lbase) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n;
       j += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t e = 2 * (uint64_t)(lbase + j);
    const uint64_t a = mix(key + (e + 1) * kGamma), b = mix(key + (e + 2) * kGamma);
    out[j] = (uint8_t)((a >> 60) | ((b >> 60) << 4));
  }
}

__global__ void fill_e8m0(uint8_t* out, int64_t n, uint64_t key, int64_t lbase) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t u = mix(key + ((uint64_t)(lbase + i) + 1) * kGamma);
    out[i] = (uint8_t)(119u + (uint32_t)(((u >> 32) * 3u) >> 32));
  }
}

}  // namespace

extern "C" {

// kind 0: 4-bit code bytes (n bytes), kind 1: scale bytes (n bytes).  Returns a hipError_t.
int synth_gpu_fill_bytes(void* out, int kind, int64_t n, int64_t lbase, uint64_t seed,
                         uint64_t tensor, void* stream) {
  if (!out || n < 0 || (kind != 0 && kind != 1)) return (int)hipErrorInvalidValue;
  if (n == 0) return 0;
  const uint64_t key = mix(mix(seed + kGamma) + (tensor + 1) * kGamma);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (kind == 0)
    hipLaunchKernelGGL(fill_fp4, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<uint8_t*>(out), n,
                       key, lbase);
  else
    hipLaunchKernelGGL(fill_e8m0, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<uint8_t*>(out),
                       n, key, lbase);
  return (int)hipGetLastError();
}


// dtype: 0 = fp32, 1 = bf16 (stored as its 16-bit pattern).  Returns a hipError_t.
int synth_gpu_fill(void* out, int dtype, int64_t d0, int64_t d1, int64_t d2, int64_t l0,
                   int64_t l1, int64_t l2, int64_t lbase, int64_t s0, int64_t s1, int64_t s2,
                   uint64_t seed, uint64_t tensor, double sigma, float offset, void* stream) {
  if (!out || d0 < 0 || d1 < 0 || d2 < 0 || (dtype != 0 && dtype != 1)) return (int)hipErrorInvalidValue;
  const int64_t total = d0 * d1 * d2;
  if (total == 0) return 0;
  Box b{d0, d1, d2, l0, l1, l2, lbase, s0, s1, s2};
  const uint64_t key = mix(mix(seed + kGamma) + (tensor + 1) * kGamma);
  const float c = (float)(sigma * 1.7320508075688772 / 65536.0);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == 1)
    hipLaunchKernelGGL(fill_box<true>, dim3((unsigned)blocks), dim3(256), 0, s, out, b, key, c, offset);
  else
    hipLaunchKernelGGL(fill_box<false>, dim3((unsigned)blocks), dim3(256), 0, s, out, b, key, c, offset);
  return (int)hipGetLastError();
}

}  // extern "C"
