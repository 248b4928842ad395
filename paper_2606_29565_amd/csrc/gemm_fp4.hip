// MXFP4 projection weights (4-bit weight-only variant) and their tiled layout:
//   W[n][k] = 2^(E[n][k/32] - 127) * e2m1(code[n][k])
//
// MXFP4 is the OCP microscaling format: 4-bit e2m1 elements (sign, 2 exponent bits,
// 1 mantissa bit: 0, 0.5, 1, 1.5, 2, 3, 4, 6 and their negatives), one 8-bit power-of-two
// scale (e8m0) per 32 consecutive elements along K.  Every product of an e2m1 value and
// a power of two is exact in bf16, so gfx950's packed fp4 -> bf16 conversion with a scale
// operand (one instruction per two weights) dequantizes without rounding, and the
// matrix cores multiply the exact weights by the (hi, lo) bf16 activations as in the
// bf16 kernel (gemm.hip streams both formats).  The weight stream shrinks to 0.53 bytes
// per weight (codes + scales), so the projection stays bound by HBM at about a quarter of
// the bf16 bytes.
//
// Tiled layout (pack_weight_fp4), per 16 rows x one 128-element step of K:
//   * a 1 KB code block: lane l = 16 g + r (row r, group g) holds 16 bytes, dword c =
//     the codes of row r at k = 32 c + 8 g + 0..7, byte b = (k = 2b, 2b+1) with the even
//     k in the low nibble -- exactly the B fragment of four 16x16x32 MFMAs;
//   * a 64-byte scale block: dword r = the four e8m0 scales of row r over the step;
// both ordered time-major like the bf16 layout (the blocks that the workgroups of a
// launch stream at the same moment are adjacent).
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

constexpr int kFp4Step = 128;                 // K elements per step

// Tiled codes <- row-major codes [N][K/2] (byte j of a row: k = 2j in the low nibble).
// Destination 16-byte unit t: lane l = t % 64 of the block at position t / 64, which
// holds row block cb and step ks (the inverse of the GEMM's block map); its dword c is the source
// dword of row 16 cb + l % 16 at byte 64 ks + 16 c + 4 (l / 16).
__global__ __launch_bounds__(256) void pack_codes_kernel(const uint32_t* __restrict__ src,
                                                         uint4* __restrict__ dst, int N, int K,
                                                         int slab) {
  const int ksteps = K / kFp4Step, nslab = ksteps / slab, nblk = N / 16;
  const int64_t total = (int64_t)N * K / 32;   // 16-byte units
  const int row_words = K / 8;                 // source dwords per row
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int lane = (int)(t & 63);
    const int64_t pos = t >> 6;
    const int cb = (int)(pos % nblk);
    const int64_t q = pos / nblk;
    const int sl = (int)(q % nslab), ts = (int)(q / nslab);
    const int ks = sl * slab + ts;
    const int64_t n = (int64_t)cb * 16 + (lane & 15);
    const uint32_t* s = src + n * row_words + ks * 16 + (lane >> 4);
    dst[t] = make_uint4(s[0], s[4], s[8], s[12]);
  }
}

// Tiled scales <- row-major e8m0 scales [N][K/32]: block dword r = row 16 cb + r's four
// scales of step ks (one source dword).
__global__ __launch_bounds__(256) void pack_scales_kernel(const uint32_t* __restrict__ src,
                                                          uint32_t* __restrict__ dst, int N, int K,
                                                          int slab) {
  const int ksteps = K / kFp4Step, nslab = ksteps / slab, nblk = N / 16;
  const int64_t total = (int64_t)N * ksteps;   // dwords
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int r = (int)(t & 15);
    const int64_t pos = t >> 4;
    const int cb = (int)(pos % nblk);
    const int64_t q = pos / nblk;
    const int sl = (int)(q % nslab), ts = (int)(q / nslab);
    const int ks = sl * slab + ts;
    dst[t] = src[((int64_t)cb * 16 + r) * ksteps + ks];
  }
}

}  // namespace

namespace k {

hipError_t pack_weight_fp4(const void* codes_src, const void* scales_src, void* codes_dst,
                           void* scales_dst, int N, int K, int slab, hipStream_t st) {
  if (N % 16 || K % kFp4Step || slab < 1 || (K / kFp4Step) % slab) return hipErrorInvalidValue;
  const int64_t units = (int64_t)N * K / 32, words = (int64_t)N * (K / kFp4Step);
  int64_t b1 = (units + 255) / 256, b2 = (words + 255) / 256;
  if (b1 > 65536) b1 = 65536;
  if (b2 > 65536) b2 = 65536;
  SPP_LAUNCH(pack_codes_kernel, dim3((unsigned)b1), dim3(256), 0, st,
                     static_cast<const uint32_t*>(codes_src), static_cast<uint4*>(codes_dst), N, K,
                     slab);
  SPP_LAUNCH(pack_scales_kernel, dim3((unsigned)b2), dim3(256), 0, st,
                     static_cast<const uint32_t*>(scales_src), static_cast<uint32_t*>(scales_dst),
                     N, K, slab);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
