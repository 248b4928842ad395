// Skinny-M projection GEMM over MXFP4 weights (4-bit weight-only variant):
//   P[split][M][N] = X[M][K-range of split] . W[N][K-range]^T,
//   W[n][k] = 2^(E[n][k/32] - 127) * e2m1(code[n][k])
//
// MXFP4 is the OCP microscaling format: 4-bit e2m1 elements (sign, 2 exponent bits,
// 1 mantissa bit: 0, 0.5, 1, 1.5, 2, 3, 4, 6 and their negatives), one 8-bit power-of-two
// scale (e8m0) per 32 consecutive elements along K.  Every product of an e2m1 value and
// a power of two is exact in bf16, so gfx950's packed fp4 -> bf16 conversion with a scale
// operand (one instruction per two weights) dequantizes without rounding, and the
// matrix cores multiply the exact weights by the (hi, lo) bf16 activations as in the
// bf16 kernel.  The weight stream shrinks to 0.53 bytes per weight (codes + scales), so
// the projection stays bound by HBM at about a quarter of the bf16 bytes.
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
constexpr int kFp4CodeBlock = 1024;           // bytes of codes per 16 rows x step
constexpr int kFp4ScaleBlock = 64;            // bytes of scales per 16 rows x step
constexpr int kActStepBytes = kFp4Step * 2;   // bf16 activation bytes per row per step

template <int STEPS, int NW, int MT>
struct Fp4Cfg {
  static constexpr int PITCH = STEPS * kActStepBytes + 16;   // LDS bytes per row
  static constexpr int ROWS = 16 * MT;
  static constexpr int UPR = STEPS * kActStepBytes / 16;     // 16-byte units per row
  static constexpr int UNITS = ROWS * UPR;                   // per part
  static constexpr int THREADS = 64 * NW;
  static constexpr int AU = (UNITS + THREADS - 1) / THREADS; // units per thread per part
};

// activation staging registers: 2 parts x AU units, flattened (index part * AU + i)
template <int STEPS, int NW, int MT>
using A4Regs = uint4[2 * Fp4Cfg<STEPS, NW, MT>::AU];

struct Fp4Map {
  int slab, nslab, nblk;
  __device__ __forceinline__ int64_t at(int cb, int ks) const {
    const int t = ks % slab, sl = ks / slab;
    return ((int64_t)t * nslab + sl) * nblk + cb;
  }
};

template <int STEPS>
struct WRegs {
  uint4 code[STEPS];
  uint32_t scale[STEPS];
};

template <int STEPS>
__device__ __forceinline__ void load_w4(WRegs<STEPS>& w, const char* codes, const char* scales,
                                        const Fp4Map& bm, int cb, int ks, int lane, bool ok) {
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int64_t b = bm.at(cb, ks + s);
    w.code[s] = ok ? ld_global(codes + b * kFp4CodeBlock + lane * 16) : make_uint4(0, 0, 0, 0);
    w.scale[s] = ok ? *reinterpret_cast<const uint32_t*>(scales + b * kFp4ScaleBlock +
                                                         (lane & 15) * 4)
                    : 0x7F7F7F7Fu;
  }
}

template <int STEPS, int NW, int MT>
__device__ __forceinline__ void load_a4(A4Regs<STEPS, NW, MT>& ar,
                                        const bf16_t* X, const bf16_t* Xlo, int M, int K, int r0,
                                        int k0) {
  using C = Fp4Cfg<STEPS, NW, MT>;
#pragma unroll
  for (int q = 0; q < 2 * C::AU; ++q) {
    const int p = q / C::AU, i = q - p * C::AU;
    const char* base = reinterpret_cast<const char*>(p == 0 ? X : Xlo);
    const int u = threadIdx.x + i * C::THREADS;
    const int rr = u / C::UPR, c = u - rr * C::UPR;
    uint4 v = make_uint4(0, 0, 0, 0);
    if ((C::UNITS % C::THREADS == 0 || u < C::UNITS) && r0 + rr < M)
      v = *reinterpret_cast<const uint4*>(base + ((int64_t)(r0 + rr) * K + k0) * 2 + c * 16);
    ar[q] = v;
  }
}

template <int STEPS, int NW, int MT>
__device__ __forceinline__ void store_a4(char* buf, const A4Regs<STEPS, NW, MT>& ar) {
  using C = Fp4Cfg<STEPS, NW, MT>;
#pragma unroll
  for (int q = 0; q < 2 * C::AU; ++q) {
    const int p = q / C::AU, i = q - p * C::AU;
    const int u = threadIdx.x + i * C::THREADS;
    const int rr = u / C::UPR, c = u - rr * C::UPR;
    if (C::UNITS % C::THREADS == 0 || u < C::UNITS)
      *reinterpret_cast<uint4*>(buf + (p * C::ROWS + rr) * C::PITCH + c * 16) = ar[q];
  }
}

// e8m0 byte j of `s` as an fp32 power of two (2^(E-127); E in [1, 254])
template <int J>
__device__ __forceinline__ float e8m0(uint32_t s) {
  return __uint_as_float(((s >> (8 * J)) & 0xFFu) << 23);
}

// B fragment (8 bf16: k = 8 g + 0..7 of chunk c) of one 32-element chunk
template <int J>
__device__ __forceinline__ uint4 dequant_chunk(uint32_t codes, uint32_t scales) {
  const float sc = e8m0<J>(scales);
  return make_uint4(
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 0)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 1)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 2)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 3)));
}

// One slice: dequantize each step's four B fragments once, then every 16-row tile and
// both activation parts multiply them.
template <int STEPS, int NW, int MT>
__device__ __forceinline__ void mma_slice4(const char* buf, const WRegs<STEPS>& w, int cl, int g,
                                           f32x4 (&acc)[MT], int M, int r0) {
  using C = Fp4Cfg<STEPS, NW, MT>;
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    uint4 b[4];
    b[0] = dequant_chunk<0>(w.code[s].x, w.scale[s]);
    b[1] = dequant_chunk<1>(w.code[s].y, w.scale[s]);
    b[2] = dequant_chunk<2>(w.code[s].z, w.scale[s]);
    b[3] = dequant_chunk<3>(w.code[s].w, w.scale[s]);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      if (r0 + t * 16 < M) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const char* row = buf + (p * C::ROWS + t * 16 + cl) * C::PITCH + s * kActStepBytes + g * 16;
#pragma unroll
          for (int c = 0; c < 4; ++c)
            acc[t] = mma_frag(*reinterpret_cast<const uint4*>(row + c * 64), b[c], acc[t], bf16_t{});
        }
      }
    }
  }
}

template <int STEPS, int NW, int MT>
__global__ __launch_bounds__(64 * NW, NW / 4) void gemm_fp4_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ Xlo, int M, int K, WeightCat w, int N,
    int iters, float* __restrict__ P) {
  using C = Fp4Cfg<STEPS, NW, MT>;
  __shared__ __attribute__((aligned(16))) char lds[2][2 * C::ROWS * C::PITCH];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, cl = lane & 15;
  const int n0 = blockIdx.y * 16 * NW + wave * 16;
  const int split = blockIdx.x;          // fastest grid dimension (XCD round-robin)
  const int kbeg = split * iters * STEPS * kFp4Step;
  const int ks0 = kbeg / kFp4Step;
  const int ksteps = K / kFp4Step;

  const int mi = n0 >= w.nbeg[2] ? 2 : (n0 >= w.nbeg[1] ? 1 : 0);
  const void* mat = mi == 2 ? w.mat[2] : (mi == 1 ? w.mat[1] : w.mat[0]);
  const void* scl = mi == 2 ? w.scale[2] : (mi == 1 ? w.scale[1] : w.scale[0]);
  const int nb = mi == 2 ? w.nbeg[2] : (mi == 1 ? w.nbeg[1] : w.nbeg[0]);
  const int ne = mi == 2 ? w.nbeg[3] : (mi == 1 ? w.nbeg[2] : w.nbeg[1]);
  const bool ok = n0 < N && n0 < ne;
  const int cb = ok ? (n0 - nb) / 16 : 0;
  const char* codes = static_cast<const char*>(mat);
  const char* scales = static_cast<const char*>(scl);
  const Fp4Map bm{w.slab, ksteps / w.slab, (ne - nb) / 16};

  for (int r0 = 0; r0 < M; r0 += C::ROWS) {
    f32x4 acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    WRegs<STEPS> wa, wb;
    A4Regs<STEPS, NW, MT> ar;
    load_a4<STEPS, NW, MT>(ar, X, Xlo, M, K, r0, kbeg);
    load_w4<STEPS>(wa, codes, scales, bm, cb, ks0, lane, ok);
    store_a4<STEPS, NW, MT>(lds[0], ar);
    for (int i = 0; i < iters; i += 2) {
      __syncthreads();  // lds[0] holds slice i; lds[1] is free
      if (i + 1 < iters) {
        load_a4<STEPS, NW, MT>(ar, X, Xlo, M, K, r0, kbeg + (i + 1) * STEPS * kFp4Step);
        load_w4<STEPS>(wb, codes, scales, bm, cb, ks0 + (i + 1) * STEPS, lane, ok);
      }
      mma_slice4<STEPS, NW, MT>(lds[0], wa, cl, g, acc, M, r0);
      if (i + 1 < iters) store_a4<STEPS, NW, MT>(lds[1], ar);
      __syncthreads();  // lds[1] holds slice i+1; lds[0] is free
      if (i + 2 < iters) {
        load_a4<STEPS, NW, MT>(ar, X, Xlo, M, K, r0, kbeg + (i + 2) * STEPS * kFp4Step);
        load_w4<STEPS>(wa, codes, scales, bm, cb, ks0 + (i + 2) * STEPS, lane, ok);
      }
      if (i + 1 < iters) mma_slice4<STEPS, NW, MT>(lds[1], wb, cl, g, acc, M, r0);
      if (i + 2 < iters) store_a4<STEPS, NW, MT>(lds[0], ar);
    }
    if (ok) {
      const int n = n0 + cl;
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = r0 + t * 16 + 4 * g + j;
          if (r < M) P[((int64_t)split * M + r) * N + n] = acc[t][j];
        }
    }
    __syncthreads();  // before the next row pass reuses lds
  }
}

// Tiled codes <- row-major codes [N][K/2] (byte j of a row: k = 2j in the low nibble).
// Destination 16-byte unit t: lane l = t % 64 of the block at position t / 64, which
// holds row block cb and step ks (inverse of Fp4Map::at); its dword c is the source
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

template <int STEPS, int NW, int MT>
hipError_t launch4(const void* X, const void* Xlo, int M, int K, const WeightCat& w, int N, int iters,
                   float* P, hipStream_t st) {
  dim3 grid(K / (kFp4Step * STEPS * iters), (N + 16 * NW - 1) / (16 * NW));
  hipLaunchKernelGGL((gemm_fp4_kernel<STEPS, NW, MT>), grid, dim3(64 * NW), 0, st,
                     static_cast<const bf16_t*>(X), static_cast<const bf16_t*>(Xlo), M, K, w, N,
                     iters, P);
  return hipGetLastError();
}

// Slices of STEPS * MT <= 8 (the double-buffered activation tile stays within the LDS).
template <int NW, int MT>
hipError_t launch4_steps(int steps, const void* X, const void* Xlo, int M, int K,
                         const WeightCat& w, int N, int iters, float* P, hipStream_t st) {
  if constexpr (MT <= 2) {
    if (steps == 4) return launch4<4, NW, MT>(X, Xlo, M, K, w, N, iters, P, st);
  }
  if constexpr (MT <= 4) {
    if (steps == 2) return launch4<2, NW, MT>(X, Xlo, M, K, w, N, iters, P, st);
  }
  if (steps == 1) return launch4<1, NW, MT>(X, Xlo, M, K, w, N, iters, P, st);
  return hipErrorInvalidValue;
}

}  // namespace

namespace k {

// Launch shape for an MXFP4 projection: 16-wave workgroups for the wide projections
// (N > K), 8-wave ones otherwise; slices of up to 4 steps (128 elements each) and
// enough K-splits to fill the chip about once.
GemmPlan gemm_plan_fp4(const Shape& s, int M, int N, int K) {
  (void)s;
  GemmPlan p{};
  p.cb = 1;
  const int ksteps = K / kFp4Step;
  p.mt = M <= 32 ? 2 : (M <= 64 ? 4 : 8);
  p.nw = N > K ? 16 : 8;
  p.steps = p.mt == 8 ? 1 : 2;
  while (p.steps > 1 && ksteps % p.steps) p.steps >>= 1;
  const int slices = ksteps / p.steps;
  const int tiles = (N + 16 * p.nw - 1) / (16 * p.nw);
  // the fewest splits whose grid reaches 256 workgroups, with at least 2 slices each
  int want = slices;
  while (want > 2 && tiles * (slices / want) < 256) want >>= 1;
  int best = 1;
  for (int c = want; c >= 1; --c)
    if (slices % c == 0) { best = c; break; }
  p.iters = best;
  p.splits = slices / p.iters;
  return p;
}

int pack_slab_steps_fp4(const Shape& s, int N, int K) {
  const GemmPlan p = gemm_plan_fp4(s, 32, N, K);
  return p.steps * p.iters;
}

hipError_t gemm_fp4(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                    const WeightCat& w, int N, float* partials, hipStream_t st) {
  (void)s;
  if (M <= 0 || p.iters < 1 || !Xlo || w.slab < 1 || K % kFp4Step || (K / kFp4Step) % w.slab ||
      (K / kFp4Step) % (p.steps * p.iters))
    return hipErrorInvalidValue;
  if (p.nw == 16) {
    if (p.mt == 2) return launch4_steps<16, 2>(p.steps, X, Xlo, M, K, w, N, p.iters, partials, st);
    if (p.mt == 4) return launch4_steps<16, 4>(p.steps, X, Xlo, M, K, w, N, p.iters, partials, st);
    return launch4_steps<16, 8>(p.steps, X, Xlo, M, K, w, N, p.iters, partials, st);
  }
  if (p.mt == 2) return launch4_steps<8, 2>(p.steps, X, Xlo, M, K, w, N, p.iters, partials, st);
  if (p.mt == 4) return launch4_steps<8, 4>(p.steps, X, Xlo, M, K, w, N, p.iters, partials, st);
  return launch4_steps<8, 8>(p.steps, X, Xlo, M, K, w, N, p.iters, partials, st);
}

hipError_t pack_weight_fp4(const void* codes_src, const void* scales_src, void* codes_dst,
                           void* scales_dst, int N, int K, int slab, hipStream_t st) {
  if (N % 16 || K % kFp4Step || slab < 1 || (K / kFp4Step) % slab) return hipErrorInvalidValue;
  const int64_t units = (int64_t)N * K / 32, words = (int64_t)N * (K / kFp4Step);
  int64_t b1 = (units + 255) / 256, b2 = (words + 255) / 256;
  if (b1 > 65536) b1 = 65536;
  if (b2 > 65536) b2 = 65536;
  hipLaunchKernelGGL(pack_codes_kernel, dim3((unsigned)b1), dim3(256), 0, st,
                     static_cast<const uint32_t*>(codes_src), static_cast<uint4*>(codes_dst), N, K,
                     slab);
  hipLaunchKernelGGL(pack_scales_kernel, dim3((unsigned)b2), dim3(256), 0, st,
                     static_cast<const uint32_t*>(scales_src), static_cast<uint32_t*>(scales_dst),
                     N, K, slab);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
