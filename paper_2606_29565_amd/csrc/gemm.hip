// Skinny-M projection GEMM for the entry rows:
//   P[split][M][N] = X[M][K-range of split] . W[N][K-range]^T
//
// The entry is short (M = 16..128 rows), so each weight byte is used for only M
// multiply-adds and the kernel is bound by streaming W from HBM.  Design:
//   * W is stored TILED: for every 16 output columns and every 128-byte step of K
//     the 16 x 128 B block is laid out exactly in the order the 64 lanes of a wave
//     consume it (two 1 KB fragments, lane-major), so every wave-wide 16-byte load
//     reads 1 KB of contiguous memory; the blocks are ordered time-major (pack_weight):
//     when every workgroup of a launch is at the t-th step of its K-range, together
//     they read one compact window of HBM instead of thousands of separate streams
//     (measured on MI355X: 6.2 TB/s for such a sweep against 5.3 TB/s for per-wave
//     streams of the same bytes);
//   * a workgroup of NW waves owns 16*NW columns and a K-range of ITERS slices of
//     STEPS steps; the slices are software-pipelined: while the matrix cores work
//     on slice i, the weights of slice i+1 are in flight into a second register
//     buffer and the activations of slice i+1 into the second half of a double-
//     buffered LDS tile shared by all NW waves;
//   * activations X are staged in LDS with padded rows; each lane reads 16-byte A
//     fragments, the matrix cores (16x16x32 bf16 / 16x16x4 fp32) accumulate MT row
//     tiles of 16 rows in registers.  A bf16 model's activation arrives as two bf16
//     arrays (hi and the rounding remainder lo), both multiplied against the same
//     weight fragment, so the fp32 activation enters the product with ~16 significant
//     bits at no extra weight traffic (the matrix cores have room to spare here);
//   * the few K-splits that remain go to P and are reduced in split order by the
//     epilogue kernel that consumes them, so results are deterministic;
//   * the split index varies fastest over the grid, so that the round-robin deal of
//     workgroups to the XCDs gives each XCD's L2 only its splits' activations.
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

constexpr int kStepBytes = 128;  // bytes of one weight row per step (8 units of 16 B)

// activation units (16 bytes) each thread stages per slice
constexpr int a_units(int elem_bytes, int steps, int nw, int mt) {
  return (16 * mt * steps * (kStepBytes / 16) + 64 * nw - 1) / (64 * nw) + 0 * elem_bytes;
}

template <typename T, int STEPS, int NW, int MT>
struct GemmCfg {
  static constexpr int KSTEP = kStepBytes / Elem<T>::kBytes;       // elements per step
  static constexpr int KS = STEPS * KSTEP;                         // elements per slice
  static constexpr int PITCH = STEPS * kStepBytes + 16;            // LDS bytes per row
  static constexpr int ROWS = 16 * MT;                             // rows staged per pass
  static constexpr int UPR = STEPS * kStepBytes / 16;              // 16-byte units per row
  static constexpr int UNITS = ROWS * UPR;
  static constexpr int THREADS = 64 * NW;
  static constexpr int AU = a_units(Elem<T>::kBytes, STEPS, NW, MT);  // A units per thread
  static constexpr int NP = Elem<T>::kBytes == 2 ? 2 : 1;          // activation parts (hi, lo)
};

// Activation staging registers: NP parts x AU units, flattened (index p * AU + i).
template <typename T, int STEPS, int NW, int MT>
using ARegs = uint4[GemmCfg<T, STEPS, NW, MT>::NP * a_units(Elem<T>::kBytes, STEPS, NW, MT)];

// Activation rows [r0, r0+ROWS) x [k0, k0+KS) of every part, one 16-byte unit per slot.
template <typename T, int STEPS, int NW, int MT>
__device__ __forceinline__ void load_a(ARegs<T, STEPS, NW, MT>& ar, const T* X, const T* Xlo,
                                       int M, int K, int r0, int k0) {
  using C = GemmCfg<T, STEPS, NW, MT>;
#pragma unroll
  for (int q = 0; q < C::NP * C::AU; ++q) {
    const int p = q / C::AU, i = q - p * C::AU;
    const char* base = reinterpret_cast<const char*>(p == 0 ? X : Xlo);
    const int u = threadIdx.x + i * C::THREADS;
    const int rr = u / C::UPR, c = u - rr * C::UPR;
    uint4 v = make_uint4(0, 0, 0, 0);
    if ((C::UNITS % C::THREADS == 0 || u < C::UNITS) && r0 + rr < M)
      v = *reinterpret_cast<const uint4*>(base + ((int64_t)(r0 + rr) * K + k0) * Elem<T>::kBytes +
                                          c * 16);
    ar[q] = v;
  }
}

template <typename T, int STEPS, int NW, int MT>
__device__ __forceinline__ void store_a(char* buf, const ARegs<T, STEPS, NW, MT>& ar) {
  using C = GemmCfg<T, STEPS, NW, MT>;
#pragma unroll
  for (int q = 0; q < C::NP * C::AU; ++q) {
    const int p = q / C::AU, i = q - p * C::AU;
    const int u = threadIdx.x + i * C::THREADS;
    const int rr = u / C::UPR, c = u - rr * C::UPR;
    if (C::UNITS % C::THREADS == 0 || u < C::UNITS)
      *reinterpret_cast<uint4*>(buf + (p * C::ROWS + rr) * C::PITCH + c * 16) = ar[q];
  }
}

// Weights of one slice: fragment (step s, half j) of lane l is 16 bytes at
// block(ks + s) + j*1024 + l*16 in the tiled layout.
// Position of block (row block cb, K-step ks) in the time-major tiled layout.
struct BlockMap {
  int slab;          // K-steps per slab
  int nslab;         // slabs per row (K-steps / slab)
  int nblk;          // 16-row blocks of the matrix
  __device__ __forceinline__ int64_t at(int cb, int ks) const {
    const int t = ks % slab, sl = ks / slab;
    return ((int64_t)t * nslab + sl) * nblk + cb;
  }
};

template <int STEPS>
__device__ __forceinline__ void load_w(uint4 (&wf)[STEPS][2], const char* wlane, const BlockMap& bm,
                                       int cb, int ks, bool ok) {
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const char* p = wlane + bm.at(cb, ks + s) * 2048;
    wf[s][0] = ok ? *reinterpret_cast<const uint4*>(p) : make_uint4(0, 0, 0, 0);
    wf[s][1] = ok ? *reinterpret_cast<const uint4*>(p + 1024) : make_uint4(0, 0, 0, 0);
  }
}

// Lane (row cl, group g) of each 16-row tile: A fragment (s, j) = row elements
// [s*KSTEP + j*4E + g*E, +E), matching the weight fragment's reduction indices.
template <typename T, int STEPS, int NW, int MT>
__device__ __forceinline__ void mma_slice(const char* buf, const uint4 (&wf)[STEPS][2], int cl,
                                          int g, f32x4 (&acc)[MT], int M, int r0) {
  using C = GemmCfg<T, STEPS, NW, MT>;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    if (r0 + t * 16 < M) {
#pragma unroll
      for (int p = 0; p < C::NP; ++p) {
        const char* row = buf + (p * C::ROWS + t * 16 + cl) * C::PITCH + g * 16;
#pragma unroll
        for (int s = 0; s < STEPS; ++s) {
          acc[t] = mma_frag(*reinterpret_cast<const uint4*>(row + s * kStepBytes), wf[s][0], acc[t], T{});
          acc[t] = mma_frag(*reinterpret_cast<const uint4*>(row + s * kStepBytes + 64), wf[s][1], acc[t], T{});
        }
      }
    }
  }
}

template <typename T, int STEPS, int NW, int MT>
__global__ __launch_bounds__(64 * NW, NW / 4) void gemm_kernel(const T* __restrict__ X,
                                                       const T* __restrict__ Xlo, int M, int K,
                                                       WeightCat w, int N, int iters,
                                                       float* __restrict__ P) {
  using C = GemmCfg<T, STEPS, NW, MT>;
  __shared__ __attribute__((aligned(16))) char lds[2][C::NP * C::ROWS * C::PITCH];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, cl = lane & 15;
  // the K-split is the fastest grid dimension: workgroups are dealt to the 8 XCDs in
  // linear order, so each XCD's L2 sees only its splits' slice of the activations
  const int n0 = blockIdx.y * 16 * NW + wave * 16;  // first column of this wave
  const int split = blockIdx.x;
  const int kbeg = split * iters * C::KS;
  const int ks0 = kbeg / C::KSTEP;                   // first global step of the range
  const int ksteps = K / C::KSTEP;

  // which concatenated matrix this wave's 16 columns come from (wave-uniform; explicit
  // selects, since a dynamic index into the by-value argument would go to scratch)
  const int mi = n0 >= w.nbeg[2] ? 2 : (n0 >= w.nbeg[1] ? 1 : 0);
  const void* mat = mi == 2 ? w.mat[2] : (mi == 1 ? w.mat[1] : w.mat[0]);
  const int nb = mi == 2 ? w.nbeg[2] : (mi == 1 ? w.nbeg[1] : w.nbeg[0]);
  const int ne = mi == 2 ? w.nbeg[3] : (mi == 1 ? w.nbeg[2] : w.nbeg[1]);
  const bool ok = n0 < N && n0 < ne;
  const int cb = ok ? (n0 - nb) / 16 : 0;
  const char* wlane = static_cast<const char*>(mat) + lane * 16;
  const BlockMap bm{w.slab, ksteps / w.slab, (ne - nb) / 16};

  for (int r0 = 0; r0 < M; r0 += C::ROWS) {
    f32x4 acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 wa[STEPS][2], wb[STEPS][2];
    ARegs<T, STEPS, NW, MT> ar;
    load_a<T, STEPS, NW, MT>(ar, X, Xlo, M, K, r0, kbeg);
    load_w<STEPS>(wa, wlane, bm, cb, ks0, ok);
    store_a<T, STEPS, NW, MT>(lds[0], ar);
    for (int i = 0; i < iters; i += 2) {
      __syncthreads();  // lds[0] holds slice i; lds[1] is free
      if (i + 1 < iters) {
        load_a<T, STEPS, NW, MT>(ar, X, Xlo, M, K, r0, kbeg + (i + 1) * C::KS);
        load_w<STEPS>(wb, wlane, bm, cb, ks0 + (i + 1) * STEPS, ok);
      }
      mma_slice<T, STEPS, NW, MT>(lds[0], wa, cl, g, acc, M, r0);
      if (i + 1 < iters) store_a<T, STEPS, NW, MT>(lds[1], ar);
      __syncthreads();  // lds[1] holds slice i+1; lds[0] is free
      if (i + 2 < iters) {
        load_a<T, STEPS, NW, MT>(ar, X, Xlo, M, K, r0, kbeg + (i + 2) * C::KS);
        load_w<STEPS>(wa, wlane, bm, cb, ks0 + (i + 2) * STEPS, ok);
      }
      if (i + 1 < iters) mma_slice<T, STEPS, NW, MT>(lds[1], wb, cl, g, acc, M, r0);
      if (i + 2 < iters) store_a<T, STEPS, NW, MT>(lds[0], ar);
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

// dst (tiled, time-major) <- src [N][K] row-major, in 16-byte units.  Thread t writes
// dst unit t: lane l = t % 64 of fragment j of the block at position pos; the block
// holds row block cb and K-step ks (the inverse of BlockMap::at), lane l takes row
// 16*cb + l%16 and 16-byte unit 8*ks + 4*j + l/16 of that row.
__global__ __launch_bounds__(256) void pack_kernel(const uint4* __restrict__ src,
                                                   uint4* __restrict__ dst, int N, int KU,
                                                   int slab) {
  const int64_t total = (int64_t)N * KU;
  const int ksteps = KU / 8, nslab = ksteps / slab, nblk = N / 16;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int lane = (int)(t & 63);
    const int j = (int)((t >> 6) & 1);
    const int64_t pos = t >> 7;
    const int cb = (int)(pos % nblk);
    const int64_t q = pos / nblk;  // = ts * nslab + sl
    const int sl = (int)(q % nslab), ts = (int)(q / nslab);
    const int ks = sl * slab + ts;
    const int64_t n = (int64_t)cb * 16 + (lane & 15);
    const int ku = ks * 8 + j * 4 + (lane >> 4);
    dst[t] = src[n * KU + ku];
  }
}

template <typename T, int STEPS, int NW, int MT>
hipError_t launch_t(const void* X, const void* Xlo, int M, int K, const WeightCat& w, int N,
                    int iters, float* P, hipStream_t s) {
  using C = GemmCfg<T, STEPS, NW, MT>;
  dim3 grid(K / (C::KS * iters), (N + 16 * NW - 1) / (16 * NW));
  hipLaunchKernelGGL((gemm_kernel<T, STEPS, NW, MT>), grid, dim3(64 * NW), 0, s,
                     static_cast<const T*>(X), static_cast<const T*>(Xlo), M, K, w, N, iters, P);
  return hipGetLastError();
}

template <typename T, int NW, int MT>
hipError_t launch_steps(int steps, const void* X, const void* Xlo, int M, int K, const WeightCat& w,
                        int N, int iters, float* P, hipStream_t s) {
  // 4-step slices: 16-wave workgroups with one 32-row tile only (with more rows, or
  // fewer waves, the staging registers would not fit)
  if constexpr (MT == 2 && NW == 16) {
    if (steps == 4) return launch_t<T, 4, NW, MT>(X, Xlo, M, K, w, N, iters, P, s);
  }
  switch (steps) {
    case 2: return launch_t<T, 2, NW, MT>(X, Xlo, M, K, w, N, iters, P, s);
    case 1: return launch_t<T, 1, NW, MT>(X, Xlo, M, K, w, N, iters, P, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch(const k::GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                  const WeightCat& w, int N, float* P, hipStream_t s) {
  if (p.nw == 16) {
    if (p.mt == 2) return launch_steps<T, 16, 2>(p.steps, X, Xlo, M, K, w, N, p.iters, P, s);
    if (p.mt == 4) return launch_steps<T, 16, 4>(p.steps, X, Xlo, M, K, w, N, p.iters, P, s);
    return launch_steps<T, 16, 8>(p.steps, X, Xlo, M, K, w, N, p.iters, P, s);
  }
  if (p.mt == 2) return launch_steps<T, 8, 2>(p.steps, X, Xlo, M, K, w, N, p.iters, P, s);
  if (p.mt == 4) return launch_steps<T, 8, 4>(p.steps, X, Xlo, M, K, w, N, p.iters, P, s);
  return launch_steps<T, 8, 8>(p.steps, X, Xlo, M, K, w, N, p.iters, P, s);
}

}  // namespace

namespace k {

// Launch shape for one projection, from sweeps on MI355X with the split (hi, lo)
// activations (8B and 32B shapes, M = 32 / 64 / 128):
//   * wide projections (MLP gate/up): long pipelined K-ranges of 8 slices; with one
//     32-row tile, 16-wave workgroups of 4-step slices where 8 such slices divide K,
//     otherwise 8-wave workgroups of 2-step slices (16-wave for 128-row tiles);
//   * deep projections (K >= 2N, MLP down): 8-wave workgroups, 8 slices of 2 steps
//     (14 of 1 step for 128-row tiles, where the LDS reads dominate);
//   * the fused QKV projection (N > K): 16-wave workgroups, 8 slices of 1 step (2 steps
//     from K = 5120, so that the split count stays near 5..8);
//   * the attention output projection: 8-wave workgroups, 1-step slices, 8 of them for
//     32-row tiles and 4 otherwise.
// 4-step slices exist only for a 16-wave, 32-row tile (elsewhere the staging registers
// would spill).
GemmPlan gemm_plan(const Shape& s, int M, int N, int K) {
  GemmPlan p{};
  const int kstep = kStepBytes / (s.bf16 ? 2 : 4);
  const int ksteps = K / kstep;
  p.mt = M <= 32 ? 2 : (M <= 64 ? 4 : 8);
  int want;
  if (N >= 16384) {
    if (p.mt == 2 && ksteps % 32 == 0) {
      p.nw = 16; p.steps = 4;
    } else {
      p.nw = p.mt == 8 ? 16 : 8; p.steps = 2;
    }
    want = 8;
  } else if (K >= 2 * N) {
    p.nw = 8;
    if (p.mt == 8) { p.steps = 1; want = 14; } else { p.steps = 2; want = 8; }
  } else if (N > K) {
    p.nw = 16; p.steps = K >= 5120 ? 2 : 1; want = 8;
  } else {
    p.nw = 8; p.steps = 1; want = p.mt == 2 ? 8 : 4;
  }
  while (p.steps > 1 && ksteps % p.steps) p.steps >>= 1;
  const int slices = ksteps / p.steps;
  if (want > slices) want = slices;
  // largest pipelined-slice count <= want that divides the slices
  int best = 1;
  for (int c = want; c >= 1; --c)
    if (slices % c == 0) { best = c; break; }
  p.iters = best;
  p.splits = slices / p.iters;
  return p;
}

hipError_t gemm(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                const WeightCat& w, int N, float* partials, hipStream_t st) {
  if (M <= 0 || p.iters < 1 || (s.bf16 && !Xlo) || w.slab < 1 || (K * (s.bf16 ? 2 : 4) / kStepBytes) % w.slab)
    return hipErrorInvalidValue;
  return s.bf16 ? launch<bf16_t>(p, X, Xlo, M, K, w, N, partials, st)
                : launch<float>(p, X, Xlo, M, K, w, N, partials, st);
}

int pack_slab_steps(const Shape& s, int N, int K) {
  const GemmPlan p = gemm_plan(s, 32, N, K);
  return p.steps * p.iters;
}

hipError_t pack_weight(int elem_bytes, const void* src, void* dst, int N, int K, int slab,
                       hipStream_t st) {
  const int KU = K * elem_bytes / 16;
  if (N % 16 || (K * elem_bytes) % kStepBytes || slab < 1 || (KU / 8) % slab)
    return hipErrorInvalidValue;
  const int64_t total = (int64_t)N * KU;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), N, KU, slab);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
