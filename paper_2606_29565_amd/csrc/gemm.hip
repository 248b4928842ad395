// Skinny-M projection GEMM for the entry rows: P[split][M][N] = X[M][K-slice] W[N][K-slice]^T.
//
// The entry is short (M = 16..128 rows), so a projection reads each weight once
// and does only M multiply-adds with it: the kernel is bound by streaming W from
// HBM.  Layout of the work:
//   * a workgroup owns 64 output columns (4 waves x 16) and one K-slice of
//     STEPS*128 bytes per weight row; the grid is (N/64, K/slice) so every weight
//     byte is read exactly once, by exactly one lane, with plenty of workgroups;
//   * each lane issues all of its weight loads (two 16-byte loads per step, 128
//     contiguous bytes per row across the 4 lanes of a column) before it waits,
//     keeping up to 16 x 16 B in flight per lane;
//   * the activation slice X[rows][K-slice] is staged once per 32-row chunk in LDS
//     (padded rows, no bank conflicts on the 16-byte reads) and shared by all waves;
//   * the matrix cores (16x16x32 bf16, or 16x16x4 fp32) contract each 16-row tile;
//   * the K-split partial sums go to P and are reduced, in split order (so the result
//     is deterministic), by the epilogue kernel that consumes them.
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

constexpr int kRowsPerChunk = 32;
constexpr int kStepBytes = 128;  // bytes of one weight row per lane-quad per step
constexpr int kMaxRowTiles = 4;  // rows held across K-slices: 64


template <typename T, int STEPS>
struct GemmCfg {
  static constexpr int KSTEP = kStepBytes / Elem<T>::kBytes;  // elements per step per row
  static constexpr int KS = STEPS * KSTEP;                    // elements in one K-slice
  static constexpr int PITCH = KS * Elem<T>::kBytes + 16;     // LDS row pitch in bytes
  static constexpr int UNITS = KS * Elem<T>::kBytes / 16;     // 16-byte units per row
};

// Stage X[r0 .. r0+31][k0 .. k0+KS) into LDS (rows past M are zero), then barrier.
template <typename T, int STEPS>
__device__ __forceinline__ void stage_rows(char* lds, const T* X, int M, int K, int k0, int r0) {
  using C = GemmCfg<T, STEPS>;
  for (int u = threadIdx.x; u < kRowsPerChunk * C::UNITS; u += 256) {
    const int rr = u / C::UNITS, c = u - rr * C::UNITS;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r0 + rr < M)
      v = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(X) +
                                          ((int64_t)(r0 + rr) * K + k0) * Elem<T>::kBytes + c * 16);
    *reinterpret_cast<uint4*>(lds + rr * C::PITCH + c * 16) = v;
  }
  __syncthreads();
}

// Both 16-row tiles of the staged 32-row chunk against this lane's weight fragments.
template <typename T, int STEPS>
__device__ __forceinline__ void mma_chunk(const char* lds, const uint4 (&wf)[STEPS][2], int cl,
                                          int g, f32x4& a0, f32x4& a1) {
  using C = GemmCfg<T, STEPS>;
  const char* r0p = lds + cl * C::PITCH + g * 32;
  const char* r1p = r0p + 16 * C::PITCH;
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    a0 = mma_frag(*reinterpret_cast<const uint4*>(r0p + s * kStepBytes), wf[s][0], a0, T{});
    a0 = mma_frag(*reinterpret_cast<const uint4*>(r0p + s * kStepBytes + 16), wf[s][1], a0, T{});
    a1 = mma_frag(*reinterpret_cast<const uint4*>(r1p + s * kStepBytes), wf[s][0], a1, T{});
    a1 = mma_frag(*reinterpret_cast<const uint4*>(r1p + s * kStepBytes + 16), wf[s][1], a1, T{});
  }
}

// Lane (column n, group g) of a 16-row tile holds rows 4g..4g+3.
__device__ __forceinline__ void store_tile(float* P, int64_t split, int M, int N, int n, int row0,
                                           int g, const f32x4& a) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = row0 + 4 * g + j;
    if (r < M) P[(split * M + r) * N + n] = a[j];
  }
}

template <typename T, int STEPS>
__device__ __forceinline__ void load_weights(uint4 (&wf)[STEPS][2], const char* wrow, int k0,
                                             bool col_ok) {
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    if (col_ok) {
      const char* p = wrow + (int64_t)k0 * Elem<T>::kBytes + s * kStepBytes;
      wf[s][0] = ld_stream(p);
      wf[s][1] = ld_stream(p + 16);
    } else {
      wf[s][0] = make_uint4(0, 0, 0, 0);
      wf[s][1] = make_uint4(0, 0, 0, 0);
    }
  }
}

template <typename T, int STEPS>
__global__ __launch_bounds__(256) void gemm_kernel(const T* __restrict__ X, int M, int K,
                                                   WeightCat w, int N, int kslices,
                                                   float* __restrict__ P) {
  using C = GemmCfg<T, STEPS>;
  __shared__ __attribute__((aligned(16))) char lds[kRowsPerChunk * C::PITCH];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, cl = lane & 15;
  const int n0 = blockIdx.x * kGemmCols + wave * 16;
  const int n = n0 + cl;
  const int split = blockIdx.y;

  // which concatenated matrix this wave's 16 columns come from (wave-uniform);
  // explicit selects: a dynamic index into the by-value argument would go to scratch
  const int mi = n0 >= w.nbeg[2] ? 2 : (n0 >= w.nbeg[1] ? 1 : 0);
  const void* mat = mi == 2 ? w.mat[2] : (mi == 1 ? w.mat[1] : w.mat[0]);
  const int nb = mi == 2 ? w.nbeg[2] : (mi == 1 ? w.nbeg[1] : w.nbeg[0]);
  const int ne = mi == 2 ? w.nbeg[3] : (mi == 1 ? w.nbeg[2] : w.nbeg[1]);
  const bool col_ok = n < N && n < ne;
  const char* wrow = static_cast<const char*>(mat) +
                     (int64_t)(col_ok ? n - nb : 0) * K * Elem<T>::kBytes + g * 32;

  uint4 wf[STEPS][2];
  if (kslices == 1) {
    // one K-slice per workgroup: weights once, then every 32-row chunk of X
    const int k0 = split * C::KS;
    load_weights<T, STEPS>(wf, wrow, k0, col_ok);
    for (int r0 = 0; r0 < M; r0 += kRowsPerChunk) {
      stage_rows<T, STEPS>(lds, X, M, K, k0, r0);
      f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
      mma_chunk<T, STEPS>(lds, wf, cl, g, a0, a1);
      if (col_ok) {
        store_tile(P, split, M, N, n, r0, g, a0);
        if (r0 + 16 < M) store_tile(P, split, M, N, n, r0 + 16, g, a1);
      }
      __syncthreads();
    }
  } else {
    // several consecutive K-slices summed in registers (M <= 64)
    f32x4 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int sl = 0; sl < kslices; ++sl) {
      const int k0 = (split * kslices + sl) * C::KS;
      load_weights<T, STEPS>(wf, wrow, k0, col_ok);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        if (c * kRowsPerChunk < M) {
          stage_rows<T, STEPS>(lds, X, M, K, k0, c * kRowsPerChunk);
          mma_chunk<T, STEPS>(lds, wf, cl, g, acc[2 * c], acc[2 * c + 1]);
          __syncthreads();
        }
      }
    }
    if (col_ok) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (t * 16 < M) store_tile(P, split, M, N, n, t * 16, g, acc[t]);
    }
  }
}

template <typename T>
int steps_for(int K) {
  constexpr int KSTEP = kStepBytes / Elem<T>::kBytes;
  for (int st = 8; st >= 1; st >>= 1)
    if (K % (st * KSTEP) == 0) return st;
  return 0;
}

template <typename T>
hipError_t launch(const void* X, int M, int K, const WeightCat& w, int N, int kslices, float* P,
                  hipStream_t s) {
  constexpr int KSTEP = kStepBytes / Elem<T>::kBytes;
  const int st = steps_for<T>(K);
  if (st == 0 || M <= 0 || kslices < 1) return hipErrorInvalidValue;
  const int total = K / (st * KSTEP);
  if (total % kslices || (kslices > 1 && M > 16 * kMaxRowTiles)) return hipErrorInvalidValue;
  dim3 grid((N + kGemmCols - 1) / kGemmCols, total / kslices);
  const T* x = static_cast<const T*>(X);
  switch (st) {
    case 8: hipLaunchKernelGGL((gemm_kernel<T, 8>), grid, dim3(256), 0, s, x, M, K, w, N, kslices, P); break;
    case 4: hipLaunchKernelGGL((gemm_kernel<T, 4>), grid, dim3(256), 0, s, x, M, K, w, N, kslices, P); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<T, 2>), grid, dim3(256), 0, s, x, M, K, w, N, kslices, P); break;
    default: hipLaunchKernelGGL((gemm_kernel<T, 1>), grid, dim3(256), 0, s, x, M, K, w, N, kslices, P); break;
  }
  return hipGetLastError();
}

}  // namespace

namespace k {

int gemm_slices(const Shape& s, int K) {
  if (s.bf16) {
    const int st = steps_for<bf16_t>(K);
    return st ? K / (st * (kStepBytes / 2)) : 0;
  }
  const int st = steps_for<float>(K);
  return st ? K / (st * (kStepBytes / 4)) : 0;
}

hipError_t gemm(const Shape& s, const void* X, int M, int K, const WeightCat& w, int N, int kslices,
                float* partials, hipStream_t st) {
  return s.bf16 ? launch<bf16_t>(X, M, K, w, N, kslices, partials, st)
                : launch<float>(X, M, K, w, N, kslices, partials, st);
}

}  // namespace k
}  // namespace spp
