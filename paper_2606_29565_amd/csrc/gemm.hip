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
//     they read one compact window of HBM instead of thousands of separate streams;
//   * a workgroup of NW waves owns 16*NW*CB columns (CB column blocks of 16 per wave)
//     and a K-range of ITERS slices of STEPS steps.  The slices are software-pipelined
//     with every load unconditional (rows past M and columns past N read clamped,
//     valid addresses and are never stored), so the compiler's wait counts are exact:
//     while the matrix cores work on slice i, the weights and activations of slice i+1
//     are in flight;
//   * activations X are staged in a double-buffered LDS tile with padded rows shared by
//     the NW waves; one 16-byte A fragment read from LDS feeds CB matrix-core steps
//     (16x16x32 bf16 / 16x16x4 fp32).  A bf16 model's activation arrives as two bf16
//     arrays (hi and the rounding remainder lo), both multiplied against the same
//     weight fragment, so the fp32 activation enters the product with ~16 significant
//     bits at no extra weight traffic; hi and lo accumulate in separate chains when
//     there would otherwise be fewer than four independent accumulators;
//   * the few K-splits that remain go to P and are reduced in split order by the
//     epilogue kernel that consumes them, so results are deterministic;
//   * the split index varies fastest over the grid, so that the round-robin deal of
//     workgroups to the XCDs gives each XCD's L2 only its splits' activations;
//   * the MLP gate/up projection can run without K-splits and finish the SwiGLU itself:
//     its waves alternate between 16-column blocks of the gate and of the up matrix at
//     the same columns, the up wave hands its accumulators to the gate wave through LDS,
//     and the gate wave writes silu(inv*gate) * (inv*up) as the down projection's input
//     (inv = the row's 1/RMS of the factored RMSNorm);
//   * MXFP4 weights (Q4: 4-bit e2m1 codes and one e8m0 scale per 32 along K, tiled by
//     pack_weight_fp4) go through the same pipeline: a step is 128 elements (a 1 KB code
//     block and a 64-byte scale block per 16 columns), dequantized exactly to bf16 in
//     registers (gfx950's scaled fp4 conversion) into the four B fragments of the step.
//     A 4-bit byte feeds four times the products of a bf16 one, so each wave takes
//     several column blocks and every A fragment read from LDS serves all of them.
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

constexpr int kStepBytes = 128;  // bytes of one weight row per step (8 units of 16 B)
constexpr int kQ4Step = 128;     // elements per step of an MXFP4 matrix
constexpr int kQ4CodeBlock = 1024, kQ4ScaleBlock = 64;  // bytes per 16 rows x step

// Padding of each staged activation row in LDS (bytes).  The A fragments are 16-byte
// reads of 16 rows x 64 bytes; measured on gfx950, they run at the full LDS rate when
// the row pitch is an odd multiple of 32 bytes, at half rate when it is an odd multiple
// of 16 (every row here is a multiple of 64 bytes, so 32 bytes of padding).
#ifndef SPP_GEMM_PAD
#define SPP_GEMM_PAD 32
#endif
#ifndef SPP_GEMM_BIG_WPE
#define SPP_GEMM_BIG_WPE 2
#endif

template <typename T, bool Q4, int STEPS, int NW, int MT, int CB>
struct GemmCfg {
  static constexpr int EB = Elem<T>::kBytes;
  static constexpr int ABYTES = Q4 ? kQ4Step * EB : kStepBytes;    // activation bytes per row per step
  static constexpr int KSTEP = ABYTES / EB;                        // elements per step
  static constexpr int KS = STEPS * KSTEP;                         // elements per slice
  static constexpr int PITCH = STEPS * ABYTES + SPP_GEMM_PAD;      // LDS bytes per row
  static constexpr int ROWS = 16 * MT;                             // rows staged per pass
  static constexpr int UPR = STEPS * ABYTES / 16;                  // 16-byte units per row
  static constexpr int UNITS = ROWS * UPR;
  static constexpr int THREADS = 64 * NW;
  static constexpr int AU = (UNITS + THREADS - 1) / THREADS;       // A units per thread
  static constexpr int NP = EB == 2 ? 2 : 1;                       // activation parts (hi, lo)
  static constexpr int NA = NP * MT * CB >= 4 ? 1 : NP;            // accumulator sets
};

// Activation rows [r0, r0+ROWS) x [k0, k0+KS) of every part, one 16-byte unit per slot
// (index p * AU + i).  Units past the tile repeat the last unit and rows past M repeat
// row M-1: the loads stay unconditional and the extra rows' results are never stored.
template <typename C>
__device__ __forceinline__ void load_a(uint4 (&ar)[C::NP * C::AU], const void* X, const void* Xlo,
                                       int M, int K, int r0, int k0) {
#pragma unroll
  for (int q = 0; q < C::NP * C::AU; ++q) {
    const int p = q / C::AU, i = q - p * C::AU;
    const char* base = static_cast<const char*>(p == 0 ? X : Xlo);
    int u = threadIdx.x + i * C::THREADS;
    if (C::UNITS % C::THREADS != 0) u = min(u, C::UNITS - 1);
    const int rr = u / C::UPR, c = u - rr * C::UPR;
    const int row = min(r0 + rr, M - 1);
    ar[q] = ld_global(base + ((int64_t)row * K + k0) * C::EB + c * 16);
  }
}

template <typename C>
__device__ __forceinline__ void store_a(char* buf, const uint4 (&ar)[C::NP * C::AU]) {
#pragma unroll
  for (int q = 0; q < C::NP * C::AU; ++q) {
    const int p = q / C::AU, i = q - p * C::AU;
    int u = threadIdx.x + i * C::THREADS;
    if (C::UNITS % C::THREADS != 0) u = min(u, C::UNITS - 1);  // a duplicate of the same bytes
    const int rr = u / C::UPR, c = u - rr * C::UPR;
    *reinterpret_cast<uint4*>(buf + (p * C::ROWS + rr) * C::PITCH + c * 16) = ar[q];
  }
}

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

// Output of the fused SwiGLU variant: act[r][f] = silu(inv[r] g[r][f]) * (inv[r] u[r][f]),
// inv[r] = 1/RMS of row r from its per-block sums of squares ss[r][nb].
struct SwigluOut {
  const float* ss;
  int nb, d;
  float eps;
  void* act;
  void* act_lo;
  int F;
};

// One wave's column block: the lane's base addresses inside the matrix that holds it
// (weights or codes; MXFP4 scales), the block index in that matrix and its block map.
struct ColBlock {
  const char* wlane;
  const char* slane;
  int cb;
  BlockMap bm;
};

// Weights of one slice in registers.  Dtype: fragment (c, step s, half j) of lane l is
// 16 bytes at block(ks + s) + j*1024 + l*16 of column block c.  MXFP4: lane l's 16 code
// bytes at block(ks + s) * 1024 + l*16 and the four scales of its row at
// block(ks + s) * 64 + (l % 16) * 4.
template <bool Q4, int CB, int STEPS>
struct WTile {
  uint4 f[CB][STEPS][2];
};
template <int CB, int STEPS>
struct WTile<true, CB, STEPS> {
  uint4 code[CB][STEPS];
  uint32_t scale[CB][STEPS];
};

template <bool Q4, int STEPS, int CB>
__device__ __forceinline__ void load_w(WTile<Q4, CB, STEPS>& w, const ColBlock (&cbk)[CB], int ks) {
#pragma unroll
  for (int c = 0; c < CB; ++c)
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int64_t b = cbk[c].bm.at(cbk[c].cb, ks + s);
      if constexpr (Q4) {
        w.code[c][s] = ld_global(cbk[c].wlane + b * kQ4CodeBlock);
        w.scale[c][s] = ld_global_u32(cbk[c].slane + b * kQ4ScaleBlock);
      } else {
        const char* p = cbk[c].wlane + b * 2048;
        w.f[c][s][0] = ld_global(p);
        w.f[c][s][1] = ld_global(p + 1024);
      }
    }
}

// e8m0 byte J of `s` as an fp32 power of two (2^(E-127); E in [1, 254])
template <int J>
__device__ __forceinline__ float e8m0(uint32_t s) {
  return __uint_as_float(((s >> (8 * J)) & 0xFFu) << 23);
}

// B fragment (8 bf16 weights: k = 32 J + 8 g + 0..7 of the step) from the code dword J
// and the scale of that 32-element chunk; every e2m1 value times a power of two in
// range is exact in bf16
template <int J>
__device__ __forceinline__ uint4 dequant_chunk(uint32_t codes, uint32_t scales) {
  const float sc = e8m0<J>(scales);
  return make_uint4(
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 0)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 1)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 2)),
      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, sc, 3)));
}

template <int J>
__device__ __forceinline__ uint32_t dword(const uint4& v) {
  return J == 0 ? v.x : (J == 1 ? v.y : (J == 2 ? v.z : v.w));
}

// One 32-element chunk J of step s of an MXFP4 slice: the CB column blocks' B fragments,
// then every part and 16-row tile reads its A fragment once for all of them.
template <typename C, int J, int STEPS, int MT, int CB>
__device__ __forceinline__ void mma_chunk_q4(const char* buf, const WTile<true, CB, STEPS>& w, int s,
                                             int cl, int g, f32x4 (&acc)[C::NA][MT][CB]) {
  uint4 b[CB];
#pragma unroll
  for (int c = 0; c < CB; ++c) b[c] = dequant_chunk<J>(dword<J>(w.code[c][s]), w.scale[c][s]);
#pragma unroll
  for (int p = 0; p < C::NP; ++p)
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const uint4 a = *reinterpret_cast<const uint4*>(buf + (p * C::ROWS + t * 16 + cl) * C::PITCH +
                                                      s * C::ABYTES + J * 64 + g * 16);
#pragma unroll
      for (int c = 0; c < CB; ++c) acc[p % C::NA][t][c] = mma_frag(a, b[c], acc[p % C::NA][t][c], bf16_t{});
    }
}

// Lane (row cl, group g) of each 16-row tile: A fragment (s, j) = row elements
// [s*KSTEP + j*4E + g*E, +E), matching the weight fragment's reduction indices.
template <typename T, typename C, bool Q4, int STEPS, int MT, int CB>
__device__ __forceinline__ void mma_slice(const char* buf, const WTile<Q4, CB, STEPS>& w, int cl, int g,
                                          f32x4 (&acc)[C::NA][MT][CB]) {
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    if constexpr (Q4) {
      mma_chunk_q4<C, 0>(buf, w, s, cl, g, acc);
      mma_chunk_q4<C, 1>(buf, w, s, cl, g, acc);
      mma_chunk_q4<C, 2>(buf, w, s, cl, g, acc);
      mma_chunk_q4<C, 3>(buf, w, s, cl, g, acc);
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int p = 0; p < C::NP; ++p)
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            const uint4 a = *reinterpret_cast<const uint4*>(buf + (p * C::ROWS + t * 16 + cl) * C::PITCH +
                                                            g * 16 + s * kStepBytes + j * 64);
#pragma unroll
            for (int c = 0; c < CB; ++c)
              acc[p % C::NA][t][c] = mma_frag(a, w.f[c][s][j], acc[p % C::NA][t][c], T{});
          }
    }
  }
}

// (with the deep prefetch up to 32 rows, two 8-wave workgroups per CU: <= 128 VGPRs)
// Waves per SIMD the register budget is held to: several for the 64-row tiles of many-row
// projections (several workgroups per CU, so one's loads overlap another's products).
template <int MT, int CB>
constexpr int gemm_waves_per_eu() { return MT == 4 && CB == 4 ? SPP_GEMM_BIG_WPE : 1; }
// The fused gate/up of more than 8 waves per workgroup: at most 128 registers, so that its
// 10-16 waves (3-4 per SIMD) fit one workgroup per CU.
template <int NW, int MT, int CB, bool SW, bool Q4>
constexpr int gemm_kernel_waves_per_eu() {
  return SW && !Q4 && NW > 8 ? 4 : gemm_waves_per_eu<MT, CB>();
}

template <typename T, bool Q4, int STEPS, int NW, int MT, int CB, bool SW>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(gemm_kernel_waves_per_eu<NW, MT, CB, SW, Q4>()))) void gemm_kernel(const T* __restrict__ X,
                                                       const T* __restrict__ Xlo, int M, int K,
                                                       WeightCat w, int N, int iters,
                                                       float* __restrict__ P, SwigluOut so,
                                                       int row_tiles, int splits, int groups) {
  using C = GemmCfg<T, Q4, STEPS, NW, MT, CB>;
  static_assert(!Q4 || C::EB == 2, "MXFP4 weights multiply bf16 activations");
  // two activation stages (the fused SwiGLU's exchange of the up sums reuses them)
  constexpr int XCH = SW ? NW / 2 * CB * MT * 4 * 64 * 4 : 0;
  constexpr int STAGE = C::NP * C::ROWS * C::PITCH > (XCH + 1) / 2 ? C::NP * C::ROWS * C::PITCH
                                                                    : (XCH + 1) / 2;
  __shared__ __attribute__((aligned(16))) char lds[2][STAGE];
  static_assert(!SW || NW % 2 == 0, "SwiGLU pairs: even waves");
  static_assert(!SW || NW / 2 * CB * MT * 4 * 64 * 4 <= (int)sizeof(lds), "SwiGLU exchange buffer");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, cl = lane & 15;
  // the K-split is the fastest grid dimension: workgroups are dealt to the 8 XCDs in
  // linear order, so each XCD's L2 sees only its splits' slice of the activations.
  // With row tiles (a 1-D grid), workgroup id goes to XCD id % 8 and its (id / 8)-th slot
  // there; an XCD's consecutive slots take every row tile of one (split, column group),
  // so the tiles that stream the same weights run together and share the XCD's L2.
  int split, cgroup, rbeg = 0, rend = M;
  if (row_tiles > 0) {
    const int id = blockIdx.x, slot = id >> 3;
    const int oct = slot / row_tiles, tile = slot - oct * row_tiles;
    const int xy = oct * 8 + (id & 7);
    if (xy >= splits * groups) return;  // padding of the last octet
    split = xy % splits;
    cgroup = xy / splits;
    rbeg = tile * C::ROWS;
    rend = min(M, rbeg + C::ROWS);
  } else {
    split = blockIdx.x;
    cgroup = blockIdx.y;
  }
  const int kbeg = split * iters * C::KS;
  const int ks0 = kbeg / C::KSTEP;                   // first global step of the range
  const int ksteps = K / C::KSTEP;

  // column block c of this wave: columns n0[c] .. n0[c]+15, from whichever concatenated
  // matrix holds them (wave-uniform; explicit selects, since a dynamic index into the
  // by-value argument would go to scratch).  A block past the last column (of N, or of
  // the concatenation, whose unused matrix pointers are null) reads block 0 of the
  // first matrix, which always exists, and stores nothing.
  ColBlock cbk[CB];
  int n0[CB];
  bool ok[CB];
#pragma unroll
  for (int c = 0; c < CB; ++c) {
    n0[c] = (cgroup * NW * CB + c * NW + wave) * 16;
    if constexpr (SW) {
      // virtual block v: gate block v/2 (v even) or up block v/2 (v odd); F = nbeg[1]
      const int fb = n0[c] / 32;  // block index within the gate and up matrices
      ok[c] = fb * 16 < w.nbeg[1];
      const int mi = (wave & 1) && ok[c] ? 1 : 0;
      cbk[c].wlane = static_cast<const char*>(mi ? w.mat[1] : w.mat[0]) + lane * 16;
      cbk[c].slane = Q4 ? static_cast<const char*>(mi ? w.scale[1] : w.scale[0]) + cl * 4 : nullptr;
      cbk[c].cb = ok[c] ? fb : 0;
      cbk[c].bm = BlockMap{w.slab, ksteps / w.slab, w.nbeg[1] / 16};
    } else {
      ok[c] = n0[c] < N && n0[c] < w.nbeg[3];
      const int nn = ok[c] ? n0[c] : 0;
      const int mi = nn >= w.nbeg[2] ? 2 : (nn >= w.nbeg[1] ? 1 : 0);
      const void* mat = mi == 2 ? w.mat[2] : (mi == 1 ? w.mat[1] : w.mat[0]);
      const void* scl = mi == 2 ? w.scale[2] : (mi == 1 ? w.scale[1] : w.scale[0]);
      const int nb = mi == 2 ? w.nbeg[2] : (mi == 1 ? w.nbeg[1] : w.nbeg[0]);
      const int ne = mi == 2 ? w.nbeg[3] : (mi == 1 ? w.nbeg[2] : w.nbeg[1]);
      cbk[c].wlane = static_cast<const char*>(mat) + lane * 16;
      cbk[c].slane = Q4 ? static_cast<const char*>(scl) + cl * 4 : nullptr;
      cbk[c].cb = (nn - nb) / 16;
      cbk[c].bm = BlockMap{w.slab, ksteps / w.slab, (ne - nb) / 16};
    }
  }

  // fused SwiGLU: the rows' sums of squares (M * nb <= THREADS floats, checked by the
  // plan) are loaded ahead of the first slice, so the prologue's wait for the activations
  // covers them, and kept in LDS for the epilogue
  __shared__ float sm_ss[SW ? C::THREADS : 1];
  float ssv = 0.f;
  if constexpr (SW) ssv = so.ss[min(rbeg * so.nb + tid, M * so.nb - 1)];
  __builtin_amdgcn_sched_barrier(0);

  for (int r0 = rbeg; r0 < rend; r0 += C::ROWS) {
    f32x4 acc[C::NA][MT][CB];
#pragma unroll
    for (int a = 0; a < C::NA; ++a)
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int c = 0; c < CB; ++c) acc[a][t][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    WTile<Q4, CB, STEPS> w0, w1;
    uint4 ar[C::NP * C::AU];
    load_a<C>(ar, X, Xlo, M, K, r0, kbeg);
    load_w<Q4, STEPS, CB>(w0, cbk, ks0);
    store_a<C>(lds[0], ar);
    if constexpr (SW) {  // (visible after the first barrier below)
      if (r0 == rbeg && tid < (rend - rbeg) * so.nb) sm_ss[tid] = ssv;
    }
    int i = 0;
    // steady state, two slices per trip: every load is unconditional
    // (with MXFP4 weights, scheduling barriers keep each slice's loads ahead of the
    // previous slice's products; the scheduler would otherwise sink them to their use)
    for (; i + 2 < iters; i += 2) {
      __syncthreads();  // lds[0] holds slice i; lds[1] is free
      load_a<C>(ar, X, Xlo, M, K, r0, kbeg + (i + 1) * C::KS);
      load_w<Q4, STEPS, CB>(w1, cbk, ks0 + (i + 1) * STEPS);
      if constexpr (Q4) __builtin_amdgcn_sched_barrier(0);
      mma_slice<T, C>(lds[0], w0, cl, g, acc);
      store_a<C>(lds[1], ar);
      __syncthreads();  // lds[1] holds slice i+1; lds[0] is free
      load_a<C>(ar, X, Xlo, M, K, r0, kbeg + (i + 2) * C::KS);
      load_w<Q4, STEPS, CB>(w0, cbk, ks0 + (i + 2) * STEPS);
      if constexpr (Q4) __builtin_amdgcn_sched_barrier(0);
      mma_slice<T, C>(lds[1], w1, cl, g, acc);
      store_a<C>(lds[0], ar);
    }
    // the last one or two slices
    __syncthreads();
    if (i + 1 < iters) {
      load_a<C>(ar, X, Xlo, M, K, r0, kbeg + (i + 1) * C::KS);
      load_w<Q4, STEPS, CB>(w1, cbk, ks0 + (i + 1) * STEPS);
      if constexpr (Q4) __builtin_amdgcn_sched_barrier(0);
      mma_slice<T, C>(lds[0], w0, cl, g, acc);
      store_a<C>(lds[1], ar);
      __syncthreads();
      mma_slice<T, C>(lds[1], w1, cl, g, acc);
    } else {
      mma_slice<T, C>(lds[0], w0, cl, g, acc);
    }
    if constexpr (SW) {
      // the up wave of each pair hands its sums to the gate wave (same lanes, same rows)
      __syncthreads();  // every wave is done with the staged activations
      float* xs = reinterpret_cast<float*>(&lds[0][0]);  // [NW/2 pairs][CB][MT][4][64 lanes]
      const int pair = wave >> 1;
      if (wave & 1) {
#pragma unroll
        for (int c = 0; c < CB; ++c)
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            f32x4 v = acc[0][t][c];
            if (C::NA == 2) v += acc[C::NA - 1][t][c];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) xs[(((pair * CB + c) * MT + t) * 4 + jj) * 64 + lane] = v[jj];
          }
      }
      __syncthreads();
      if (!(wave & 1)) {
        T* act = static_cast<T*>(so.act);
        T* act_lo = static_cast<T*>(so.act_lo);
#pragma unroll
        for (int c = 0; c < CB; ++c) {
          if (!ok[c]) continue;
          const int f = (n0[c] / 32) * 16 + cl;  // output column in [0, F)
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            f32x4 v = acc[0][t][c];
            if (C::NA == 2) v += acc[C::NA - 1][t][c];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const int r = r0 + t * 16 + 4 * g + jj;
              if (r < M) {
                const float inv = row_inv(sm_ss, r - rbeg, so.nb, so.d, so.eps);
                const float a = v[jj] * inv;
                const float b = xs[(((pair * CB + c) * MT + t) * 4 + jj) * 64 + lane] * inv;
                store_act(act, act_lo, (int64_t)r * so.F + f, a / (1.f + __expf(-a)) * b);
              }
            }
          }
        }
      }
    } else {
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        if (ok[c]) {
          const int n = n0[c] + cl;
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            f32x4 v = acc[0][t][c];
            if (C::NA == 2) v += acc[C::NA - 1][t][c];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const int r = r0 + t * 16 + 4 * g + jj;
              if (r < M) P[((int64_t)split * M + r) * N + n] = v[jj];
            }
          }
        }
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

template <typename T, bool Q4, int STEPS, int NW, int MT, int CB, bool SW>
hipError_t launch_t(const void* X, const void* Xlo, int M, int K, const WeightCat& w, int N,
                    int iters, int row_tiles, float* P, const SwigluOut& so, hipStream_t s) {
  using C = GemmCfg<T, Q4, STEPS, NW, MT, CB>;
  const int splits = K / (C::KS * iters), groups = (N + 16 * NW * CB - 1) / (16 * NW * CB);
  // row tiles: one tile of C::ROWS rows per workgroup (and, fused, its rows' sums of
  // squares staged one per thread)
  if (row_tiles > 0 && (row_tiles != (M + C::ROWS - 1) / C::ROWS ||
                        (SW && (C::ROWS * so.nb > C::THREADS || splits != 1))))
    return hipErrorInvalidValue;
  const dim3 grid = row_tiles > 0 ? dim3((splits * groups + 7) / 8 * 8 * row_tiles, 1)
                                   : dim3(splits, groups);
  SPP_LAUNCH((gemm_kernel<T, Q4, STEPS, NW, MT, CB, SW>), grid, dim3(64 * NW), 0, s,
                     static_cast<const T*>(X), static_cast<const T*>(Xlo), M, K, w, N, iters, P,
                     so, row_tiles, splits, groups);
  return hipGetLastError();
}

// The instantiated launch shapes (waves, 16-row tiles, column blocks per wave, steps per
// slice): those the plans below pick, for dtype and MXFP4 weights, with and without the
// fused SwiGLU.
#ifndef SPP_GEMM_SHAPES
#define SPP_GEMM_SHAPES(X) \
  X(16, 1, 1, 2) X(16, 1, 1, 4) X(16, 2, 1, 2) X(16, 2, 1, 4) X(16, 4, 1, 2) X(16, 4, 1, 4) \
  X(16, 8, 1, 1) X(8, 8, 2, 1) X(4, 2, 2, 2) X(4, 2, 2, 1)                                   \
  X(4, 1, 2, 2) X(5, 1, 2, 2) X(6, 1, 2, 2) X(8, 1, 2, 2) X(5, 2, 2, 2) X(6, 2, 2, 2)       \
  X(8, 2, 2, 2) X(4, 4, 4, 1) \
  X(4, 1, 2, 4) X(5, 1, 2, 4) X(6, 1, 2, 4) X(8, 1, 2, 4) X(4, 2, 2, 4) X(5, 2, 2, 4) X(6, 2, 2, 4) \
  X(8, 2, 2, 4)
#endif
#ifndef SPP_GEMM_SWIGLU_SHAPES
#define SPP_GEMM_SWIGLU_SHAPES(X) \
  X(8, 1, 1, 4) X(8, 2, 1, 4) X(8, 4, 1, 4) X(8, 1, 1, 2) X(8, 2, 1, 2) X(8, 4, 1, 2) \
  X(10, 1, 1, 2) X(10, 2, 1, 2) X(12, 1, 1, 2) X(12, 2, 1, 2) X(14, 1, 1, 2) X(14, 2, 1, 2) \
  X(16, 1, 1, 2) X(16, 2, 1, 2) \
  X(4, 4, 4, 1)
#endif
#ifndef SPP_GEMM_Q4_SHAPES
#define SPP_GEMM_Q4_SHAPES(X) X(8, 1, 2, 1) X(8, 2, 2, 1) X(8, 4, 2, 1) X(8, 8, 2, 1) X(8, 2, 4, 1)
#endif
#ifndef SPP_GEMM_Q4_SWIGLU_SHAPES
#define SPP_GEMM_Q4_SWIGLU_SHAPES(X) X(8, 1, 2, 1) X(8, 2, 2, 1) X(8, 4, 2, 1)
#endif

template <typename T, bool Q4, bool SW>
hipError_t launch(const k::GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                  const WeightCat& w, int N, float* P, const SwigluOut& so, hipStream_t s) {
#define SPP_GEMM_TRY(nw_, mt_, cb_, st_)                                                    \
  if (p.nw == nw_ && p.mt == mt_ && p.cb == cb_ && p.steps == st_)                          \
    return launch_t<T, Q4, st_, nw_, mt_, cb_, SW>(X, Xlo, M, K, w, N, p.iters, p.row_tiles, P, \
                                                   so, s);
  if constexpr (Q4 && SW) {
    SPP_GEMM_Q4_SWIGLU_SHAPES(SPP_GEMM_TRY)
  } else if constexpr (Q4) {
    SPP_GEMM_Q4_SHAPES(SPP_GEMM_TRY)
  } else if constexpr (SW) {
    SPP_GEMM_SWIGLU_SHAPES(SPP_GEMM_TRY)
  } else {
    SPP_GEMM_SHAPES(SPP_GEMM_TRY)
  }
#undef SPP_GEMM_TRY
  return hipErrorInvalidValue;
}

}  // namespace

namespace k {

// Launch shape for one projection, from sweeps on MI355X at the 8B projection sizes with
// the split (hi, lo) activations (M = 32 and 128):
//   * up to 64 rows: 16-wave workgroups of one column block per wave; 4-step slices for
//     the wide MLP gate/up projection (N >= 16384), 2-step slices elsewhere;
//   * 128-row tiles: 1-step slices (the LDS reads of the activation tile dominate), the
//     gate/up projection with 8-wave workgroups of two column blocks per wave;
//   * the K-range is split as finely as keeps the grid within one workgroup per CU
//     (256) with at least two pipelined slices per workgroup: a second wave of
//     workgroups, or shorter pipelines, cost more than the idle CUs.
GemmPlan gemm_plan(const Shape& s, int M, int N, int K) {
  GemmPlan p{};
  const int kstep = kStepBytes / (s.bf16 ? 2 : 4);
  const int ksteps = K / kstep;
  p.mt = M <= 16 ? 1 : (M <= 32 ? 2 : (M <= 64 ? 4 : 8));
  if (p.mt <= 2 && N < 16384 && ksteps % 2 == 0) {
    // up to 32 rows, projections narrower than 16384 outputs: 4-wave workgroups of two
    // column blocks per wave in 2-step slices fill the chip with half the K-splits of
    // 16-wave workgroups, so the consumer reads half the partials.  Where the K-splits
    // that divide the slices leave that grid below 80% of the 256 CUs, 5, 6 or 8 waves per
    // workgroup are tried for the fullest grid.  Fewer waves per workgroup, or one column
    // block per wave, measured slower: the loads in flight per CU fall.  Where the grid had
    // to be widened and a second workgroup per CU would fill it (the 32B QKV and O
    // projections: 512 workgroups of 5 waves), 4-step slices at one workgroup per CU keep
    // the same weight bytes in flight with half the K-splits, so the consumer reads half
    // the partials: QKV + epilogue and O + residual together 1.4-4 µs less per layer than
    // the two-per-CU plan (the 32B QKV: 5 waves, 4 splits of 5 slices; O: 8 splits of 4).
    auto fill = [&](int nw, int cap, int min_slices, int n_slices, int* sp_out) {
      const int groups = (N + 32 * nw - 1) / (32 * nw);
      int best = 0;
      for (int sp = 1; sp <= n_slices; ++sp)
        if (n_slices % sp == 0 && (sp == 1 || n_slices / sp >= min_slices) && groups * sp <= cap)
          best = sp;
      *sp_out = best;
      return groups * best;
    };
    p.cb = 2;
    p.steps = 2;
    p.nw = 4;
    int slices = ksteps / 2;
    int w = fill(4, 256, 2, slices, &p.splits);
    if (w < 205) {
      bool wide = false;  // a second workgroup per CU would fill the grid
      int sp2 = 0;
      for (int nw : {4, 5, 6, 8})
        if (fill(nw, 512, 4, slices, &sp2) >= 410) {
          wide = true;
          break;
        }
      int cap = 256, min_slices = 2;
      if (wide && ksteps % 4 == 0) {
        p.steps = 4;
        slices = ksteps / 4;
        min_slices = 4;
        w = fill(4, cap, min_slices, slices, &p.splits);
      } else if (wide) {  // (no 4-step slices: two workgroups per CU)
        cap = 512;
        min_slices = 4;
        w = fill(4, cap, min_slices, slices, &p.splits);
      }
      for (int nw : {5, 6, 8}) {
        int sp = 0;
        const int wn = fill(nw, cap, min_slices, slices, &sp);
        if (wn > w) {
          w = wn;
          p.nw = nw;
          p.splits = sp;
        }
      }
    }
    p.iters = slices / p.splits;
    return p;
  }
  if (M > 256) {
    // many rows (the batched sessions' entries): every workgroup runs one 64-row tile over
    // the K-range of its split instead of passes over all rows, so each weight byte is read
    // from HBM once per split and shared by the tiles through the XCD's L2; four column
    // blocks per wave make each activation fragment read from LDS feed four matrix-core
    // steps (one or two per read left the projections bound by LDS reads), and the 64-row
    // tile keeps a wave within 256 registers, so two 4-wave workgroups share a CU.  The
    // K-split count (dividing the slices, >= 2 slices each, at most 8) is the smallest that
    // fills the rounds of 512 resident workgroups to 85%, else the one that fills them best.
    p.mt = 4;
    p.nw = 4;
    p.cb = 4;
    p.steps = 1;
    p.row_tiles = (M + 63) / 64;
    const int groups = (N + 255) / 256;
    double best = -1.0;
    p.splits = 1;
    for (int sp = 1; sp <= 8 && sp <= ksteps / 2; ++sp) {
      if (ksteps % sp) continue;
      const int w = p.row_tiles * groups * sp;
      const double eff = (double)w / (((w + 511) / 512) * 512.0);
      if (eff > best + 1e-9) {
        best = eff;
        p.splits = sp;
      }
      if (eff >= 0.85) break;
    }
    p.iters = ksteps / p.splits;
    return p;
  }
  if (p.mt == 8) {
    p.steps = 1;
    if (N >= 16384) { p.nw = 8; p.cb = 2; } else { p.nw = 16; p.cb = 1; }
  } else {
    p.nw = 16; p.cb = 1;
    p.steps = N >= 16384 && ksteps % 4 == 0 ? 4 : 2;
  }
  while (p.steps > 1 && ksteps % p.steps) p.steps >>= 1;
  const int slices = ksteps / p.steps;
  const int groups = (N + 16 * p.nw * p.cb - 1) / (16 * p.nw * p.cb);
  // most splits that divide the slices, keep >= 2 slices each and fit 256 workgroups
  int best = 1;
  for (int sp = 1; sp <= slices; ++sp)
    if (slices % sp == 0 && (sp == 1 || slices / sp >= 2) && sp * groups <= 256) best = sp;
  p.splits = best;
  p.iters = slices / best;
  return p;
}

hipError_t gemm(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                const WeightCat& w, int N, float* partials, hipStream_t st) {
  if (M <= 0 || p.iters < 1 || (s.bf16 && !Xlo) || w.slab < 1 || (K * (s.bf16 ? 2 : 4) / kStepBytes) % w.slab)
    return hipErrorInvalidValue;
  const SwigluOut none{};
  return s.bf16 ? launch<bf16_t, false, false>(p, X, Xlo, M, K, w, N, partials, none, st)
                : launch<float, false, false>(p, X, Xlo, M, K, w, N, partials, none, st);
}

// The fused gate/up + SwiGLU projection (no K-splits): 8-wave workgroups of four gate/up
// block pairs (64 output columns) cover the full K in 4-step slices; used up to 64 rows,
// where the grid (F / 64 workgroups; 224 for F = 14336) still fills the chip.  Up to 32
// rows, when a wider workgroup leaves the busiest CU fewer column blocks (one workgroup
// per CU: rounds of 256 workgroups times the waves of each), 10-16 waves in 2-step slices
// within 128 registers take the projection in fewer rounds: F = 27648 gives 432 8-wave
// workgroups (256, then 176 with a third of the CUs idle) or 247 of 14 waves in one round,
// 8.5% faster.  Larger row counts return splits = 0: they take gemm_plan's split-K plan
// and the SwiGLU kernel.
GemmPlan gemm_plan_swiglu(const Shape& s, int M, int F, int K) {
  GemmPlan p{};
  const int kstep = kStepBytes / (s.bf16 ? 2 : 4);
  const int ksteps = K / kstep;
  if (M > 256 && s.bf16 && F % 128 == 0 && 64 * res_blocks(s) <= 256) {
    // many rows: the 64-row tiles of gemm_plan over the full K (the SwiGLU needs every
    // split's sum), gate and up column blocks on alternate waves as below
    p.mt = 4;
    p.nw = 4;
    p.cb = 4;
    p.steps = 1;
    p.iters = ksteps;
    p.splits = 1;
    p.row_tiles = (M + 63) / 64;
    return p;
  }
  if (M > 64 || F % 16 || M * res_blocks(s) > 512) return p;  // splits = 0: not fused
  p.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  p.nw = 8;
  p.cb = 1;
  p.steps = ksteps % 4 == 0 ? 4 : 2;
  if (p.mt <= 2 && ksteps % 2 == 0) {
    const int blocks = 2 * ((F + 15) / 16);  // gate and up column blocks
    auto busiest = [&](int nw) {               // column blocks of the busiest CU
      const int groups = (blocks + nw - 1) / nw;
      return (groups + 255) / 256 * nw;
    };
    for (int nw : {10, 12, 14, 16})
      if (busiest(nw) < busiest(p.nw)) {
        p.nw = nw;
        p.steps = 2;
      }
  }
  if (ksteps % p.steps) return GemmPlan{};
  p.iters = ksteps / p.steps;
  p.splits = 1;
  return p;
}

hipError_t gemm_swiglu(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M,
                       int K, const WeightCat& w, int F, const float* ss, void* act, void* act_lo,
                       hipStream_t st) {
  if (M <= 0 || p.splits != 1 || p.iters < 1 || (s.bf16 && !Xlo) || w.slab < 1 ||
      (K * (s.bf16 ? 2 : 4) / kStepBytes) % w.slab || w.nbeg[1] != F || w.nbeg[2] != 2 * F)
    return hipErrorInvalidValue;
  const SwigluOut so{ss, res_blocks(s), s.d, s.eps, act, act_lo, F};
  return s.bf16 ? launch<bf16_t, false, true>(p, X, Xlo, M, K, w, 2 * F, nullptr, so, st)
                : launch<float, false, true>(p, X, Xlo, M, K, w, 2 * F, nullptr, so, st);
}

int pack_slab_steps_gateup(const Shape& s, int F, int K) {
  const GemmPlan p = gemm_plan_swiglu(s, 32, F, K);
  return p.splits == 1 ? p.steps * p.iters : pack_slab_steps(s, 2 * F, K);
}

int pack_slab_steps(const Shape& s, int N, int K) {
  const GemmPlan p = gemm_plan(s, 32, N, K);
  return p.steps * p.iters;
}

// MXFP4 launch shape (K-steps of 128 elements), from sweeps at the 70B projection sizes:
// 8-wave workgroups of two column blocks per wave (one A fragment from LDS feeds both,
// which halves the LDS reads per weight byte: with a 4-bit weight feeding four times the
// products of a bf16 one, those reads and the matrix cores, not HBM, bound the kernel),
// 1-step slices; the fewest K-splits whose grid fills the chip once, with at least two
// slices each (the fp32 partials weigh more against 4-bit weights than against bf16).
// The wide MLP gate/up at 17-32 rows (N >= 32768, run unfused: see gemm_plan_swiglu_fp4)
// takes four column blocks per wave instead, so each A fragment feeds four products, with
// the most K-splits that keep the grid within one round (the 70B MLP: 2 splits, 224
// workgroups): 79.7-81.7 -> 68.8-69.4 µs plus a 5.5 µs SwiGLU against the fused kernel.
// Four blocks for the other 70B projections measured no better (QKV, down) or slower (O).
GemmPlan gemm_plan_fp4(const Shape& s, int M, int N, int K) {
  (void)s;
  GemmPlan p{};
  const int ksteps = K / kQ4Step;
  p.mt = M <= 16 ? 1 : (M <= 32 ? 2 : (M <= 64 ? 4 : 8));
  const bool wide = N >= 32768 && p.mt == 2;
  p.nw = 8;
  p.cb = wide ? 4 : 2;
  p.steps = 1;
  const int slices = ksteps / p.steps;
  const int groups = (N + 16 * p.nw * p.cb - 1) / (16 * p.nw * p.cb);
  int best = 1;
  for (int sp = 1; sp <= slices; ++sp) {
    if (slices % sp || (sp > 1 && slices / sp < 2)) continue;
    if (wide && sp > 1 && sp * groups > 256) break;
    best = sp;
    if (sp * groups >= 256) break;
  }
  p.splits = best;
  p.iters = slices / best;
  return p;
}

int pack_slab_steps_fp4(const Shape& s, int N, int K) {
  const GemmPlan p = gemm_plan_fp4(s, 32, N, K);
  return p.steps * p.iters;
}

hipError_t gemm_fp4(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                    const WeightCat& w, int N, float* partials, hipStream_t st) {
  if (M <= 0 || p.iters < 1 || !s.bf16 || !Xlo || w.slab < 1 || K % kQ4Step ||
      (K / kQ4Step) % w.slab || (K / kQ4Step) % (p.steps * p.iters))
    return hipErrorInvalidValue;
  const SwigluOut none{};
  return launch<bf16_t, true, false>(p, X, Xlo, M, K, w, N, partials, none, st);
}

// Fused gate/up + SwiGLU over MXFP4 weights: 8-wave workgroups of two column blocks per
// wave (four gate/up pairs of two blocks: 128 output columns) over the full K; up to 64
// rows (F / 128 workgroups: 224 for F = 28672).  splits = 0 where it does not apply.
GemmPlan gemm_plan_swiglu_fp4(const Shape& s, int M, int F, int K) {
  GemmPlan p{};
  const int ksteps = K / kQ4Step;
  if (!s.bf16 || M > 64 || F % 16 || K % kQ4Step || M * res_blocks(s) > 512) return p;
  // 17-32 rows of a wide MLP: unfused, with four column blocks per wave (gemm_plan_fp4)
  if (M > 16 && M <= 32 && 2 * F >= 32768) return p;
  p.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  p.nw = 8;
  p.cb = 2;
  p.steps = 1;
  p.iters = ksteps / p.steps;
  p.splits = 1;
  return p;
}

hipError_t gemm_swiglu_fp4(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M,
                           int K, const WeightCat& w, int F, const float* ss, void* act,
                           void* act_lo, hipStream_t st) {
  if (M <= 0 || p.splits != 1 || p.iters < 1 || !s.bf16 || !Xlo || w.slab < 1 || K % kQ4Step ||
      (K / kQ4Step) % w.slab || w.nbeg[1] != F || w.nbeg[2] != 2 * F)
    return hipErrorInvalidValue;
  const SwigluOut so{ss, res_blocks(s), s.d, s.eps, act, act_lo, F};
  return launch<bf16_t, true, true>(p, X, Xlo, M, K, w, 2 * F, nullptr, so, st);
}

int pack_slab_steps_gateup_fp4(const Shape& s, int F, int K) {
  const GemmPlan p = gemm_plan_swiglu_fp4(s, 32, F, K);
  return p.splits == 1 ? p.steps * p.iters : pack_slab_steps_fp4(s, 2 * F, K);
}

hipError_t pack_weight(int elem_bytes, const void* src, void* dst, int N, int K, int slab,
                       hipStream_t st) {
  const int KU = K * elem_bytes / 16;
  if (N % 16 || (K * elem_bytes) % kStepBytes || slab < 1 || (KU / 8) % slab)
    return hipErrorInvalidValue;
  const int64_t total = (int64_t)N * KU;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  SPP_LAUNCH(pack_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), N, KU, slab);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
