// Vocabulary-sized work: the LM head at the decision point with its reductions
// fused in, and the serve-time scan of a cached distribution.
//
// lmhead_gemv: one row z = rmsnorm(x_last) * g_final against W_lm[V][d] (the largest
// single weight stream of the step).  Each lane keeps its slice of z in registers
// and streams two weight rows at a time (all loads of both rows in flight; the rows
// are dealt to the waves of the whole grid in turn, so that together they read one
// compact window of W_lm), a butterfly shuffle sums each row, and the same wave keeps
// a running top-2 (value desc, index asc), a running (max, sum of exp) for the
// log-sum-exp and a nonfinite flag.  A second kernel merges the workgroup partials in
// a fixed tree order, so the result is deterministic (no per-workgroup fences).
//
// scan: the same reductions over already computed fp32 distributions (the gate's
// vocabulary scan, and the batched LM head's), one grid column per distribution, then
// one merge workgroup for the whole batch.
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

struct Acc {  // running reductions
  Top2 t;
  float m, s;
  uint32_t nonfinite;
};

__device__ __forceinline__ void acc_init(Acc& a) {
  top2_init(a.t);
  a.m = -INFINITY;
  a.s = 0.f;
  a.nonfinite = 0;
}

__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;
  s = (m == -INFINITY ? 0.f : s * __expf(m - M)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - M));
  m = M;
}

__device__ __forceinline__ void acc_push(Acc& a, float v, int i, bool with_lse) {
  if (isnan(v)) {
    a.nonfinite = 1;
    return;
  }
  if (isinf(v)) a.nonfinite = 1;
  top2_push(a.t, v, i);
  if (with_lse && !isinf(v)) {
    if (v > a.m) {
      a.s = a.s * __expf(a.m - v) + 1.f;
      a.m = v;
    } else {
      a.s += __expf(v - a.m);
    }
  }
}

__device__ __forceinline__ void acc_merge(Acc& a, const Acc& b) {
  top2_merge(a.t, b.t);
  lse_merge(a.m, a.s, b.m, b.s);
  a.nonfinite |= b.nonfinite;
}

__device__ __forceinline__ Acc shfl_acc(const Acc& a, int o) {
  Acc b;
  b.t.v1 = __shfl_xor(a.t.v1, o, 64);
  b.t.v2 = __shfl_xor(a.t.v2, o, 64);
  b.t.i1 = __shfl_xor(a.t.i1, o, 64);
  b.t.i2 = __shfl_xor(a.t.i2, o, 64);
  b.m = __shfl_xor(a.m, o, 64);
  b.s = __shfl_xor(a.s, o, 64);
  b.nonfinite = __shfl_xor(a.nonfinite, o, 64);
  return b;
}

__device__ __forceinline__ Acc wave_acc(Acc a) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) acc_merge(a, shfl_acc(a, o));
  return a;
}

__device__ __forceinline__ ScanPartial to_partial(const Acc& a) {
  ScanPartial p;
  p.v1 = a.t.v1;
  p.v2 = a.t.v2;
  p.i1 = a.t.i1;
  p.i2 = a.t.i2;
  p.m = a.m;
  p.s = a.s;
  p.nonfinite = a.nonfinite;
  p.pad = 0;
  return p;
}

__device__ __forceinline__ Acc from_partial(const ScanPartial& p) {
  Acc a;
  a.t.v1 = p.v1;
  a.t.v2 = p.v2;
  a.t.i1 = p.i1;
  a.t.i2 = p.i2;
  a.m = p.m;
  a.s = p.s;
  a.nonfinite = p.nonfinite;
  return a;
}

// Block-level: merge the NW waves' accumulators (wave order), result valid in thread 0.
template <int NW = 4>
__device__ __forceinline__ Acc block_acc(Acc a, ScanPartial* red) {
  a = wave_acc(a);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[wave] = to_partial(a);
  __syncthreads();
  Acc r = from_partial(red[0]);
  for (int w = 1; w < NW; ++w) acc_merge(r, from_partial(red[w]));
  return r;
}

// Merges the `nb` partials of one distribution in a fixed order (so the result does not
// depend on which workgroup finished when) and writes the result to device memory (the
// session's summary, read after the step's completion).  Every thread of the block
// calls it.
__device__ void publish(const ScanPartial* parts, int nb, ScanResult* result,
                        const uint32_t* bitmap, bool with_lse, uint32_t seq, ScanPartial* red,
                        const uint32_t* range) {
  Acc a;
  acc_init(a);
  for (int b = threadIdx.x; b < nb; b += 256) {
    const ScanPartial p = parts[b];
    acc_merge(a, from_partial(p));
  }
  a = block_acc(a, red);
  if (threadIdx.x == 0) {
    ScanResult r;
    r.argmax = a.t.i1;
    r.second = a.t.i2;
    r.top1 = a.t.v1;
    r.top2 = a.t.v2;
    r.lse = (with_lse && !a.nonfinite) ? a.m + __logf(a.s) : __builtin_nanf("");
    uint32_t flags = a.nonfinite ? 1u : 0u;
    if (bitmap && a.t.i1 >= 0 && a.t.i1 != 0x7FFFFFFF)
      flags |= ((bitmap[a.t.i1 >> 5] >> (a.t.i1 & 31)) & 1u) << 1;
    if (range) flags |= *range & kRangeFlag;
    r.flags = flags;
    r.seq = seq;
    r.pad = 0;
    *result = r;
  }
}

// FULL: d is a multiple of 64 * E, so every lane's chunks are in the row and the loads
// need no predicate.
template <typename T, int NC, bool FULL>
__global__ __launch_bounds__(256) void lmhead_kernel(Shape s, const float* __restrict__ x_row,
                                                     const T* __restrict__ gf,
                                                     const T* __restrict__ W,
                                                     const float* __restrict__ bias,
                                                     float* __restrict__ dist,
                                                     const uint32_t* __restrict__ bitmap,
                                                     ScanPartial* parts,
                                                     ScanResult* result) {
  __shared__ ScanPartial red[4];
  constexpr int E = Elem<T>::kPerFrag;
  const int d = s.d, V = s.vocab;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // z slice of this lane: chunk c covers elements [c*64E + lane*E, +E)
  float z[NC][E];
  bool ok[NC];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k0 = c * 64 * E + lane * E;
    ok[c] = FULL || k0 < d;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      z[c][e] = ok[c] ? x_row[k0 + e] : 0.f;
      ss += z[c][e] * z[c][e];
    }
  }
  const float inv = rsqrtf(wave_sum(ss) / d + s.eps);
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < E; ++e)
      z[c][e] = ok[c] ? z[c][e] * inv * load_elem(gf, c * 64 * E + lane * E + e) : 0.f;

  Acc acc;
  acc_init(acc);
  // wave gw takes rows gw, gw + nw, gw + 2 nw, ... (two per trip): at any moment the
  // waves of the grid read one compact window of rows, not one stream per workgroup.
  // Two register sets alternate, so the next trip's rows (and their biases) are in flight
  // while this trip's are reduced.  Every load is unconditional (rows past V read the
  // last row again, never used; without a bias the biases read x_row and are discarded),
  // so the compiler's wait counts stay exact across the trips.
  const int nw = gridDim.x * 4, gw = blockIdx.x * 4 + wave;
  const float* bsrc = bias ? bias : x_row;
  auto issue = [&](int r, uint4 (&a)[NC], uint4 (&b)[NC], float& sa, float& sb) {
    const int ra = r < V ? r : V - 1, rb = r + nw < V ? r + nw : ra;
    const char* pa = reinterpret_cast<const char*>(W + (int64_t)ra * d);
    const char* pb = reinterpret_cast<const char*>(W + (int64_t)rb * d);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int off = (c * 64 * E + lane * E) * Elem<T>::kBytes;
      a[c] = ok[c] ? ld_stream(pa + off) : make_uint4(0, 0, 0, 0);
      b[c] = ok[c] ? ld_stream(pb + off) : make_uint4(0, 0, 0, 0);
    }
    sa = bsrc[bias ? ra : 0];
    sb = bsrc[bias ? rb : 0];
  };
  auto reduce = [&](int r, const uint4 (&a)[NC], const uint4 (&b)[NC], float sa, float sb) {
    const int r2 = r + nw;
    float da = 0.f, db = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float fa[E], fb[E];
      frag_to_f32(a[c], fa);
      frag_to_f32(b[c], fb);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        da += z[c][e] * fa[e];
        db += z[c][e] * fb[e];
      }
    }
    da = wave_sum(da);
    db = wave_sum(db);
    const float la = da + (bias ? sa : 0.f);
    if (lane == 0) dist[r] = la;
    acc_push(acc, la, r, true);
    if (r2 < V) {
      const float lb = db + (bias ? sb : 0.f);
      if (lane == 0) dist[r2] = lb;
      acc_push(acc, lb, r2, true);
    }
  };
  // trips of this wave: rows gw + 2 nw k, k < trips
  const int trips = gw < V ? (V - gw + 2 * nw - 1) / (2 * nw) : 0;
  uint4 wa0[NC], wb0[NC], wa1[NC], wb1[NC];
  float ba0, bb0, ba1, bb1;
  issue(gw, wa0, wb0, ba0, bb0);
  int k = 0;
  for (; k + 2 < trips; k += 2) {
    issue(gw + (k + 1) * 2 * nw, wa1, wb1, ba1, bb1);
    reduce(gw + k * 2 * nw, wa0, wb0, ba0, bb0);
    issue(gw + (k + 2) * 2 * nw, wa0, wb0, ba0, bb0);
    reduce(gw + (k + 1) * 2 * nw, wa1, wb1, ba1, bb1);
  }
  if (k + 1 < trips) {
    issue(gw + (k + 1) * 2 * nw, wa1, wb1, ba1, bb1);
    reduce(gw + k * 2 * nw, wa0, wb0, ba0, bb0);
    reduce(gw + (k + 1) * 2 * nw, wa1, wb1, ba1, bb1);
  } else if (k < trips) {
    reduce(gw + k * 2 * nw, wa0, wb0, ba0, bb0);
  }
  // every lane holds the same wave accumulator; merge the 4 waves
  __syncthreads();
  if (lane == 0) red[wave] = to_partial(acc);
  __syncthreads();
  if (tid == 0) {
    Acc a = from_partial(red[0]);
    for (int w = 1; w < 4; ++w) acc_merge(a, from_partial(red[w]));
    parts[blockIdx.x] = to_partial(a);
  }
}

// The LM head's second phase: merges the workgroups' partials in order and publishes.
__global__ __launch_bounds__(256) void lmhead_merge_kernel(const ScanPartial* parts, int nb,
                                                           ScanResult* result,
                                                           const uint32_t* bitmap,
                                                           const uint32_t* range) {
  __shared__ ScanPartial red[4];
  publish(parts, nb, result, bitmap, true, 1u, red, range);
}

// First phase of a scan: grid (blocks, distributions).  Block x of distribution b takes
// an equal share of the vocabulary's 16-byte units (the last block also takes the scalar
// tail when vocab % 4 != 0) and keeps four of its loads in flight per thread.  With
// `src`, dist[b][v] = sum over splits of src[split][b][v] (+ bias[v]) is formed and
// stored on the way.
__device__ __forceinline__ float4 scan_load4(const k::ScanJob& job, const float* dist, const float* src,
                                             int64_t sstride, int v) {
  if (!src) return *reinterpret_cast<const float4*>(dist + v);
  float4 q = *reinterpret_cast<const float4*>(src + v);
  for (int k = 1; k < job.src_splits; ++k) {
    const float4 p = *reinterpret_cast<const float4*>(src + k * sstride + v);
    q.x += p.x;
    q.y += p.y;
    q.z += p.z;
    q.w += p.w;
  }
  if (job.bias) {
    const float4 bb = *reinterpret_cast<const float4*>(job.bias + v);
    q.x += bb.x;
    q.y += bb.y;
    q.z += bb.z;
    q.w += bb.w;
  }
  return q;
}

template <int TPB>
__global__ __launch_bounds__(TPB) void scan_kernel(int V, k::ScanJob job) {
  __shared__ ScanPartial red[TPB / 64];
  const int b = blockIdx.y, nb = gridDim.x, n = gridDim.y;
  float* dist = job.dist[b];
  const float* src = job.src ? job.src + (int64_t)b * V : nullptr;
  const int64_t sstride = (int64_t)n * V;  // between partial splits of src
  Acc a;
  acc_init(a);
  if ((V & 3) == 0) {
    const int V4 = V >> 2;
    const int u0 = (int)((int64_t)blockIdx.x * V4 / nb), u1 = (int)((int64_t)(blockIdx.x + 1) * V4 / nb);
    constexpr int IN = 8;  // loads in flight per thread: one round trip per block
                           // (scan_launch gives a block at most ~8 units per thread)
    for (int u = u0 + threadIdx.x; u < u1; u += IN * TPB) {
      float4 q[IN];
#pragma unroll
      for (int i = 0; i < IN; ++i) {
        const int ui = u + i * TPB;
        if (ui < u1) q[i] = scan_load4(job, dist, src, sstride, 4 * ui);
      }
#pragma unroll
      for (int i = 0; i < IN; ++i) {
        const int ui = u + i * TPB;
        if (ui < u1) {
          if (src) *reinterpret_cast<float4*>(dist + 4 * ui) = q[i];
          acc_push(a, q[i].x, 4 * ui, job.with_lse);
          acc_push(a, q[i].y, 4 * ui + 1, job.with_lse);
          acc_push(a, q[i].z, 4 * ui + 2, job.with_lse);
          acc_push(a, q[i].w, 4 * ui + 3, job.with_lse);
        }
      }
    }
  } else {
    const int v0 = (int)((int64_t)blockIdx.x * V / nb), v1 = (int)((int64_t)(blockIdx.x + 1) * V / nb);
    for (int v = v0 + threadIdx.x; v < v1; v += TPB) {
      float y;
      if (src) {
        y = src[v];
        for (int k = 1; k < job.src_splits; ++k) y += src[k * sstride + v];
        if (job.bias) y += job.bias[v];
        dist[v] = y;
      } else {
        y = dist[v];
      }
      acc_push(a, y, v, job.with_lse);
    }
  }
  a = block_acc<TPB / 64>(a, red);
  if (threadIdx.x == 0) job.parts[(int64_t)b * nb + blockIdx.x] = to_partial(a);
}

// Second phase of the scan: ONE workgroup of 16 waves merges every distribution's
// partials (wave w takes distributions w, w + 16, ...; lane l holds partial l, nb <= 64)
// in a fixed order into LDS; then wave 0 writes all results (lane b result b).  When the
// results go to host memory (job.done), that one wave makes them visible to the host
// (one system-scope fence, which writes back its L2) and publishes the batch's sequence
// number: a fence per distribution, or per wave, would write the L2 back that many times.
__global__ __launch_bounds__(1024) void scan_merge_kernel(int n, int nb, k::ScanJob job) {
  __shared__ __attribute__((aligned(32))) ScanResult res[k::kScanMax];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // every partial this lane merges is requested before the first is used: one round trip
  constexpr int PER = k::kScanMax / 16;  // distributions per wave
  ScanPartial pp[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int b = wave + 16 * q;
    if (b < n && lane < nb) pp[q] = job.parts[(int64_t)b * nb + lane];
  }
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int b = wave + 16 * q;
    if (b >= n) break;
    Acc a;
    acc_init(a);
    if (lane < nb) a = from_partial(pp[q]);
    a = wave_acc(a);
    if (lane == 0) {
      ScanResult r;
      r.argmax = a.t.i1;
      r.second = a.t.i2;
      r.top1 = a.t.v1;
      r.top2 = a.t.v2;
      r.lse = (job.with_lse && !a.nonfinite) ? a.m + __logf(a.s) : __builtin_nanf("");
      uint32_t flags = a.nonfinite ? 1u : 0u;
      const uint32_t* bitmap = job.bitmap[b];
      if (bitmap && a.t.i1 >= 0 && a.t.i1 != 0x7FFFFFFF)
        flags |= ((bitmap[a.t.i1 >> 5] >> (a.t.i1 & 31)) & 1u) << 1;
      if (job.flag_src[b]) flags |= *job.flag_src[b] & kRangeFlag;
      r.flags = flags;
      r.seq = job.seq;
      r.pad = 0;
      res[b] = r;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  if (lane < n) {  // two 16-byte stores per result (the record is 32-byte aligned)
    const uint4* src = reinterpret_cast<const uint4*>(&res[lane]);
    uint4* dst = reinterpret_cast<uint4*>(job.result[lane]);
    dst[0] = src[0];
    dst[1] = src[1];
  }
  if (job.done) {
    __threadfence_system();  // every lane's results, before the number the host polls
    if (lane == 0) *reinterpret_cast<volatile uint32_t*>(job.done) = job.seq;
    __threadfence_system();
  }
}

template <typename T>
hipError_t launch_lmhead(const Shape& s, const float* x_row, const void* g_final, const void* w_lm,
                         const float* bias, float* dist, const uint32_t* bitmap,
                         ScanPartial* parts, ScanResult* result, const uint32_t* range,
                         hipStream_t st) {
  constexpr int E = Elem<T>::kPerFrag;
  const int nc = (s.d + 64 * E - 1) / (64 * E);
  const int nb = k::lmhead_blocks(s);
  const T* g = static_cast<const T*>(g_final);
  const T* W = static_cast<const T*>(w_lm);
  const bool full = s.d % (64 * E) == 0;
#define SPP_LMHEAD(NCV)                                                                        \
  if (full)                                                                                    \
    SPP_LAUNCH((lmhead_kernel<T, NCV, true>), dim3(nb), dim3(256), 0, st, s, x_row, g, W, bias, \
               dist, bitmap, parts, result);                                                   \
  else                                                                                         \
    SPP_LAUNCH((lmhead_kernel<T, NCV, false>), dim3(nb), dim3(256), 0, st, s, x_row, g, W, bias, \
               dist, bitmap, parts, result)
  switch (nc) {
    case 1: SPP_LMHEAD(1); break;
    case 2: SPP_LMHEAD(2); break;
    case 4: SPP_LMHEAD(4); break;
    case 8: SPP_LMHEAD(8); break;
    case 10: SPP_LMHEAD(10); break;
    case 16: SPP_LMHEAD(16); break;
    default: return hipErrorInvalidValue;
  }
#undef SPP_LMHEAD
  SPP_LAUNCH(lmhead_merge_kernel, dim3(1), dim3(256), 0, st, parts, nb, result, bitmap, range);
  return hipGetLastError();
}

}  // namespace

namespace k {

// One 4-wave workgroup per CU of the MI355X (256 CUs): measured against 128 to 1024
// workgroups at the 8B and 70B vocabularies, more waves in flight streamed W_lm slower.
#ifndef SPP_LMHEAD_MAX_BLOCKS
#define SPP_LMHEAD_MAX_BLOCKS 256
#endif
int lmhead_blocks(const Shape& s) {
  int nb = (s.vocab + 31) / 32;  // at least 32 rows per block
  return nb < SPP_LMHEAD_MAX_BLOCKS ? (nb < 1 ? 1 : nb) : SPP_LMHEAD_MAX_BLOCKS;
}

hipError_t lmhead_gemv(const Shape& s, const float* x_row, const void* g_final, const void* w_lm,
                       const float* bias, float* dist, const uint32_t* bitmap,
                       ScanPartial* parts, ScanResult* result, const uint32_t* range,
                       hipStream_t st) {
  return s.bf16 ? launch_lmhead<bf16_t>(s, x_row, g_final, w_lm, bias, dist, bitmap, parts,
                                        result, range, st)
                : launch_lmhead<float>(s, x_row, g_final, w_lm, bias, dist, bitmap, parts,
                                       result, range, st);
}

// Launch shape of a scan of n distributions of `vocab` logits: 256-thread blocks, about
// 1024 of them over the batch (a batch of 64 fills the chip four times over; 1024-thread
// blocks, one per CU, measured slower), between 4 and 64 per distribution, and no block
// with fewer than one of the vocabulary's 16-byte units per thread.
void scan_launch(int vocab, int n, int* nb, int* tpb) {
  n = n < 1 ? 1 : n;
  *tpb = 256;
  *nb = 1024 / n;
  if (*nb < 4) *nb = 4;
  if (*nb > kScanMaxBlocks) *nb = kScanMaxBlocks;
  const int cap = (vocab + 4 * *tpb - 1) / (4 * *tpb);
  if (*nb > cap) *nb = cap;
  if (*nb < 1) *nb = 1;
}

int scan_blocks(int vocab, int n) {
  int nb, tpb;
  scan_launch(vocab, n, &nb, &tpb);
  return nb;
}

hipError_t scan(const Shape& s, int n, const ScanJob& job, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (n > kScanMax) return hipErrorInvalidValue;
  int nb, tpb;
  scan_launch(s.vocab, n, &nb, &tpb);
  SPP_LAUNCH(scan_kernel<256>, dim3(nb, n), dim3(tpb), 0, st, s.vocab, job);
  SPP_LAUNCH(scan_merge_kernel, dim3(1), dim3(1024), 0, st, n, nb, job);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
