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
// a merge kernel with one workgroup per distribution.
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

// Block-level: merge the 4 waves' accumulators (wave order), result valid in thread 0.
__device__ __forceinline__ Acc block_acc(Acc a, ScanPartial* red) {
  a = wave_acc(a);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[wave] = to_partial(a);
  __syncthreads();
  Acc r = from_partial(red[0]);
  for (int w = 1; w < 4; ++w) acc_merge(r, from_partial(red[w]));
  return r;
}

// Merges the `nb` partials of one distribution in a fixed order (so the result does not
// depend on which workgroup finished when) and publishes the result: the fields, a
// system-scope fence, then the sequence number the host polls.  Every thread of the
// block calls it.
__device__ void publish(const ScanPartial* parts, int nb, ScanResult* result,
                        const uint32_t* bitmap, bool with_lse, uint32_t seq, ScanPartial* red) {
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
    r.flags = flags;
    r.pad = 0;
    volatile ScanResult* vr = result;
    vr->argmax = r.argmax;
    vr->second = r.second;
    vr->top1 = r.top1;
    vr->top2 = r.top2;
    vr->lse = r.lse;
    vr->flags = r.flags;
    __threadfence_system();
    vr->seq = seq;
    __threadfence_system();
  }
}

template <typename T, int NC>
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
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  // z slice of this lane: chunk c covers elements [c*64E + lane*E, +E)
  float z[NC][E];
  bool ok[NC];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k0 = c * 64 * E + lane * E;
    ok[c] = k0 < d;
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
  // waves of the grid read one compact window of rows, not one stream per workgroup
  const int nw = gridDim.x * 4, gw = blockIdx.x * 4 + wave;
  for (int r = gw; r < V; r += 2 * nw) {
    const int r2 = r + nw;
    const bool has2 = r2 < V;
    uint4 wa[NC], wb[NC];
    const char* pa = reinterpret_cast<const char*>(W + (int64_t)r * d);
    const char* pb = reinterpret_cast<const char*>(W + (int64_t)(has2 ? r2 : r) * d);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int off = (c * 64 * E + lane * E) * Elem<T>::kBytes;
      wa[c] = ok[c] ? ld_stream(pa + off) : make_uint4(0, 0, 0, 0);
      wb[c] = (ok[c] && has2) ? ld_stream(pb + off)
                              : make_uint4(0, 0, 0, 0);
    }
    float da = 0.f, db = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float fa[E], fb[E];
      frag_to_f32(wa[c], fa);
      frag_to_f32(wb[c], fb);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        da += z[c][e] * fa[e];
        db += z[c][e] * fb[e];
      }
    }
    da = wave_sum(da);
    db = wave_sum(db);
    const float la = da + (bias ? bias[r] : 0.f);
    if (lane == 0) dist[r] = la;
    acc_push(acc, la, r, true);
    if (has2) {
      const float lb = db + (bias ? bias[r2] : 0.f);
      if (lane == 0) dist[r2] = lb;
      acc_push(acc, lb, r2, true);
    }
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
                                                           const uint32_t* bitmap) {
  __shared__ ScanPartial red[4];
  publish(parts, nb, result, bitmap, true, 1u, red);
}

__global__ __launch_bounds__(256) void scan_kernel(int V, k::ScanJob job) {
  __shared__ ScanPartial red[4];
  const int b = blockIdx.y, nb = gridDim.x, n = gridDim.y;
  const int per = ((V + nb - 1) / nb + 1023) / 1024 * 1024;
  const int beg = blockIdx.x * per, end = min(V, beg + per);
  float* dist = job.dist[b];
  const bool vec = (V & 3) == 0;
  const float* src = job.src ? job.src + (int64_t)b * V : nullptr;
  const int64_t sstride = (int64_t)n * V;  // between partial splits of src
  Acc a;
  acc_init(a);
  for (int v = beg + 4 * threadIdx.x; v < end; v += 1024) {
    float x[4];
    if (vec && v + 3 < end) {
      float4 q;
      if (src) {
        q = *reinterpret_cast<const float4*>(src + v);
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
        *reinterpret_cast<float4*>(dist + v) = q;
      } else {
        q = *reinterpret_cast<const float4*>(dist + v);
      }
      x[0] = q.x; x[1] = q.y; x[2] = q.z; x[3] = q.w;
#pragma unroll
      for (int e = 0; e < 4; ++e) acc_push(a, x[e], v + e, job.with_lse);
    } else {
      for (int e = 0; e < 4 && v + e < end; ++e) {
        float y;
        if (src) {
          y = src[v + e];
          for (int k = 1; k < job.src_splits; ++k) y += src[k * sstride + v + e];
          if (job.bias) y += job.bias[v + e];
          dist[v + e] = y;
        } else {
          y = dist[v + e];
        }
        acc_push(a, y, v + e, job.with_lse);
      }
    }
  }
  a = block_acc(a, red);
  if (threadIdx.x == 0) job.parts[(int64_t)b * nb + blockIdx.x] = to_partial(a);
}

// Second phase of the scan: one workgroup per distribution merges the first phase's
// partials (the kernel boundary orders them; no per-workgroup fences or tickets, which
// on a multi-XCD device cost an L2 write-back each) and publishes the result.
__global__ __launch_bounds__(256) void scan_merge_kernel(int nb, k::ScanJob job) {
  __shared__ ScanPartial red[4];
  const int b = blockIdx.x;
  publish(job.parts + (int64_t)b * nb, nb, job.result[b], job.bitmap[b], job.with_lse != 0,
          job.seq, red);
}

template <typename T>
hipError_t launch_lmhead(const Shape& s, const float* x_row, const void* g_final, const void* w_lm,
                         const float* bias, float* dist, const uint32_t* bitmap,
                         ScanPartial* parts, ScanResult* result, hipStream_t st) {
  constexpr int E = Elem<T>::kPerFrag;
  const int nc = (s.d + 64 * E - 1) / (64 * E);
  const int nb = k::lmhead_blocks(s);
  const T* g = static_cast<const T*>(g_final);
  const T* W = static_cast<const T*>(w_lm);
#define SPP_LMHEAD(NCV)                                                                        \
  SPP_LAUNCH((lmhead_kernel<T, NCV>), dim3(nb), dim3(256), 0, st, s, x_row, g, W, bias, \
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
  SPP_LAUNCH(lmhead_merge_kernel, dim3(1), dim3(256), 0, st, parts, nb, result, bitmap);
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
                       ScanPartial* parts, ScanResult* result, hipStream_t st) {
  return s.bf16 ? launch_lmhead<bf16_t>(s, x_row, g_final, w_lm, bias, dist, bitmap, parts,
                                        result, st)
                : launch_lmhead<float>(s, x_row, g_final, w_lm, bias, dist, bitmap, parts,
                                       result, st);
}

int scan_blocks(int vocab) {
  int nb = (vocab + 2047) / 2048;
  return nb < 1 ? 1 : (nb > 64 ? 64 : nb);
}

hipError_t scan(const Shape& s, int n, const ScanJob& job, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int nb = scan_blocks(s.vocab);
  SPP_LAUNCH(scan_kernel, dim3(nb, n), dim3(256), 0, st, s.vocab, job);
  SPP_LAUNCH(scan_merge_kernel, dim3(n), dim3(256), 0, st, nb, job);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
