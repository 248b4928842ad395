// Row-wise kernels around the projections: embedding gather + RMSNorm, the QKV
// epilogue (split-K reduction, rotary embedding, KV append in place), residual
// add + RMSNorm, SwiGLU, and the final norm of the decision-point rows.
// All of them are small next to the weight streams; they read the GEMM partials
// once and write their outputs once.
#include <cmath>

#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

__device__ __forceinline__ float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// x[r] = E[token[r]] (fp32), h[r] = x[r] / sqrt(mean(x^2) + eps) * g, and the rotary
// table of row r: (cos, sin) of pos[r] * base^(-2i/dh), angles in double.
template <typename T>
__global__ __launch_bounds__(256) void embed_norm_kernel(Shape s, const StepParams* sp,
                                                         const T* E, const T* g, float* x, T* h,
                                                         T* h_lo, float2* rope) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const int d = s.d;
  const int tok = sp_tokens(sp)[r];
  const T* er = E + (int64_t)tok * d;
  float* xr = x + (int64_t)r * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = load_elem(er, i);
    xr[i] = v;
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum_256(ss, red) / d + s.eps);
  for (int i = threadIdx.x; i < d; i += 256)
    store_act(h, h_lo, (int64_t)r * d + i, xr[i] * inv * load_elem(g, i));
  const int half = s.dh / 2;
  const double P = (double)sp_pos(sp)[r];
  for (int i = threadIdx.x; i < half; i += 256) {
    const double th = P * pow(s.rope_base, -2.0 * i / s.dh);
    double sn, cs;
    sincos(th, &sn, &cs);
    rope[(int64_t)r * half + i] = make_float2((float)cs, (float)sn);
  }
}

// One wave per (row, head) of the fused QKV output.  Heads [0, n_q) are queries,
// [n_q, n_q+n_kv) keys, then values.  Rotates q and k (pairs i, i + dh/2), writes q,
// scaled by qscale, to q_out[row][head][dh], and appends k and v to the session's cache
// at the row's absolute position: K as [kv_head][cap][dh], V transposed as
// [kv_head][dh][cap].
template <typename T>
__global__ __launch_bounds__(64) void qkv_epilogue_kernel(Shape s, const StepParams* sp,
                                                          int layer, const float* P, int splits,
                                                          const float2* rope, float qscale,
                                                          T* q_out, T* q_lo) {
  const int r = blockIdx.x, hh = blockIdx.y;
  const int M = sp->n_rows;
  const int dh = s.dh, half = dh / 2;
  const int N = (s.n_q + 2 * s.n_kv) * dh;
  const int64_t split_stride = (int64_t)M * N;
  const int64_t pr = (int64_t)r * N + (int64_t)hh * dh;
  const int kind = hh < s.n_q ? 0 : (hh < s.n_q + s.n_kv ? 1 : 2);
  const Segment sg = sp->seg[sp_rowseg(sp)[r]];
  const int pos = sp_pos(sp)[r];
  const int64_t cap = sg.cap;
  const int64_t layer_off = (int64_t)layer * 2 * s.n_kv * cap * dh;
  T* kvb = static_cast<T*>(sg.kv) + layer_off;
  for (int i = threadIdx.x; i < half; i += 64) {
    float a = add_splits(0.f, P, split_stride, splits, pr + i);
    float b = add_splits(0.f, P, split_stride, splits, pr + i + half);
    if (kind < 2) {
      const float2 cs = rope[(int64_t)r * half + i];
      const float a2 = a * cs.x - b * cs.y;
      const float b2 = a * cs.y + b * cs.x;
      a = a2;
      b = b2;
    }
    if (kind == 0) {
      const int64_t qo = ((int64_t)r * s.n_q + hh) * dh;
      store_act(q_out, q_lo, qo + i, a * qscale);
      store_act(q_out, q_lo, qo + i + half, b * qscale);
    } else if (kind == 1) {
      const int c = hh - s.n_q;
      T* k = kvb + ((int64_t)c * cap + pos) * dh;
      store_elem(k, i, a);
      store_elem(k, i + half, b);
    } else {
      const int c = hh - s.n_q - s.n_kv;
      T* vt = kvb + (int64_t)s.n_kv * cap * dh + (int64_t)c * dh * cap;
      store_elem(vt, (int64_t)i * cap + pos, a);
      store_elem(vt, (int64_t)(i + half) * cap + pos, b);
    }
  }
}

// x[r] += sum over splits of P[split][r]; then, if g is given, h[r] = rmsnorm(x[r]) * g.
// One 1024-thread block per row: every thread owns float4 column groups c = 4*tid + 4096*k
// and issues the loads of x and of all the split partials of its groups before adding
// them (in split order), so a row costs about one memory round trip.
constexpr int kResidThreads = 1024;
constexpr int kResidMaxGroups = 4;  // d_model up to 16384

template <typename T>
__global__ __launch_bounds__(kResidThreads) void residual_norm_kernel(Shape s, int M,
                                                                      const float* P, int splits,
                                                                      float* x, const T* g, T* h,
                                                                      T* h_lo) {
  __shared__ float red[kResidThreads / 64];
  const int r = blockIdx.x, d = s.d;
  float* xr = x + (int64_t)r * d;
  float4 v[kResidMaxGroups];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kResidMaxGroups; ++k) {
    const int c = 4 * threadIdx.x + 4 * kResidThreads * k;
    if (c < d) {
      v[k] = *reinterpret_cast<const float4*>(xr + c);
      v[k] = add_splits4(v[k], P, (int64_t)M * d, splits, (int64_t)r * d + c);
      *reinterpret_cast<float4*>(xr + c) = v[k];
      ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
    }
  }
  if (g == nullptr) return;
  ss = wave_sum(ss);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kResidThreads / 64; ++w) tot += red[w];
  const float inv = rsqrtf(tot / d + s.eps);
#pragma unroll
  for (int k = 0; k < kResidMaxGroups; ++k) {
    const int c = 4 * threadIdx.x + 4 * kResidThreads * k;
    if (c < d) {
      const float4 o = make_float4(v[k].x * inv * load_elem(g, c), v[k].y * inv * load_elem(g, c + 1),
                                   v[k].z * inv * load_elem(g, c + 2), v[k].w * inv * load_elem(g, c + 3));
      store_act4(h, h_lo, (int64_t)r * d + c, o);
    }
  }
}

// act[r][f] = silu(gate) * up, gate = sum_split P[.][r][f], up = sum_split P[.][r][F + f];
// four consecutive f per thread (F is a multiple of 32).
template <typename T>
__global__ __launch_bounds__(256) void swiglu_kernel(Shape s, int M, const float* P, int splits,
                                                     T* act, T* act_lo) {
  const int F = s.ffn;
  const int64_t N = 2 * (int64_t)F;
  const int64_t total = (int64_t)M * F / 4;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int64_t r = (t * 4) / F, f = t * 4 - r * F;
    const float4 a = add_splits4(z, P, (int64_t)M * N, splits, r * N + f);
    const float4 b = add_splits4(z, P, (int64_t)M * N, splits, r * N + F + f);
    const float4 o = make_float4(a.x / (1.f + __expf(-a.x)) * b.x, a.y / (1.f + __expf(-a.y)) * b.y,
                                 a.z / (1.f + __expf(-a.z)) * b.z, a.w / (1.f + __expf(-a.w)) * b.w);
    store_act4(act, act_lo, t * 4, o);
  }
}

// z[i] = rmsnorm(x[last row of segment i]) * g_final, in the model dtype.
template <typename T>
__global__ __launch_bounds__(256) void final_norm_rows_kernel(Shape s, const StepParams* sp,
                                                              const float* x, const T* g, T* z,
                                                              T* z_lo) {
  __shared__ float red[4];
  const int i = blockIdx.x, d = s.d;
  const Segment sg = sp->seg[i];
  const float* xr = x + (int64_t)(sg.row0 + sg.len - 1) * d;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) ss += xr[k] * xr[k];
  const float inv = rsqrtf(block_sum_256(ss, red) / d + s.eps);
  for (int k = threadIdx.x; k < d; k += 256)
    store_act(z, z_lo, (int64_t)i * d + k, xr[k] * inv * load_elem(g, k));
}

__global__ __launch_bounds__(256) void copy_kernel(uint4* __restrict__ dst,
                                                   const uint4* __restrict__ src, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256)
    dst[i] = src[i];
}

__global__ void copy_tail_kernel(char* dst, const char* src, size_t n) {
  for (size_t i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src[i];
}

}  // namespace

namespace k {

hipError_t embed_norm(const Shape& s, const StepParams* dp, int n_rows, const void* embed,
                      const void* g, float* x, void* h, void* h_lo, float2* rope, hipStream_t st) {
  if (s.bf16)
    hipLaunchKernelGGL(embed_norm_kernel<bf16_t>, dim3(n_rows), dim3(256), 0, st, s, dp,
                       static_cast<const bf16_t*>(embed), static_cast<const bf16_t*>(g), x,
                       static_cast<bf16_t*>(h), static_cast<bf16_t*>(h_lo), rope);
  else
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(n_rows), dim3(256), 0, st, s, dp,
                       static_cast<const float*>(embed), static_cast<const float*>(g), x,
                       static_cast<float*>(h), static_cast<float*>(h_lo), rope);
  return hipGetLastError();
}

hipError_t qkv_epilogue(const Shape& s, const StepParams* dp, int n_rows, int layer,
                        const float* partials, int splits, const float2* rope, void* q_out,
                        void* q_lo, hipStream_t st) {
  dim3 grid(n_rows, s.n_q + 2 * s.n_kv);
  // queries leave pre-scaled by log2(e) / sqrt(dh): the attention softmax works in base 2
  const float qscale = (float)(1.4426950408889634 / std::sqrt((double)s.dh));
  if (s.bf16)
    hipLaunchKernelGGL(qkv_epilogue_kernel<bf16_t>, grid, dim3(64), 0, st, s, dp, layer, partials,
                       splits, rope, qscale, static_cast<bf16_t*>(q_out), static_cast<bf16_t*>(q_lo));
  else
    hipLaunchKernelGGL(qkv_epilogue_kernel<float>, grid, dim3(64), 0, st, s, dp, layer, partials,
                       splits, rope, qscale, static_cast<float*>(q_out), static_cast<float*>(q_lo));
  return hipGetLastError();
}

hipError_t residual_norm(const Shape& s, int n_rows, const float* partials, int splits, float* x,
                         const void* g, void* h, void* h_lo, hipStream_t st) {
  if (s.d % 4 || s.d > 4 * kResidThreads * kResidMaxGroups) return hipErrorInvalidValue;
  if (s.bf16)
    hipLaunchKernelGGL(residual_norm_kernel<bf16_t>, dim3(n_rows), dim3(kResidThreads), 0, st, s,
                       n_rows, partials, splits, x, static_cast<const bf16_t*>(g),
                       static_cast<bf16_t*>(h), static_cast<bf16_t*>(h_lo));
  else
    hipLaunchKernelGGL(residual_norm_kernel<float>, dim3(n_rows), dim3(kResidThreads), 0, st, s,
                       n_rows, partials, splits, x, static_cast<const float*>(g),
                       static_cast<float*>(h), static_cast<float*>(h_lo));
  return hipGetLastError();
}

hipError_t swiglu(const Shape& s, int n_rows, const float* partials, int splits, void* act,
                  void* act_lo, hipStream_t st) {
  const int64_t total = (int64_t)n_rows * s.ffn / 4;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (s.bf16)
    hipLaunchKernelGGL(swiglu_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, st, s, n_rows,
                       partials, splits, static_cast<bf16_t*>(act), static_cast<bf16_t*>(act_lo));
  else
    hipLaunchKernelGGL(swiglu_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st, s, n_rows,
                       partials, splits, static_cast<float*>(act), static_cast<float*>(act_lo));
  return hipGetLastError();
}

hipError_t final_norm_rows(const Shape& s, const StepParams* dp, int n_segs, const float* x,
                           const void* g_final, void* z, void* z_lo, hipStream_t st) {
  if (s.bf16)
    hipLaunchKernelGGL(final_norm_rows_kernel<bf16_t>, dim3(n_segs), dim3(256), 0, st, s, dp, x,
                       static_cast<const bf16_t*>(g_final), static_cast<bf16_t*>(z),
                       static_cast<bf16_t*>(z_lo));
  else
    hipLaunchKernelGGL(final_norm_rows_kernel<float>, dim3(n_segs), dim3(256), 0, st, s, dp, x,
                       static_cast<const float*>(g_final), static_cast<float*>(z),
                       static_cast<float*>(z_lo));
  return hipGetLastError();
}

hipError_t copy_bytes(void* dst, const void* src, size_t n, hipStream_t st) {
  const size_t n16 = n / 16;
  if (n16) {
    size_t blocks = (n16 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<uint4*>(dst), static_cast<const uint4*>(src), n16);
  }
  if (n % 16)
    hipLaunchKernelGGL(copy_tail_kernel, dim3(1), dim3(64), 0, st,
                       static_cast<char*>(dst) + n16 * 16, static_cast<const char*>(src) + n16 * 16,
                       n % 16);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
