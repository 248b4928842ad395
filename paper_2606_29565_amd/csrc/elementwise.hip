// Row-wise kernels around the projections: the embedding gather, the QKV epilogue
// (split-K reduction, rotary embedding, KV append in place), the residual add, SwiGLU,
// and the final norm of the decision-point rows.  All of them are small next to the
// weight streams; they read the GEMM partials once and write their outputs once.
//
// RMSNorm is split across kernels.  It scales each row, so
//   (RMSNorm(x) * g) W = inv * ((x * g) W),   inv = 1 / sqrt(mean(x^2) + eps).
// The kernel that produces x (embedding, residual) writes y = x * g as the projection's
// input, plus the sums of squares of x over 1024-column blocks.  The kernel that consumes
// the projection's split sums (QKV epilogue, SwiGLU) multiplies them by inv.  No kernel
// has to see a whole row at once, so the row kernels spread over (row, block) grids.
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

// Grid (rows, blocks of 1024 columns): x[r] = E[token[r]] (fp32), y[r] = x[r] * g in the
// (hi, lo) split, ss[r][block] = sum of x^2 over the block; block 0 also writes the
// rotary table of row r: (cos, sin) of pos[r] * base^(-2i/dh), angles in double.
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(Shape s, StepView sv, const T* E,
                                                    const T* g, float* x, T* y, T* y_lo,
                                                    float* ss, uint32_t* range) {
  __shared__ float red[4];
  const int r = blockIdx.x, blk = blockIdx.y, d = s.d;
  // the step's range words start clear (every later kernel of the step orders after this)
  if (r == 0 && blk == 0)
    for (int i = threadIdx.x; i < sv.p->n_segments; i += 256) range[i] = 0u;
  const int tok = sv.token[r];
  const int c = blk * 1024 + threadIdx.x * 4;
  float q = 0.f;
  if (c < d) {
    const T* er = E + (int64_t)tok * d + c;
    const float4 v = make_float4(load_elem(er, 0), load_elem(er, 1), load_elem(er, 2), load_elem(er, 3));
    *reinterpret_cast<float4*>(x + (int64_t)r * d + c) = v;
    store_act4(y, y_lo, (int64_t)r * d + c,
               make_float4(v.x * load_elem(g, c), v.y * load_elem(g, c + 1), v.z * load_elem(g, c + 2),
                           v.w * load_elem(g, c + 3)));
    q = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  q = block_sum_256(q, red);
  if (threadIdx.x == 0) ss[(int64_t)r * gridDim.y + blk] = q;
}

__global__ __launch_bounds__(64) void rope_kernel(Shape s, StepView sv, float2* rope) {
  const int r = blockIdx.x, half = s.dh / 2;
  const double P = (double)sv.row[r].pos;
  for (int i = threadIdx.x; i < half; i += 64) {
    const double th = P * pow(s.rope_base, -2.0 * i / s.dh);
    double sn, cs;
    sincos(th, &sn, &cs);
    rope[(int64_t)r * half + i] = make_float2((float)cs, (float)sn);
  }
}

// One wave per (row, head) of the fused QKV output.  Heads [0, n_q) are queries,
// [n_q, n_q+n_kv) keys, then values.  The split sums are scaled by the row's 1 / RMS
// (the projection's input was x * g).  Rotates q and k (pairs i, i + dh/2), writes q,
// scaled by qscale, to q_out[row][head][dh] (fp16 for bf16 models, whose attention
// multiplies in fp16; fp32 otherwise), and appends k and v to the session's cache
// at the row's absolute position: K as [kv_head][cap][dh], V transposed as
// [kv_head][dh][cap].
// With TV (dh / 8 rows or more), the value heads' waves are laid out over (32-row chunk,
// 8 dims) units instead: lane (r, j) takes dims 4j..4j+3 of its row, and each store writes
// 32 consecutive positions of one V^T row (a wave per row writes 2-byte cells scattered
// over dh V^T rows).  The grid can then be wider than M; the extra columns return.
template <typename T, bool TV>
__global__ __launch_bounds__(64) void qkv_epilogue_kernel(Shape s, StepView sv, int M,
                                                          int layer, const float* P, int splits,
                                                          const float* ss, int nb,
                                                          const float2* rope, float qscale,
                                                          T* q_out, T* q_lo, uint32_t* range) {
  // (M comes as an argument, not from the step record, so the partial loads do not
  // wait for a load of the record)
  const int r = blockIdx.x, hh = blockIdx.y;
  const int dh = s.dh, half = dh / 2;
  const int N = (s.n_q + 2 * s.n_kv) * dh;
  const int64_t split_stride = (int64_t)M * N;
  const int64_t pr = (int64_t)r * N + (int64_t)hh * dh;
  const int kind = hh < s.n_q ? 0 : (hh < s.n_q + s.n_kv ? 1 : 2);
  if constexpr (TV) {
    if (kind == 2) {
      // Up to 32 rows (one chunk), unit r takes slice r.  Beyond, units go in groups of 8
      // to one XCD (workgroup i runs on XCD i % 8): the 4 slices of one 32-dim stretch (one
      // 128-byte line of each partial row) for a pair of chunks (one 64-position V^T
      // stretch), so that both the partial lines and the V^T lines they fill stay in one L2.
      const int rr = threadIdx.x & 31, j = threadIdx.x >> 5, lines = dh / 32;
      int chunk = 0, slice = r;
      if (M > 32) {
        const int k = r / 8, G = (k / 8) * 8 + r % 8, within = k % 8;
        chunk = (G / lines) * 2 + within / 4;
        slice = (G % lines) * 4 + within % 4;
      } else if (r >= dh / 8) {
        return;
      }
      const int rw = chunk * 32 + rr;
      if (rw >= M) return;
      const int d0 = slice * 8 + 4 * j;
      const RowInfo ri = sv.row[rw];
      const int64_t cap = ri.cap;
      const float inv = row_inv(ss, rw, nb, s.d, s.eps);
      // split sums in split order, 8 loads in flight (16 would double the kernel's VGPRs
      // and halve its waves in flight for every head)
      const float* pv = P + (int64_t)rw * N + (int64_t)hh * dh + d0;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int k0 = 0; k0 < splits; k0 += 8) {
        float4 t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (k0 + u < splits) t[u] = *reinterpret_cast<const float4*>(pv + (k0 + u) * split_stride);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (k0 + u < splits) v = make_float4(v.x + t[u].x, v.y + t[u].y, v.z + t[u].z, v.w + t[u].w);
      }
      T* vt = static_cast<T*>(ri.kv) + (int64_t)layer * 2 * s.n_kv * cap * dh +
              (int64_t)s.n_kv * cap * dh + (int64_t)(hh - s.n_q - s.n_kv) * dh * cap +
              (int64_t)d0 * cap + ri.pos;
      store_elem(vt, 0, v.x * inv);
      store_elem(vt, cap, v.y * inv);
      store_elem(vt, 2 * cap, v.z * inv);
      store_elem(vt, 3 * cap, v.w * inv);
      return;
    }
  }
  if (r >= M) return;  // (TV grids can be wider than the rows)
  const RowInfo ri = sv.row[r];
  const int seg = ri.seg, pos = ri.pos;
  const int64_t cap = ri.cap;
  const int64_t layer_off = (int64_t)layer * 2 * s.n_kv * cap * dh;
  T* kvb = static_cast<T*>(ri.kv) + layer_off;
  const float inv = row_inv(ss, r, nb, s.d, s.eps);
  for (int i = threadIdx.x; i < half; i += 64) {
    float a = add_splits(0.f, P, split_stride, splits, pr + i) * inv;
    float b = add_splits(0.f, P, split_stride, splits, pr + i + half) * inv;
    if (kind < 2) {
      const float2 cs = rope[(int64_t)r * half + i];
      const float a2 = a * cs.x - b * cs.y;
      const float b2 = a * cs.y + b * cs.x;
      a = a2;
      b = b2;
    }
    if (kind == 0) {
      const int64_t qo = ((int64_t)r * s.n_q + hh) * dh;
      if constexpr (Elem<T>::kBytes == 2) {
        // bf16 models: the attention multiplies in fp16, so q leaves as one fp16 array
        _Float16* qh = reinterpret_cast<_Float16*>(q_out);
        const float qa = a * qscale, qb = b * qscale;
        qh[qo + i] = (_Float16)qa;
        qh[qo + i + half] = (_Float16)qb;
        if (!(fmaxf(fabsf(qa), fabsf(qb)) <= kF16Max)) atomicOr(range + seg, kRangeFlag);
      } else {
        store_act(q_out, q_lo, qo + i, a * qscale);
        store_act(q_out, q_lo, qo + i + half, b * qscale);
      }
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

// Grid (rows, blocks of 1024 columns): x[r] += sum over splits of P[split][r] (added in
// split order, every split's load in flight at once); if g is given, y[r] = x[r] * g in
// the (hi, lo) split; ss[r][block] = sum of x^2 over the block.
template <typename T>
__global__ __launch_bounds__(256) void residual_kernel(Shape s, int M, const float* P, int splits,
                                                       float* x, const T* g, T* y, T* y_lo,
                                                       float* ss) {
  __shared__ float red[4];
  const int r = blockIdx.x, blk = blockIdx.y, d = s.d;
  float* xr = x + (int64_t)r * d;
  const int c = blk * 1024 + threadIdx.x * 4;
  float q = 0.f;
  if (c < d) {
    float4 v = *reinterpret_cast<const float4*>(xr + c);
    v = add_splits4(v, P, (int64_t)M * d, splits, (int64_t)r * d + c);
    *reinterpret_cast<float4*>(xr + c) = v;
    if (g)
      store_act4(y, y_lo, (int64_t)r * d + c,
                 make_float4(v.x * load_elem(g, c), v.y * load_elem(g, c + 1),
                             v.z * load_elem(g, c + 2), v.w * load_elem(g, c + 3)));
    q = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  q = block_sum_256(q, red);
  if (threadIdx.x == 0) ss[(int64_t)r * gridDim.y + blk] = q;
}

// act[r][f] = silu(gate) * up, gate = inv[r] * sum_split P[.][r][f], up = inv[r] *
// sum_split P[.][r][F + f] (inv[r]: the row's 1 / RMS; the projection's input was x * g);
// four consecutive f per thread (F is a multiple of 32).
// (S: the split-count bucket of add_splits4_n, so that the gate and up loads of a thread go
// out together in one round trip)
template <typename T, int S>
__global__ __launch_bounds__(256) void swiglu_kernel(Shape s, int M, const float* P, int splits,
                                                     const float* ss, int nb, T* act, T* act_lo) {
  const int F = s.ffn;
  const int64_t N = 2 * (int64_t)F;
  const int64_t total = (int64_t)M * F / 4;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
    const int64_t r = (t * 4) / F, f = t * 4 - r * F;
    const float inv = row_inv(ss, (int)r, nb, s.d, s.eps);
    float4 a = add_splits4_n<S>(z, P, (int64_t)M * N, splits, r * N + f);
    float4 b = add_splits4_n<S>(z, P, (int64_t)M * N, splits, r * N + F + f);
    a = make_float4(a.x * inv, a.y * inv, a.z * inv, a.w * inv);
    b = make_float4(b.x * inv, b.y * inv, b.z * inv, b.w * inv);
    const float4 o = make_float4(a.x / (1.f + __expf(-a.x)) * b.x, a.y / (1.f + __expf(-a.y)) * b.y,
                                 a.z / (1.f + __expf(-a.z)) * b.z, a.w / (1.f + __expf(-a.w)) * b.w);
    store_act4(act, act_lo, t * 4, o);
  }
}

// z[i] = rmsnorm(x[last row of segment i]) * g_final, in the model dtype.
template <typename T>
__global__ __launch_bounds__(256) void final_norm_rows_kernel(Shape s, StepView sv,
                                                              const float* x, const T* g, T* z,
                                                              T* z_lo) {
  __shared__ float red[4];
  const int i = blockIdx.x, d = s.d;
  const Segment sg = sv.p->seg[i];
  const float* xr = x + (int64_t)(sg.row0 + sg.len - 1) * d;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) ss += xr[k] * xr[k];
  const float inv = rsqrtf(block_sum_256(ss, red) / d + s.eps);
  for (int k = threadIdx.x; k < d; k += 256)
    store_act(z, z_lo, (int64_t)i * d + k, xr[k] * inv * load_elem(g, k));
}

// Sliding-window shift (Sec. 3.6, a mutation that relocates positions): the committed
// cells [delta, delta + n_new) of every layer move down to [0, n_new).  RoPE turns the
// key of position p by the angles p * theta_i, so a key moving from p to p - delta is
// turned back by delta * theta_i; values move unchanged.  One workgroup per (kv head,
// layer, K or V) moves its cells in ascending chunks: every source of a chunk is read
// (and the reads completed) before the workgroup's barrier, and only then is any cell of
// the chunk written, so the in-place move never reads a cell it already overwrote (later
// chunks read only cells above this chunk's destinations).
template <typename T>
__global__ __launch_bounds__(256) void shift_kernel(Shape s, void* kv, int64_t cap, int n_new,
                                                    int delta) {
  constexpr int CH = 64;  // cells per chunk
  __shared__ float2 rot[128];  // (cos, sin) of -delta * theta_i, i < dh / 2
  const int c = blockIdx.x, layer = blockIdx.y, which = blockIdx.z;
  const int dh = s.dh, half = dh / 2;
  T* base = static_cast<T*>(kv) + (int64_t)layer * 2 * s.n_kv * cap * dh;
  if (which == 0) {
    for (int i = threadIdx.x; i < half; i += 256) {
      const double th = -(double)delta * pow(s.rope_base, -2.0 * i / dh);
      double sn, cs;
      sincos(th, &sn, &cs);
      rot[i] = make_float2((float)cs, (float)sn);
    }
    __syncthreads();
    T* K = base + (int64_t)c * cap * dh;
    const int items = CH * half;  // (cell, pair) items of a chunk
    for (int a = 0; a < n_new; a += CH) {
      constexpr int PER = (CH * 64 + 255) / 256;  // items per thread (dh <= 128)
      float va[PER], vb[PER];
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int it = threadIdx.x + q * 256;
        const int cell = a + it / half, i = it % half;
        const bool ok = it < items && cell < n_new;
        const int64_t src = ((int64_t)(ok ? cell : 0) + delta) * dh + i;
        va[q] = load_elem(K, src);
        vb[q] = load_elem(K, src + half);
      }
      __builtin_amdgcn_s_waitcnt(0);  // this thread's reads are complete
      __syncthreads();                // ... and every other thread's
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int it = threadIdx.x + q * 256;
        const int cell = a + it / half, i = it % half;
        if (it < items && cell < n_new) {
          const float2 r = rot[i];
          const int64_t dst = (int64_t)cell * dh + i;
          store_elem(K, dst, va[q] * r.x - vb[q] * r.y);
          store_elem(K, dst + half, va[q] * r.y + vb[q] * r.x);
        }
      }
      __syncthreads();  // the chunk's writes are issued before the next chunk's reads
    }
  } else {
    T* Vt = base + (int64_t)s.n_kv * cap * dh + (int64_t)c * dh * cap;  // [dh][cap]
    constexpr int CV = 256;                    // positions per chunk
    for (int a = 0; a < n_new; a += CV) {
      constexpr int PER = CV * 128 / 256;      // elements per thread (dh <= 128)
      float v[PER];
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int it = threadIdx.x + q * 256;
        const int row = it / CV, pos = a + it % CV;
        const bool ok = row < dh && pos < n_new;
        v[q] = load_elem(Vt, (int64_t)(ok ? row : 0) * cap + (ok ? pos : 0) + delta);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int it = threadIdx.x + q * 256;
        const int row = it / CV, pos = a + it % CV;
        if (row < dh && pos < n_new) store_elem(Vt, (int64_t)row * cap + pos, v[q]);
      }
      __syncthreads();
    }
  }
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

int res_blocks(const Shape& s) { return (s.d + 1023) / 1024; }

hipError_t embed(const Shape& s, const StepView& dp, int n_rows, const void* emb, const void* g,
                 float* x, void* y, void* y_lo, float* ss, float2* rope, uint32_t* range,
                 hipStream_t st) {
  if (s.d % 4) return hipErrorInvalidValue;
  dim3 grid(n_rows, res_blocks(s));
  if (s.bf16)
    SPP_LAUNCH(embed_kernel<bf16_t>, grid, dim3(256), 0, st, s, dp,
                       static_cast<const bf16_t*>(emb), static_cast<const bf16_t*>(g), x,
                       static_cast<bf16_t*>(y), static_cast<bf16_t*>(y_lo), ss, range);
  else
    SPP_LAUNCH(embed_kernel<float>, grid, dim3(256), 0, st, s, dp,
                       static_cast<const float*>(emb), static_cast<const float*>(g), x,
                       static_cast<float*>(y), static_cast<float*>(y_lo), ss, range);
  SPP_LAUNCH(rope_kernel, dim3(n_rows), dim3(64), 0, st, s, dp, rope);
  return hipGetLastError();
}

hipError_t qkv_epilogue(const Shape& s, const StepView& dp, int n_rows, int layer,
                        const float* partials, int splits, const float* ss, const float2* rope,
                        void* q_out, void* q_lo, uint32_t* range, hipStream_t st) {
  const int nb = res_blocks(s);
  // TV from dh / 8 rows (one unit per slice of the one chunk); beyond 32 rows, 8 units per
  // group and 8 groups per 64 workgroups
  const bool tv = s.dh % 32 == 0 && n_rows >= s.dh / 8;
  const int tv_groups = (n_rows + 63) / 64 * (s.dh / 32);
  dim3 grid(tv && n_rows > 32 ? std::max(n_rows, (tv_groups + 7) / 8 * 64) : n_rows,
            s.n_q + 2 * s.n_kv);
  // queries leave pre-scaled by log2(e) / sqrt(dh): the attention softmax works in base 2
  const float qscale = (float)(1.4426950408889634 / std::sqrt((double)s.dh));
#define SPP_QKV_EPI(T, TV)                                                                       \
  SPP_LAUNCH((qkv_epilogue_kernel<T, TV>), grid, dim3(64), 0, st, s, dp, n_rows, layer, partials, \
             splits, ss, nb, rope, qscale, static_cast<T*>(q_out), static_cast<T*>(q_lo), range)
  if (s.bf16) {
    if (tv) SPP_QKV_EPI(bf16_t, true); else SPP_QKV_EPI(bf16_t, false);
  } else {
    if (tv) SPP_QKV_EPI(float, true); else SPP_QKV_EPI(float, false);
  }
#undef SPP_QKV_EPI
  return hipGetLastError();
}

hipError_t residual(const Shape& s, int n_rows, const float* partials, int splits, float* x,
                    const void* g, void* y, void* y_lo, float* ss, hipStream_t st) {
  if (s.d % 4) return hipErrorInvalidValue;
  dim3 grid(n_rows, res_blocks(s));
  if (s.bf16)
    SPP_LAUNCH(residual_kernel<bf16_t>, grid, dim3(256), 0, st, s, n_rows, partials, splits,
                       x, static_cast<const bf16_t*>(g), static_cast<bf16_t*>(y),
                       static_cast<bf16_t*>(y_lo), ss);
  else
    SPP_LAUNCH(residual_kernel<float>, grid, dim3(256), 0, st, s, n_rows, partials, splits,
                       x, static_cast<const float*>(g), static_cast<float*>(y),
                       static_cast<float*>(y_lo), ss);
  return hipGetLastError();
}

hipError_t swiglu(const Shape& s, int n_rows, const float* partials, int splits, const float* ss,
                  void* act, void* act_lo, hipStream_t st) {
  if (splits < 1) return hipErrorInvalidValue;
  const int nb = res_blocks(s);
  const int64_t total = (int64_t)n_rows * s.ffn / 4;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
#define SPP_SWI(T, S)                                                                          \
  SPP_LAUNCH((swiglu_kernel<T, S>), dim3((unsigned)blocks), dim3(256), 0, st, s, n_rows,       \
             partials, splits, ss, nb, static_cast<T*>(act), static_cast<T*>(act_lo))
#define SPP_SWI_S(T)                            \
  switch (split_bucket(splits)) {               \
    case 4: SPP_SWI(T, 4); break;               \
    case 8: SPP_SWI(T, 8); break;               \
    case 16: SPP_SWI(T, 16); break;             \
    default: SPP_SWI(T, 0); break;              \
  }
  if (s.bf16) {
    SPP_SWI_S(bf16_t)
  } else {
    SPP_SWI_S(float)
  }
#undef SPP_SWI_S
#undef SPP_SWI
  return hipGetLastError();
}

hipError_t final_norm_rows(const Shape& s, const StepView& dp, int n_segs, const float* x,
                           const void* g_final, void* z, void* z_lo, hipStream_t st) {
  if (s.bf16)
    SPP_LAUNCH(final_norm_rows_kernel<bf16_t>, dim3(n_segs), dim3(256), 0, st, s, dp, x,
                       static_cast<const bf16_t*>(g_final), static_cast<bf16_t*>(z),
                       static_cast<bf16_t*>(z_lo));
  else
    SPP_LAUNCH(final_norm_rows_kernel<float>, dim3(n_segs), dim3(256), 0, st, s, dp, x,
                       static_cast<const float*>(g_final), static_cast<float*>(z),
                       static_cast<float*>(z_lo));
  return hipGetLastError();
}

hipError_t shift_cells(const Shape& s, void* kv, int64_t cap, int n_new, int delta,
                       hipStream_t st) {
  if (n_new <= 0) return hipSuccess;
  if (delta < 1 || s.dh > 128 || s.dh % 2) return hipErrorInvalidValue;
  dim3 grid(s.n_kv, s.n_layers, 2);
  if (s.bf16)
    SPP_LAUNCH(shift_kernel<bf16_t>, grid, dim3(256), 0, st, s, kv, cap, n_new, delta);
  else
    SPP_LAUNCH(shift_kernel<float>, grid, dim3(256), 0, st, s, kv, cap, n_new, delta);
  return hipGetLastError();
}

hipError_t copy_bytes(void* dst, const void* src, size_t n, hipStream_t st) {
  const size_t n16 = n / 16;
  if (n16) {
    size_t blocks = (n16 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    SPP_LAUNCH(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<uint4*>(dst), static_cast<const uint4*>(src), n16);
  }
  if (n % 16)
    SPP_LAUNCH(copy_tail_kernel, dim3(1), dim3(64), 0, st,
                       static_cast<char*>(dst) + n16 * 16, static_cast<const char*>(src) + n16 * 16,
                       n % 16);
  return hipGetLastError();
}

}  // namespace k
}  // namespace spp
