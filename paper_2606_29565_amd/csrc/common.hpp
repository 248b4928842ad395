// Device helpers shared by the gfx950 kernels: element types, bf16 rounding,
// 16-byte fragments and the matrix-core step over one fragment.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct bf16_t {  // storage tag for bf16 (16-bit patterns)
  uint16_t bits;
};

template <typename T>
struct Elem;
template <>
struct Elem<bf16_t> {
  static constexpr int kBytes = 2;
  static constexpr int kPerFrag = 8;  // elements in a 16-byte fragment
};
template <>
struct Elem<float> {
  static constexpr int kBytes = 4;
  static constexpr int kPerFrag = 4;
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load of data that is read once per pass (the LM head weights): non-temporal,
// so it does not displace reused lines from the caches.
__device__ __forceinline__ uint4 ld_stream(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(static_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// 16-byte load through a pointer known to address device global memory.  A pointer
// read from memory is generic to the compiler, which would otherwise use a flat load;
// pending flat loads make every later wait a wait for all of them.
__device__ __forceinline__ uint4 ld_global(const void* p) {
  typedef const __attribute__((address_space(1))) u32x4 g_u32x4;
  const u32x4 v = *(g_u32x4*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint32_t ld_global_u32(const void* p) {
  return *(const __attribute__((address_space(1))) uint32_t*)p;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16, round to nearest, ties to even (the gfx950 conversion instruction).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two fp32 values as a packed bf16 pair (first value in the low half), rounded to nearest
// even, and the pair of their rounding remainders, also as bf16: v = hi + lo to ~16 bits.
__device__ __forceinline__ void split_pair(float a, float b, uint32_t& hi, uint32_t& lo) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 h = {(__bf16)a, (__bf16)b};
  hi = __builtin_bit_cast(uint32_t, h);
  // the rounded values read back from the packed word (one shift, one mask)
  const bf16x2 l = {(__bf16)(a - __uint_as_float(hi << 16)),
                    (__bf16)(b - __uint_as_float(hi & 0xFFFF0000u))};
  lo = __builtin_bit_cast(uint32_t, l);
}

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<bf16_t>(const bf16_t* p, int64_t i) {
  return bf16_to_f32(p[i].bits);
}

template <typename T>
__device__ __forceinline__ void store_elem(T* p, int64_t i, float v);
template <>
__device__ __forceinline__ void store_elem<float>(float* p, int64_t i, float v) { p[i] = v; }
template <>
__device__ __forceinline__ void store_elem<bf16_t>(bf16_t* p, int64_t i, float v) {
  p[i].bits = f32_to_bf16(v);
}

// Activation feeding a matrix-core product.  bf16 models store it as a pair of bf16
// arrays, hi = bf16(v) and lo = bf16(v - hi), and multiply both halves against the
// weights, so the product sees ~16 significant bits of the fp32 activation; fp32 models
// store v itself (lo unused).
template <typename T>
__device__ __forceinline__ void store_act(T* hi, T* lo, int64_t i, float v);
template <>
__device__ __forceinline__ void store_act<float>(float* hi, float*, int64_t i, float v) { hi[i] = v; }
template <>
__device__ __forceinline__ void store_act<bf16_t>(bf16_t* hi, bf16_t* lo, int64_t i, float v) {
  const uint16_t h = f32_to_bf16(v);
  hi[i].bits = h;
  lo[i].bits = f32_to_bf16(v - bf16_to_f32(h));
}

// Four consecutive activations [i, i+4), i a multiple of 4.
template <typename T>
__device__ __forceinline__ void store_act4(T* hi, T* lo, int64_t i, float4 v);
template <>
__device__ __forceinline__ void store_act4<float>(float* hi, float*, int64_t i, float4 v) {
  *reinterpret_cast<float4*>(hi + i) = v;
}
template <>
__device__ __forceinline__ void store_act4<bf16_t>(bf16_t* hi, bf16_t* lo, int64_t i, float4 v) {
  uint2 h, l;
  split_pair(v.x, v.y, h.x, l.x);
  split_pair(v.z, v.w, h.y, l.y);
  *reinterpret_cast<uint2*>(hi + i) = h;
  *reinterpret_cast<uint2*>(lo + i) = l;
}

// Unpack a 16-byte fragment into floats (8 for bf16, 4 for fp32).
__device__ __forceinline__ void frag_to_f32(const uint4& f, float (&out)[8]) {
  const uint32_t w[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void frag_to_f32(const uint4& f, float (&out)[4]) {
  out[0] = __uint_as_float(f.x);
  out[1] = __uint_as_float(f.y);
  out[2] = __uint_as_float(f.z);
  out[3] = __uint_as_float(f.w);
}

// One matrix-core step over a 16-byte fragment per lane, 16x16 output tile.
// Lane l holds row (l & 15) of A and column (l & 15) of B; group g = l >> 4 holds
// the fragment's elements for reduction indices {g*E .. g*E+E-1} of the step, where
// E = 8 (bf16: one 16x16x32 instruction) or 4 (fp32: four 16x16x4 instructions, the
// j-th of which takes element j of every group).  Any consistent assignment of the
// reduction index to (group, element) gives the same contraction, so A and B only
// need to use the same one.  D: lane l holds rows 4g..4g+3 of column (l & 15).
__device__ __forceinline__ f32x4 mma_frag(const uint4& a, const uint4& b, f32x4 c, bf16_t) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_frag(const uint4& a, const uint4& b, f32x4 c, float) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

// 1 / RMS of row r from its per-block sums of squares.
__device__ __forceinline__ float row_inv(const float* ss, int r, int nb, int d, float eps) {
  float t = 0.f;
  for (int b = 0; b < nb; ++b) t += ss[(int64_t)r * nb + b];
  return rsqrtf(t / d + eps);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// (value, index) pair order used by every top-2: larger value first, then lower index;
// NaN is never a candidate (callers skip it and raise the nonfinite flag instead).
struct Top2 {
  float v1, v2;
  int i1, i2;
};
__device__ __forceinline__ bool before(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}
__device__ __forceinline__ void top2_init(Top2& t) {
  t.v1 = t.v2 = -INFINITY;
  t.i1 = t.i2 = 0x7FFFFFFF;
}
__device__ __forceinline__ void top2_push(Top2& t, float v, int i) {
  if (before(v, i, t.v1, t.i1)) {
    t.v2 = t.v1;
    t.i2 = t.i1;
    t.v1 = v;
    t.i1 = i;
  } else if (before(v, i, t.v2, t.i2)) {
    t.v2 = v;
    t.i2 = i;
  }
}
__device__ __forceinline__ void top2_merge(Top2& t, const Top2& o) {
  top2_push(t, o.v1, o.i1);
  top2_push(t, o.v2, o.i2);
}
__device__ __forceinline__ Top2 wave_top2(Top2 t) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    Top2 u;
    u.v1 = __shfl_xor(t.v1, o, 64);
    u.i1 = __shfl_xor(t.i1, o, 64);
    u.v2 = __shfl_xor(t.v2, o, 64);
    u.i2 = __shfl_xor(t.i2, o, 64);
    top2_merge(t, u);
  }
  return t;
}

// x + P[0][off] + P[1][off] + ... + P[splits-1][off] (float4 at element offset `off`,
// consecutive splits `stride` elements apart), added in split order; the loads of up
// to sixteen splits are in flight together.
__device__ __forceinline__ float4 add_splits4(float4 x, const float* P, int64_t stride, int splits,
                                              int64_t off) {
  for (int k0 = 0; k0 < splits; k0 += 16) {
    float4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (k0 + u < splits) v[u] = *reinterpret_cast<const float4*>(P + (int64_t)(k0 + u) * stride + off);
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (k0 + u < splits) {
        x.x += v[u].x;
        x.y += v[u].y;
        x.z += v[u].z;
        x.w += v[u].w;
      }
  }
  return x;
}

// Scalar form: x + sum over splits of P[split * stride + off], in split order.
__device__ __forceinline__ float add_splits(float x, const float* P, int64_t stride, int splits,
                                            int64_t off) {
  for (int k0 = 0; k0 < splits; k0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (k0 + u < splits) v[u] = P[(int64_t)(k0 + u) * stride + off];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (k0 + u < splits) x += v[u];
  }
  return x;
}

// Straight-line form for at most S splits (S = 4, 8 or 16; the host picks the bucket with
// split_bucket): every split's load is issued, unconditionally (indices past `splits` read
// the last split again and are not added), before the first add, and the code has no
// loop or branch, so the loads of a kernel's other operands can go out with them and one
// wait covers all.  The sums are added in split order, as above.  S = 0 is the loop.
template <int S>
__device__ __forceinline__ float4 add_splits4_n(float4 x, const float* P, int64_t stride, int splits,
                                                int64_t off) {
  if constexpr (S == 0) {
    return add_splits4(x, P, stride, splits, off);
  } else {
    float4 v[S];
#pragma unroll
    for (int u = 0; u < S; ++u)
      v[u] = *reinterpret_cast<const float4*>(P + (int64_t)(u < splits ? u : splits - 1) * stride + off);
#pragma unroll
    for (int u = 0; u < S; ++u)
      if (u < splits) {
        x.x += v[u].x;
        x.y += v[u].y;
        x.z += v[u].z;
        x.w += v[u].w;
      }
    return x;
  }
}
// The bucket S of add_splits4_n for a split count: 4, 8 or 16, or 0 (the loop) beyond.
inline int split_bucket(int splits) {
  return splits <= 4 ? 4 : (splits <= 8 ? 8 : (splits <= 16 ? 16 : 0));
}

}  // namespace spp
