// Delta attention: the entry's queries against the session's resident KV cells plus
// the entry's own (just appended) cells, causal within the entry, grouped-query.
//
// The work is split over (segment, kv head, 64-row group, 512-key chunk) items so a
// long cache fills the chip; the G query heads of one kv head share every K/V tile,
// so each byte of the cache is read from HBM once per 64 query rows.  Per item:
//   * a 64-key tile of K ([key][dh], rows contiguous in the cache) and of V^T
//     ([dh][key], the cache keeps V transposed so this is contiguous too) is staged
//     in LDS, the next tile's loads already in flight in registers;
//   * S^T = K Q^T on the matrix cores: lane (query q, group g) then holds the scores
//     of keys 4g..4g+3 of every 16-key block for query q (bf16 models multiply the
//     (hi, lo) halves of q, and later of P, so neither loses precision to bf16);
//   * online softmax in base 2 (scale log2(e)/sqrt(dh) folded in), max and sum kept
//     per query, reduced over the 4 lanes of a query with two shuffles;
//   * O^T += V^T P^T on the matrix cores, which needs exactly the P values the lane
//     already holds, so P never leaves registers;
//   * the unnormalised O, the running max m and the sum l go to a partial buffer and
//     a combine kernel merges the chunks of each row in chunk order.
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

template <typename T, int DH>
struct AttnCfg {
  static constexpr int SZ = Elem<T>::kBytes;
  static constexpr int E = Elem<T>::kPerFrag;
  static constexpr int NF = DH * SZ / 64;            // 16-byte Q fragments per lane
  static constexpr int KPITCH = DH * SZ + 16;        // LDS bytes per key row of K
  static constexpr int VPITCH = kAttnTile * SZ + 16; // LDS bytes per dh row of V^T
  static constexpr int K_UNITS = kAttnTile * DH * SZ / 16;
  static constexpr int V_UNITS = DH * kAttnTile * SZ / 16;
  static constexpr int UNITS_PER_THREAD = (K_UNITS + V_UNITS) / 256;
  static constexpr int NO = DH / 16;                 // O^T accumulator blocks
};

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_kernel(Shape s, const StepParams* sp, int layer,
                                                   const T* __restrict__ Q, const T* __restrict__ Qlo,
                                                   float* __restrict__ Opart,
                                                   float2* __restrict__ MLpart) {
  using C = AttnCfg<T, DH>;
  __shared__ __attribute__((aligned(16))) char k_lds[kAttnTile * C::KPITCH];
  __shared__ __attribute__((aligned(16))) char v_lds[DH * C::VPITCH];

  const AttnItem it = sp_items(sp)[blockIdx.x];
  const Segment sg = sp->seg[it.seg];
  const int G = s.n_q / s.n_kv;
  const int R = sg.len * G;  // query rows of this kv head in the segment
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, ql = lane & 15;

  const int qr = it.rowgrp * kAttnRows + wave * 16 + ql;  // this lane's query row
  const bool row_ok = qr < R;
  const int j = row_ok ? qr / G : 0;
  const int head = it.kvh * G + (row_ok ? qr % G : 0);
  const int key_limit = row_ok ? sg.n_past + j + 1 : 0;  // causal: keys < limit visible

  const int last_row = min(it.rowgrp * kAttnRows + kAttnRows, R) - 1;
  const int wg_limit = sg.n_past + last_row / G + 1;
  const int kbeg = it.chunk * kAttnChunk;
  const int kend = min(kbeg + kAttnChunk, wg_limit);

  const int64_t cap = sg.cap;
  const T* kvb = static_cast<const T*>(sg.kv) + (int64_t)layer * 2 * s.n_kv * cap * DH;
  const char* kc = reinterpret_cast<const char*>(kvb + (int64_t)it.kvh * cap * DH);
  const char* vt = reinterpret_cast<const char*>(kvb + (int64_t)s.n_kv * cap * DH +
                                                 (int64_t)it.kvh * DH * cap);

  // Q^T fragments of this lane's query: dims [t*4E + g*E, +E).  bf16 models carry q as a
  // (hi, lo) pair and P as a (hi, lo) pair too, so that the scores and the weighted sum see
  // ~16 significant bits of the fp32 values (the matrix cores multiply both halves).
  constexpr int NP = C::SZ == 2 ? 2 : 1;
  uint4 qf[NP][C::NF];
  {
    const int64_t qoff = ((int64_t)(sg.row0 + j) * s.n_q + head) * DH;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const char* qrow = reinterpret_cast<const char*>((p == 0 ? Q : Qlo) + qoff);
#pragma unroll
      for (int t = 0; t < C::NF; ++t)
        qf[p][t] = row_ok ? *reinterpret_cast<const uint4*>(qrow + (t * 4 * C::E + g * C::E) * C::SZ)
                          : make_uint4(0, 0, 0, 0);
    }
  }

  f32x4 acc_o[C::NO];
#pragma unroll
  for (int u = 0; u < C::NO; ++u) acc_o[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float c2 = 1.4426950408889634f * rsqrtf((float)DH);

  // register staging of one tile: units [0, K_UNITS) are K, then V^T
  uint4 stage[C::UNITS_PER_THREAD];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < C::UNITS_PER_THREAD; ++i) {
      const int u = tid + i * 256;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (u < C::K_UNITS) {
        constexpr int UPR = DH * C::SZ / 16;
        const int key = u / UPR, c = u - key * UPR;
        if (kt + key < kend)
          v = *reinterpret_cast<const uint4*>(kc + ((int64_t)(kt + key) * DH) * C::SZ + c * 16);
      } else {
        constexpr int UPR = kAttnTile * C::SZ / 16;
        const int uu = u - C::K_UNITS;
        const int row = uu / UPR, c = uu - row * UPR;
        constexpr int KEYS_PER_UNIT = 16 / C::SZ;
        const int key0 = kt + c * KEYS_PER_UNIT;
        if (key0 < kend) {
          v = *reinterpret_cast<const uint4*>(vt + ((int64_t)row * cap + key0) * C::SZ);
          if (key0 + KEYS_PER_UNIT > kend) {  // zero the values of keys past the end
            uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < KEYS_PER_UNIT; ++e) {
              if (key0 + e >= kend) {
                if (C::SZ == 4) w[e] = 0;
                else w[e / 2] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
              }
            }
            v = make_uint4(w[0], w[1], w[2], w[3]);
          }
        }
      }
      stage[i] = v;
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < C::UNITS_PER_THREAD; ++i) {
      const int u = tid + i * 256;
      if (u < C::K_UNITS) {
        constexpr int UPR = DH * C::SZ / 16;
        const int key = u / UPR, c = u - key * UPR;
        *reinterpret_cast<uint4*>(k_lds + key * C::KPITCH + c * 16) = stage[i];
      } else {
        constexpr int UPR = kAttnTile * C::SZ / 16;
        const int uu = u - C::K_UNITS;
        const int row = uu / UPR, c = uu - row * UPR;
        *reinterpret_cast<uint4*>(v_lds + row * C::VPITCH + c * 16) = stage[i];
      }
    }
  };

  if (kbeg < kend) load_tile(kbeg);
  for (int kt = kbeg; kt < kend; kt += kAttnTile) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (kt + kAttnTile < kend) load_tile(kt + kAttnTile);

    // ---- scores S^T for the 4 key blocks of the tile
    f32x4 sc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
      const char* krow = k_lds + (kb * 16 + ql) * C::KPITCH + g * C::E * C::SZ;
#pragma unroll
      for (int t = 0; t < C::NF; ++t) {
        const uint4 kf = *reinterpret_cast<const uint4*>(krow + t * 4 * C::E * C::SZ);
#pragma unroll
        for (int p = 0; p < NP; ++p) a = mma_frag(kf, qf[p][t], a, T{});
      }
      sc[kb] = a;
    }
    // ---- mask, tile max
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kt + kb * 16 + 4 * g + e;
        const float v = (key < key_limit && key < kend) ? sc[kb][e] * c2 : -INFINITY;
        sc[kb][e] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = m_new == -INFINITY ? 1.f : exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = m_new == -INFINITY ? 0.f : exp2f(sc[kb][e] - m_new);
        sc[kb][e] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int u = 0; u < C::NO; ++u) acc_o[u] *= alpha;

    // ---- O^T += V^T P^T
    if constexpr (C::SZ == 2) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {  // 32 keys: blocks 2c and 2c+1
        uint16_t ph[8], pl[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = sc[2 * c + e / 4][e % 4];
          ph[e] = f32_to_bf16(pv);
          pl[e] = f32_to_bf16(pv - bf16_to_f32(ph[e]));
        }
        const uint4 pf_hi = make_uint4(ph[0] | ((uint32_t)ph[1] << 16), ph[2] | ((uint32_t)ph[3] << 16),
                                       ph[4] | ((uint32_t)ph[5] << 16), ph[6] | ((uint32_t)ph[7] << 16));
        const uint4 pf_lo = make_uint4(pl[0] | ((uint32_t)pl[1] << 16), pl[2] | ((uint32_t)pl[3] << 16),
                                       pl[4] | ((uint32_t)pl[5] << 16), pl[6] | ((uint32_t)pl[7] << 16));
#pragma unroll
        for (int u = 0; u < C::NO; ++u) {
          const char* vrow = v_lds + (u * 16 + ql) * C::VPITCH;
          const uint2 v0 = *reinterpret_cast<const uint2*>(vrow + ((2 * c) * 16 + 4 * g) * 2);
          const uint2 v1 = *reinterpret_cast<const uint2*>(vrow + ((2 * c + 1) * 16 + 4 * g) * 2);
          const uint4 vf = make_uint4(v0.x, v0.y, v1.x, v1.y);
          acc_o[u] = mma_frag(vf, pf_hi, acc_o[u], T{});
          acc_o[u] = mma_frag(vf, pf_lo, acc_o[u], T{});
        }
      }
    } else {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const uint4 pf = make_uint4(__float_as_uint(sc[kb][0]), __float_as_uint(sc[kb][1]),
                                    __float_as_uint(sc[kb][2]), __float_as_uint(sc[kb][3]));
#pragma unroll
        for (int u = 0; u < C::NO; ++u) {
          const char* vrow = v_lds + (u * 16 + ql) * C::VPITCH;
          acc_o[u] = mma_frag(*reinterpret_cast<const uint4*>(vrow + (kb * 16 + 4 * g) * 4), pf,
                              acc_o[u], T{});
        }
      }
    }
  }

  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const int64_t prow = (int64_t)blockIdx.x * kAttnRows + wave * 16 + ql;
#pragma unroll
  for (int u = 0; u < C::NO; ++u)
    *reinterpret_cast<f32x4*>(Opart + prow * DH + u * 16 + 4 * g) = acc_o[u];
  if (g == 0) MLpart[prow] = make_float2(m_run, l_run);
}

// One wave per query row of a (segment, kv head, row group): merge its chunks.  The
// chunk maxima and sums are read by different lanes at once; the O partials of four
// chunks are loaded before any is used, so the chain of dependent loads stays short.
template <typename T, int DH>
__global__ __launch_bounds__(256) void combine_kernel(Shape s, const StepParams* sp,
                                                      const float* __restrict__ Opart,
                                                      const float2* __restrict__ MLpart, T* out,
                                                      T* out_lo) {
  const AttnGroup gr = sp_groups(sp)[blockIdx.x];
  const Segment sg = sp->seg[gr.seg];
  const int G = s.n_q / s.n_kv;
  const int R = sg.len * G;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rl = blockIdx.y * 4 + wave;  // row within the group
  const int qr = gr.rowgrp * kAttnRows + rl;
  if (qr >= R) return;
  const int j = qr / G, head = gr.kvh * G + qr % G;
  const int n = gr.n_items;
  const int64_t base = (int64_t)gr.first_item * kAttnRows + rl;
  float mx = -INFINITY;
  for (int c = lane; c < n; c += 64) {
    const float2 ml = MLpart[base + (int64_t)c * kAttnRows];
    if (ml.y > 0.f) mx = fmaxf(mx, ml.x);
  }
  mx = wave_max(mx);
  float L = 0.f;
  for (int c = lane; c < n; c += 64) {
    const float2 ml = MLpart[base + (int64_t)c * kAttnRows];
    if (ml.y > 0.f) L += ml.y * exp2f(ml.x - mx);
  }
  L = wave_sum(L);
  constexpr int PER = DH / 64;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  int c = 0;
  for (; c + 4 <= n; c += 4) {
    float2 ml[4];
    float o[4][PER];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t prow = base + (int64_t)(c + u) * kAttnRows;
      ml[u] = MLpart[prow];
#pragma unroll
      for (int e = 0; e < PER; ++e) o[u][e] = Opart[prow * DH + lane + 64 * e];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float w = ml[u].y > 0.f ? exp2f(ml[u].x - mx) : 0.f;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] += w * o[u][e];
    }
  }
  for (; c < n; ++c) {
    const int64_t prow = base + (int64_t)c * kAttnRows;
    const float2 ml = MLpart[prow];
    const float w = ml.y > 0.f ? exp2f(ml.x - mx) : 0.f;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += w * Opart[prow * DH + lane + 64 * e];
  }
  const float inv = 1.f / L;
  const int64_t o = ((int64_t)(sg.row0 + j) * s.n_q + head) * DH;
#pragma unroll
  for (int e = 0; e < PER; ++e) store_act(out, out_lo, o + lane + 64 * e, acc[e] * inv);
}

template <typename T, int DH>
hipError_t launch_attn(const Shape& s, const StepParams* dp, int n_items, int layer, const void* q,
                       const void* q_lo, float* o_part, float2* ml_part, hipStream_t st) {
  hipLaunchKernelGGL((attn_kernel<T, DH>), dim3(n_items), dim3(256), 0, st, s, dp, layer,
                     static_cast<const T*>(q), static_cast<const T*>(q_lo), o_part, ml_part);
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t launch_combine(const Shape& s, const StepParams* dp, int n_groups, const float* o_part,
                          const float2* ml_part, void* out, void* out_lo, hipStream_t st) {
  hipLaunchKernelGGL((combine_kernel<T, DH>), dim3(n_groups, kAttnRows / 4), dim3(256), 0, st, s,
                     dp, o_part, ml_part, static_cast<T*>(out), static_cast<T*>(out_lo));
  return hipGetLastError();
}

}  // namespace

namespace k {

hipError_t attention(const Shape& s, const StepParams* dp, int n_items, int layer, const void* q,
                     const void* q_lo, float* o_part, float2* ml_part, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (s.bf16)
    return s.dh == 128
               ? launch_attn<bf16_t, 128>(s, dp, n_items, layer, q, q_lo, o_part, ml_part, st)
               : launch_attn<bf16_t, 64>(s, dp, n_items, layer, q, q_lo, o_part, ml_part, st);
  // fp32 models: head_dim 64 only (checked at model creation)
  return launch_attn<float, 64>(s, dp, n_items, layer, q, q_lo, o_part, ml_part, st);
}

hipError_t attention_combine(const Shape& s, const StepParams* dp, int n_groups,
                             const float* o_part, const float2* ml_part, void* out, void* out_lo,
                             hipStream_t st) {
  if (n_groups <= 0) return hipSuccess;
  if (s.bf16)
    return s.dh == 128
               ? launch_combine<bf16_t, 128>(s, dp, n_groups, o_part, ml_part, out, out_lo, st)
               : launch_combine<bf16_t, 64>(s, dp, n_groups, o_part, ml_part, out, out_lo, st);
  return launch_combine<float, 64>(s, dp, n_groups, o_part, ml_part, out, out_lo, st);
}

}  // namespace k
}  // namespace spp
