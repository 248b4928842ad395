// Delta attention: the entry's queries against the session's resident KV cells plus
// the entry's own (just appended) cells, causal within the entry, grouped-query.
//
// A work item is (segment, kv head, group of 128 query rows, key range).  The 128 rows
// are the (token, query head) pairs of the kv head, so the G query heads that share a
// kv head read each K/V byte once.  The host sizes the key ranges so that the items
// fill the chip once.  bf16 models run attn_kernel_h (fp16 matrix cores, described
// there); fp32 models run attn_kernel, 8 waves of 16 query rows each per item:
//   * 128-key tiles of K ([key][dh], contiguous in the cache) and of V^T ([dh][key],
//     the cache keeps V transposed so this is contiguous too) are double-buffered in
//     LDS; the next tile is in flight in registers while the matrix cores work on the
//     current one, and is stored to LDS only after that work, so a whole tile's compute
//     hides its memory latency;
//   * S^T = K Q^T on the matrix cores: lane (query q, group g) then holds the scores
//     of keys 4g..4g+3 of every 16-key block for query q.  The queries arrive scaled
//     by log2(e)/sqrt(dh), so the scores are already base-2 softmax exponents;
//   * online softmax: max and sum per query, reduced over the 4 lanes of a query with
//     two shuffles; the running output is rescaled only when some row's max grew;
//     tiles that no row of the wave needs to mask skip the mask;
//   * O^T += V^T P^T on the matrix cores, which needs exactly the P values the lane
//     already holds, so P never leaves registers;
//   * the unnormalised O, the running max m and the sum l go to a partial buffer, and a
//     combine kernel merges the key ranges of each row in order.
#include "common.hpp"
#include "kernels.hpp"

namespace spp {
namespace {

template <typename T, int DH>
struct AttnCfg {
  static constexpr int SZ = Elem<T>::kBytes;
  static constexpr int E = Elem<T>::kPerFrag;
  static constexpr int NP = SZ == 2 ? 2 : 1;          // query / P parts (hi, lo)
  static constexpr int NF = DH * SZ / 64;             // 16-byte Q fragments per lane
  static constexpr int KPITCH = DH * SZ + 16;         // LDS bytes per key row of K
  // LDS bytes per dh row of V^T: bf16 rows are padded by 8 bytes so that the 8-byte
  // fragment reads of 16 lanes (rows 66 dwords apart) hit 32 distinct banks
  static constexpr int VPITCH = kAttnTile * SZ + (SZ == 2 ? 8 : 16);
  static constexpr int NSUB = kAttnTile / kAttnSub;   // matrix-core passes per tile
  static constexpr int KBYTES = kAttnTile * KPITCH;
  static constexpr int BUF = KBYTES + DH * VPITCH;    // one LDS stage (K then V^T)
  static constexpr int THREADS = 64 * kAttnWaves;
  static constexpr int K_UNITS = kAttnTile * DH * SZ / 16;
  static constexpr int V_UNITS = DH * kAttnTile * SZ / 16;
  static constexpr int KPT = K_UNITS / THREADS;       // K units per thread per tile
  static constexpr int UPT = (K_UNITS + V_UNITS) / THREADS;
  static constexpr int UPR_K = DH * SZ / 16;          // units per key row of K
  static constexpr int UPR_V = kAttnTile * SZ / 16;   // units per dh row of V^T
  static constexpr int KEYS_PER_UNIT = 16 / SZ;
  static constexpr int NO = DH / 16;                  // O^T accumulator blocks
  static_assert(K_UNITS % THREADS == 0 && V_UNITS % THREADS == 0, "tile split");
};

template <typename T, int DH>
__global__ __launch_bounds__(64 * kAttnWaves, 2) void attn_kernel(
    Shape s, StepView sv, int layer, const T* __restrict__ Q, const T* __restrict__ Qlo,
    float* __restrict__ Opart, float2* __restrict__ MLpart) {
  using C = AttnCfg<T, DH>;
  __shared__ __attribute__((aligned(16))) char lds[2][C::BUF];

  const AttnItem it = sv.item[blockIdx.x];
  const Segment sg = it.sg;
  const int G = s.n_q / s.n_kv;
  const int R = sg.len * G;  // query rows of this kv head in the segment
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, ql = lane & 15;

  const int wrow0 = it.rowgrp * kAttnRows + wave * 16;  // first row of this wave
  const bool wave_live = wrow0 < R;
  const int qr = wrow0 + ql;  // this lane's query row
  const bool row_ok = qr < R;
  const int j = row_ok ? qr / G : 0;
  const int head = it.kvh * G + (row_ok ? qr % G : 0);
  const int key_limit = row_ok ? sg.n_past + j + 1 : 0;  // causal: keys < limit visible
  // every row of the wave sees keys below this bound (rows are ordered by token)
  const int wave_limit = sg.n_past + wrow0 / G + 1;

  const int kbeg = it.k0, kend = it.k1;
  const int n_tiles = kend > kbeg ? (kend - kbeg + kAttnTile - 1) / kAttnTile : 0;

  const int64_t cap = sg.cap;
  const T* kvb = static_cast<const T*>(sg.kv) + (int64_t)layer * 2 * s.n_kv * cap * DH;
  const char* kc = reinterpret_cast<const char*>(kvb + (int64_t)it.kvh * cap * DH);
  const char* vt = reinterpret_cast<const char*>(kvb + (int64_t)s.n_kv * cap * DH +
                                                 (int64_t)it.kvh * DH * cap);

  // Q^T fragments of this lane's query: dims [t*4E + g*E, +E), both halves.
  uint4 qf[C::NP][C::NF];
  {
    const int64_t qoff = ((int64_t)(sg.row0 + j) * s.n_q + head) * DH;
#pragma unroll
    for (int p = 0; p < C::NP; ++p) {
      const char* qrow = reinterpret_cast<const char*>((p == 0 ? Q : Qlo) + qoff);
#pragma unroll
      for (int t = 0; t < C::NF; ++t)
        qf[p][t] = row_ok ? ld_global(qrow + (t * 4 * C::E + g * C::E) * C::SZ)
                          : make_uint4(0, 0, 0, 0);
    }
  }

  f32x4 acc_o[C::NO];
#pragma unroll
  for (int u = 0; u < C::NO; ++u) acc_o[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // ---- tile staging: units [0, K_UNITS) are K rows, the rest V^T rows.  A unit past
  // the range reads the range's first cell instead (the store discards it), so every
  // thread issues the same loads whatever the range.  A staged tile is an SSA vector
  // value, never an addressable array, so it stays in registers.
  typedef uint32_t Stage __attribute__((ext_vector_type(4 * C::UPT)));
  auto load_tile = [&](int kt) -> Stage {
    Stage st;
#pragma unroll
    for (int i = 0; i < C::UPT; ++i) {
      const int u = tid + i * C::THREADS;
      uint4 v;
      if (i < C::KPT) {
        const int key = u / C::UPR_K, c = u - key * C::UPR_K;
        const int cell = kt + key < kend ? kt + key : kbeg;
        v = ld_global(kc + ((int64_t)cell * DH) * C::SZ + c * 16);
      } else {
        const int uu = u - C::K_UNITS;
        const int row = uu / C::UPR_V, c = uu - row * C::UPR_V;
        const int key0 = kt + c * C::KEYS_PER_UNIT;
        // in bounds: key0 is a multiple of 8 below kend, so the 8 cells end within
        // round_up(kend, 64) <= cap
        const int cell = key0 < kend ? key0 : kbeg;
        v = ld_global(vt + ((int64_t)row * cap + cell) * C::SZ);
      }
      st[4 * i] = v.x;
      st[4 * i + 1] = v.y;
      st[4 * i + 2] = v.z;
      st[4 * i + 3] = v.w;
    }
    return st;
  };
  // K rows past the range are left as loaded (their scores are masked); V^T values of
  // cells past the range are zeroed, since a zero weight times a stale value must stay 0.
  auto store_tile = [&](char* buf, Stage st, int kt) {
#pragma unroll
    for (int i = 0; i < C::UPT; ++i) {
      const int u = tid + i * C::THREADS;
      uint4 v = make_uint4(st[4 * i], st[4 * i + 1], st[4 * i + 2], st[4 * i + 3]);
      if (i < C::KPT) {
        const int key = u / C::UPR_K, c = u - key * C::UPR_K;
        *reinterpret_cast<uint4*>(buf + key * C::KPITCH + c * 16) = v;
      } else {
        const int uu = u - C::K_UNITS;
        const int row = uu / C::UPR_V, c = uu - row * C::UPR_V;
        const int nv = kend - (kt + c * C::KEYS_PER_UNIT);  // cells of the unit in range
        if constexpr (C::SZ == 2) {
          v.x &= (nv > 0 ? 0x0000FFFFu : 0u) | (nv > 1 ? 0xFFFF0000u : 0u);
          v.y &= (nv > 2 ? 0x0000FFFFu : 0u) | (nv > 3 ? 0xFFFF0000u : 0u);
          v.z &= (nv > 4 ? 0x0000FFFFu : 0u) | (nv > 5 ? 0xFFFF0000u : 0u);
          v.w &= (nv > 6 ? 0x0000FFFFu : 0u) | (nv > 7 ? 0xFFFF0000u : 0u);
        } else {
          v.x = nv > 0 ? v.x : 0u;
          v.y = nv > 1 ? v.y : 0u;
          v.z = nv > 2 ? v.z : 0u;
          v.w = nv > 3 ? v.w : 0u;
        }
        char* dv = buf + C::KBYTES + row * C::VPITCH + c * 16;  // 8-byte aligned
        reinterpret_cast<uint2*>(dv)[0] = make_uint2(v.x, v.y);
        reinterpret_cast<uint2*>(dv)[1] = make_uint2(v.z, v.w);
      }
    }
  };

  // ---- one tile against the wave's 16 query rows.  All fragments of a phase are read
  // from LDS before the first matrix-core step uses one, so the wave waits for LDS once
  // per phase; the V^T fragments are requested before the softmax arithmetic.
  auto compute_sub = [&](const char* kl, const char* vl, int kt) {
    uint4 kf[4][C::NF];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int t = 0; t < C::NF; ++t)
        kf[kb][t] = *reinterpret_cast<const uint4*>(kl + (kb * 16 + ql) * C::KPITCH +
                                                    (t * 4 * C::E + g * C::E) * C::SZ);
    f32x4 sc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) sc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < C::NF; ++t)
#pragma unroll
      for (int p = 0; p < C::NP; ++p)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) sc[kb] = mma_frag(kf[kb][t], qf[p][t], sc[kb], T{});

    // V^T fragments for O^T += V^T P^T: bf16 takes 32 keys per step (key blocks 2c and
    // 2c+1, 4 keys of each per lane group), fp32 16 keys (block kb)
    constexpr int VS = C::SZ == 2 ? 2 : 4;
    uint4 vf[VS][C::NO];
#pragma unroll
    for (int c = 0; c < VS; ++c)
#pragma unroll
      for (int u = 0; u < C::NO; ++u) {
        const char* vrow = vl + (u * 16 + ql) * C::VPITCH;
        if constexpr (C::SZ == 2) {
          const uint2 v0 = *reinterpret_cast<const uint2*>(vrow + ((2 * c) * 16 + 4 * g) * 2);
          const uint2 v1 = *reinterpret_cast<const uint2*>(vrow + ((2 * c + 1) * 16 + 4 * g) * 2);
          vf[c][u] = make_uint4(v0.x, v0.y, v1.x, v1.y);
        } else {
          vf[c][u] = *reinterpret_cast<const uint4*>(vrow + (c * 16 + 4 * g) * 4);
        }
      }

    const bool full = kt + kAttnSub <= kend && kt + kAttnSub <= wave_limit;
    if (!full) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = kt + kb * 16 + 4 * g + e;
          if (!(key < key_limit && key < kend)) sc[kb][e] = -INFINITY;
        }
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) mt = fmaxf(mt, sc[kb][e]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    if (mt > m_run) {  // this row's max grew: rescale its sum and output
      const float alpha = __builtin_amdgcn_exp2f(m_run - mt);  // m_run = -inf gives 0
      l_run *= alpha;
#pragma unroll
      for (int u = 0; u < C::NO; ++u) acc_o[u] *= alpha;
      m_run = mt;
    }
    // exponent base; a row with nothing visible yet keeps every p at 0
    const float mref = m_run == -INFINITY ? 0.f : m_run;
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = __builtin_amdgcn_exp2f(sc[kb][e] - mref);
        sc[kb][e] = p;
        psum += p;
      }
    l_run += psum;

    if constexpr (C::SZ == 2) {
      uint4 pf[2][2];  // [step c][hi, lo]
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        uint32_t ph[4], pl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          split_pair(sc[2 * c + e / 2][2 * (e % 2)], sc[2 * c + e / 2][2 * (e % 2) + 1], ph[e], pl[e]);
        pf[c][0] = make_uint4(ph[0], ph[1], ph[2], ph[3]);
        pf[c][1] = make_uint4(pl[0], pl[1], pl[2], pl[3]);
      }
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int u = 0; u < C::NO; ++u) acc_o[u] = mma_frag(vf[c][u], pf[c][p], acc_o[u], T{});
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint4 pf = make_uint4(__float_as_uint(sc[c][0]), __float_as_uint(sc[c][1]),
                                    __float_as_uint(sc[c][2]), __float_as_uint(sc[c][3]));
#pragma unroll
        for (int u = 0; u < C::NO; ++u) acc_o[u] = mma_frag(vf[c][u], pf, acc_o[u], T{});
      }
    }
  };

  auto compute = [&](const char* buf, int kt) {
    if (!wave_live) return;
#pragma unroll
    for (int sub = 0; sub < C::NSUB; ++sub)
      if (kt + sub * kAttnSub < kend)
        compute_sub(buf + sub * kAttnSub * C::KPITCH, buf + C::KBYTES + sub * kAttnSub * C::SZ,
                    kt + sub * kAttnSub);
  };

  // ---- pipeline: tile i computes from lds[i & 1] while tile i+1 is in flight; tile i+1
  // goes to LDS after that compute.  One register set, one code path per tile.
  Stage st = load_tile(kbeg);
  store_tile(lds[0], st, kbeg);
  st = load_tile(kbeg + kAttnTile);
  __syncthreads();
  for (int i = 0; i < n_tiles; ++i) {
    const int kt = kbeg + i * kAttnTile;
    compute(lds[i & 1], kt);
    // (unconditional: past the last tile it fills a buffer nobody reads)
    store_tile(lds[(i + 1) & 1], st, kt + kAttnTile);
    st = load_tile(kt + 2 * kAttnTile);
    __syncthreads();  // lds[(i+1) & 1] holds tile i+1; lds[i & 1] is free
  }

  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const int64_t prow = (int64_t)blockIdx.x * kAttnRows + wave * 16 + ql;
#pragma unroll
  for (int u = 0; u < C::NO; ++u)
    *reinterpret_cast<f32x4*>(Opart + prow * DH + u * 16 + 4 * g) = acc_o[u];
  if (g == 0) MLpart[prow] = make_float2(m_run, l_run);
}

// bf16 models: the work item covers up to 256 query rows -- every row of a (segment, kv
// head) up to 64 entry tokens of a 4-query-head group or 32 of an 8-head one -- so each
// K/V byte is read once for all of them, and it is computed on the matrix cores in fp16.
// Every bf16 cell with magnitude in [2^-14, 65504] is exactly representable in fp16 (8
// significant bits of 11), so K and V lose nothing when each staged tile is converted in
// LDS; the query (written in fp16 by the QKV epilogue) and the softmax weights P enter
// with 11 significant bits, where a plain bf16 operand would keep 8.  Work split:
//   * 32x32x16 matrix-core steps: a wave owns a query block of 32 rows, so each K or V^T
//     fragment read from LDS feeds 32 queries;
//   * the 8 waves are QBP query-block slots x KP key parts (QBP the item's query blocks
//     rounded up to a power of two, KP = min(8 / QBP, 4)): wave (qb, kp) takes the 32-key
//     blocks kp, kp + KP, ... of every 128-key tile for rows [32 qb, 32 qb + 32); the key
//     parts of a query block merge in LDS at the end;
//   * S^T = K Q^T: lane l holds the scores of query l % 32 for keys
//     8 (i / 4) + 4 (l / 32) + i % 4, i < 16, of a 32-key block; O^T += V^T P^T takes those
//     same keys 16 at a time, so V^T rows keep each 16-key group in the order (0-3, 8-11,
//     4-7, 12-15) and a lane's 8 keys are one 16-byte LDS read;
//   * the softmax reference m of a row is raised only when some score of the wave
//     exceeds it by more than 8 (base 2): the common block needs no cross-lane reduction
//     and no rescale, P stays <= 2^8, and the scores arrive from the matrix cores already
//     offset by -m (the accumulator starts at -m);
//   * each lane sums its own P; the two lanes of a query are reduced once at the end;
//   * an item alone in its row group writes the attention output (hi, lo) itself; the
//     others leave the output normalized by its own sum in fp16 (11 significant bits,
//     half the bytes of fp32) with the (max, sum) pair in fp32, for the merge kernel.
template <int DH>
struct AttnHCfg {
  static constexpr int NT = DH / 16;                  // 16-dim steps (Q^T fragments per lane)
  static constexpr int ND = DH / 32;                  // 32-dim output blocks
  // LDS bytes per V^T row and per K row: odd multiples of 16 bytes.  A fragment read
  // takes 16 consecutive rows at one column per 16 lanes, and at this pitch they fall on
  // 16 distinct groups of 4 of the 64 banks (at an odd multiple of 32 bytes, rows r and
  // r + 8 share banks: the bank-conflict counter read 4-7x higher)
  static constexpr int PITCH = kAttnTile * 2 + 16;
  static constexpr int KPITCH = DH * 2 + 16;
  static constexpr int KBYTES = kAttnTile * KPITCH;
  static constexpr int QPITCH = DH * 2 + 16;          // LDS bytes per staged query row
  // one LDS stage: K then V^T, and at least the item's staged queries
  static constexpr int BUF = KBYTES + DH * PITCH > kAttnRowsH * QPITCH ? KBYTES + DH * PITCH
                                                                       : kAttnRowsH * QPITCH;
  static constexpr int THREADS = 64 * kAttnWaves;
  static constexpr int K_UNITS = kAttnTile * DH * 2 / 16;
  static constexpr int V_UNITS = DH * kAttnTile * 2 / 16;
  static constexpr int KPT = K_UNITS / THREADS;
  static constexpr int UPT = (K_UNITS + V_UNITS) / THREADS;
  static constexpr int UPR_K = DH * 2 / 16;
  static constexpr int UPR_V = kAttnTile * 2 / 16;
  static constexpr int QBLOCKS = kAttnRowsH / 32;     // query blocks of an item
  static constexpr int SLOT = (ND * 16 + 2) * 64;     // floats of one wave's merge state
  static_assert(K_UNITS % THREADS == 0 && V_UNITS % THREADS == 0, "tile split");
  static_assert(kAttnWaves == 8 && kAttnTile == 128 && QBLOCKS == 8, "work split");
  // the end-of-item merge (one slot per wave) fits in the tile buffers
  static_assert(kAttnWaves * SLOT * 4 <= 2 * BUF, "merge buffer");
  static_assert(QBLOCKS * 32 * QPITCH <= BUF, "q staging");
};

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  const f16x2 h = {(_Float16)a, (_Float16)b};  // round to nearest even
  return __builtin_bit_cast(uint32_t, h);
}
// eight bf16 (one 16-byte unit) as eight fp16; `mx` keeps the largest magnitude seen
// (an input above 65504 has no finite fp16 value)
__device__ __forceinline__ uint4 bf16x8_to_f16(const uint4 v, float& mx) {
  float f[8];
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) mx = fmaxf(mx, fabsf(f[i]));
  return make_uint4(pack_f16(f[0], f[1]), pack_f16(f[2], f[3]), pack_f16(f[4], f[5]),
                    pack_f16(f[6], f[7]));
}
__device__ __forceinline__ f32x16 mma32_f16(const uint4& a, const uint4& b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

template <int DH>
__global__ __launch_bounds__(64 * kAttnWaves, 1) void attn_kernel_h(
    Shape s, StepView sv, int layer, const uint16_t* __restrict__ Q,
    uint16_t* __restrict__ Opart, float2* __restrict__ MLpart, bf16_t* out, bf16_t* out_lo,
    uint32_t* range) {
  using C = AttnHCfg<DH>;
  __shared__ __attribute__((aligned(16))) char lds[2][C::BUF];

  const AttnItem it = sv.item[blockIdx.x];
  const Segment sg = it.sg;
  const int G = s.n_q / s.n_kv;
  const int R = sg.len * G;  // query rows of this kv head in the segment
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, ql = lane & 31;

  // the item's query blocks, and this wave's (query block, key part)
  const int row0 = it.rowgrp * kAttnRowsH;
  const int QB = (min(kAttnRowsH, R - row0) + 31) / 32;
  const int QBP = QB > 4 ? 8 : (QB > 2 ? 4 : (QB > 1 ? 2 : 1));
  const int KP = min(8 / QBP, 4);
  const int qb = wave % QBP, kp = wave / QBP;
  const bool wave_live = kp < KP && qb < QB;

  const int wrow0 = row0 + qb * 32;  // first row of this wave
  const int qr = wrow0 + ql;         // this lane's query row
  const bool row_ok = wave_live && qr < R;
  const int j = row_ok ? qr / G : 0;
  const int head = it.kvh * G + (row_ok ? qr % G : 0);
  const int key_limit = row_ok ? sg.n_past + j + 1 : 0;  // causal: keys < limit visible
  // every row of the wave sees keys below this bound (rows are ordered by token)
  const int wave_limit = sg.n_past + wrow0 / G + 1;

  const int kbeg = it.k0, kend = it.k1;
  const int n_tiles = kend > kbeg ? (kend - kbeg + kAttnTile - 1) / kAttnTile : 0;

  const int64_t cap = sg.cap;
  const bf16_t* kvb = static_cast<const bf16_t*>(sg.kv) + (int64_t)layer * 2 * s.n_kv * cap * DH;
  const char* kc = reinterpret_cast<const char*>(kvb + (int64_t)it.kvh * cap * DH);
  const char* vt = reinterpret_cast<const char*>(kvb + (int64_t)s.n_kv * cap * DH +
                                                 (int64_t)it.kvh * DH * cap);

  f32x16 acc_o[C::ND];
#pragma unroll
  for (int u = 0; u < C::ND; ++u)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc_o[u][i] = 0.f;
  float m_ref = -INFINITY;  // softmax reference of this lane's row (base 2)
  float l_run = 0.f;        // this lane's share of the row's sum of P
  float cell_max = 0.f;     // largest |K|, |V| this thread staged (fp16 range check)

  // ---- tile staging, in two halves: the K half (units [0, K_UNITS), K rows) and the V
  // half (the V^T rows), bf16 as in the cache.  A unit past the range reads the range's
  // first cell instead (the store discards it), so every thread issues the same loads
  // whatever the range.
  // (byte offsets within one kv head's K or V^T fit 32 bits: cap <= 2^24 cells, checked
  // at session creation)
  typedef uint32_t Half __attribute__((ext_vector_type(4 * C::KPT)));
  static_assert(C::UPT == 2 * C::KPT, "equal halves");
  auto load_k = [&](int kt) -> Half {
    Half st;
#pragma unroll
    for (int i = 0; i < C::KPT; ++i) {
      const int u = tid + i * C::THREADS;
      const int key = u / C::UPR_K, c = u - key * C::UPR_K;
      const int cell = kt + key < kend ? kt + key : kbeg;
      const uint4 v = ld_global(kc + ((uint32_t)cell * DH * 2u + c * 16));
      st[4 * i] = v.x;
      st[4 * i + 1] = v.y;
      st[4 * i + 2] = v.z;
      st[4 * i + 3] = v.w;
    }
    return st;
  };
  auto load_v = [&](int kt) -> Half {
    Half st;
#pragma unroll
    for (int i = 0; i < C::KPT; ++i) {
      const int uu = tid + i * C::THREADS;
      const int row = uu / C::UPR_V, c = uu - row * C::UPR_V;
      const int key0 = kt + c * 8;
      // in bounds: key0 is a multiple of 8 below kend, so the 8 cells end within
      // round_up(kend, 64) <= cap
      const int cell = key0 < kend ? key0 : kbeg;
      const uint4 v = ld_global(vt + ((uint32_t)row * (uint32_t)cap + cell) * 2u);
      st[4 * i] = v.x;
      st[4 * i + 1] = v.y;
      st[4 * i + 2] = v.z;
      st[4 * i + 3] = v.w;
    }
    return st;
  };
  // To LDS as fp16.  K rows past the range are kept (their scores are masked); V^T cells
  // past the range are zeroed, since a zero weight times a stale value must stay 0.  A
  // V^T unit holds keys 8a..8a+7 of a 16-key group (a = c % 2): its first four keys go
  // to group positions 4a..4a+3, its last four to 8+4a..8+4a+3.
  auto store_k = [&](char* buf, Half st) {
#pragma unroll
    for (int i = 0; i < C::KPT; ++i) {
      const int u = tid + i * C::THREADS;
      const uint4 v = make_uint4(st[4 * i], st[4 * i + 1], st[4 * i + 2], st[4 * i + 3]);
      const int key = u / C::UPR_K, c = u - key * C::UPR_K;
      *reinterpret_cast<uint4*>(buf + key * C::KPITCH + c * 16) = bf16x8_to_f16(v, cell_max);
    }
  };
  auto store_v = [&](char* buf, Half st, int kt) {
#pragma unroll
    for (int i = 0; i < C::KPT; ++i) {
      const int uu = tid + i * C::THREADS;
      uint4 v = make_uint4(st[4 * i], st[4 * i + 1], st[4 * i + 2], st[4 * i + 3]);
      const int row = uu / C::UPR_V, c = uu - row * C::UPR_V;
      const int nv = kend - (kt + c * 8);  // cells of the unit in range
      v.x &= (nv > 0 ? 0x0000FFFFu : 0u) | (nv > 1 ? 0xFFFF0000u : 0u);
      v.y &= (nv > 2 ? 0x0000FFFFu : 0u) | (nv > 3 ? 0xFFFF0000u : 0u);
      v.z &= (nv > 4 ? 0x0000FFFFu : 0u) | (nv > 5 ? 0xFFFF0000u : 0u);
      v.w &= (nv > 6 ? 0x0000FFFFu : 0u) | (nv > 7 ? 0xFFFF0000u : 0u);
      const uint4 hv = bf16x8_to_f16(v, cell_max);
      char* dv = buf + C::KBYTES + row * C::PITCH + (c >> 1) * 32 + (c & 1) * 8;
      reinterpret_cast<uint2*>(dv)[0] = make_uint2(hv.x, hv.y);
      reinterpret_cast<uint2*>(dv + 16)[0] = make_uint2(hv.z, hv.w);
    }
  };

  uint4 qf[C::NT];  // Q^T fragment t of this lane's query: dims [16 t + 8 h, +8)

  // ---- one 32-key block (keys kt + 32 kb .. +31 of the staged tile) against the wave's
  // 32 query rows
  auto compute_block = [&](const char* buf, int kt, int kb) {
    const int key0 = kt + kb * 32;
    const float moff = m_ref == -INFINITY ? 0.f : m_ref;
    f32x16 sc;
#pragma unroll
    for (int i = 0; i < 16; ++i) sc[i] = -moff;
    {
      const char* kr = buf + (kb * 32 + ql) * C::KPITCH + h * 16;
      uint4 kf[C::NT];
#pragma unroll
      for (int t = 0; t < C::NT; ++t) kf[t] = *reinterpret_cast<const uint4*>(kr + t * 32);
#pragma unroll
      for (int t = 0; t < C::NT; ++t) sc = mma32_f16(kf[t], qf[t], sc);
    }
    // V^T fragments of the block's two 16-key steps
    uint4 vf[2][C::ND];
#pragma unroll
    for (int st2 = 0; st2 < 2; ++st2)
#pragma unroll
      for (int u = 0; u < C::ND; ++u)
        vf[st2][u] = *reinterpret_cast<const uint4*>(buf + C::KBYTES + (u * 32 + ql) * C::PITCH +
                                                     (kb * 32 + st2 * 16 + h * 8) * 2);
    const bool full = key0 + 32 <= kend && key0 + 32 <= wave_limit;
    if (!full) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = key0 + 8 * (i >> 2) + 4 * h + (i & 3);
        if (!(key < key_limit && key < kend)) sc[i] = -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sc[i]);
    // raise the reference when a visible score would exceed it by more than 2^8 (or the
    // row had none yet): rare after the first block, so a wave-uniform branch
    const bool need = mx > (m_ref == -INFINITY ? -INFINITY : 8.f);
    if (__builtin_amdgcn_ballot_w64(need)) {
      float rm = mx + moff;  // this lane's largest score (or -inf)
      rm = fmaxf(rm, __shfl_xor(rm, 32, 64));
      const float m_new = fmaxf(m_ref, rm);
      if (m_new != m_ref) {
        const float alpha = __builtin_amdgcn_exp2f(m_ref - m_new);  // m_ref = -inf gives 0
        l_run *= alpha;
#pragma unroll
        for (int u = 0; u < C::ND; ++u) acc_o[u] *= alpha;
        const float d = m_new - moff;
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[i] -= d;
        m_ref = m_new;
      }
    }
    uint4 pf[2];
#pragma unroll
    for (int st2 = 0; st2 < 2; ++st2) {
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) p[e] = __builtin_amdgcn_exp2f(sc[8 * st2 + e]);
#pragma unroll
      for (int e = 0; e < 8; ++e) l_run += p[e];
      pf[st2] = make_uint4(pack_f16(p[0], p[1]), pack_f16(p[2], p[3]), pack_f16(p[4], p[5]),
                           pack_f16(p[6], p[7]));
    }
#pragma unroll
    for (int st2 = 0; st2 < 2; ++st2)
#pragma unroll
      for (int u = 0; u < C::ND; ++u) acc_o[u] = mma32_f16(vf[st2][u], pf[st2], acc_o[u]);
  };

  auto compute = [&](const char* buf, int kt) {
    if (!wave_live) return;
    for (int kb = kp; kb < kAttnTile / 32; kb += KP)
      if (kt + kb * 32 < kend) compute_block(buf, kt, kb);
  };

  // ---- pipeline: tile i computes from lds[i & 1].  The K and V halves of a tile are
  // loaded and stored at different points of an iteration (K half before the compute, V
  // half after it), each half re-issued as soon as it is stored, so two halves are
  // always in flight (the next tile's V half and the one after's K half during the
  // compute) and the memory pipe does not drain at a barrier.
  // q goes through LDS (the second tile buffer is still free): wave w stages query block
  // w (one copy per block, whichever waves compute it), its loads issued first, the first
  // two tiles' right behind them, and all three are consumed before the first barrier,
  // so the latencies overlap and q's loads cannot drift behind the tiles' (loads
  // complete in order: waiting for q leaves the tiles in flight)
  uint4 qv[C::NT];
  {
    const int lr = row0 + wave * 32 + ql;  // row this lane stages (wave = query block)
    const bool ok = wave < QB && lr < R;
    const int lj = ok ? lr / G : 0, lh = it.kvh * G + (ok ? lr % G : 0);
    const char* qh = reinterpret_cast<const char*>(Q) + (((int64_t)(sg.row0 + lj) * s.n_q + lh) * DH) * 2;
#pragma unroll
    for (int t = 0; t < C::NT; ++t) qv[t] = ld_global(qh + (t * 16 + h * 8) * 2);
  }
  __builtin_amdgcn_sched_barrier(0);  // keep the q loads ahead of the tile loads
  const Half k0 = load_k(kbeg);
  const Half v0 = load_v(kbeg);
  Half kh = load_k(kbeg + kAttnTile);
  Half vh = load_v(kbeg + kAttnTile);
  {
    char* qs = &lds[1][0] + (wave * 32 + ql) * C::QPITCH + h * 16;  // [block][32 rows][dh]
#pragma unroll
    for (int t = 0; t < C::NT; ++t) *reinterpret_cast<uint4*>(qs + t * 32) = qv[t];
  }
  store_k(lds[0], k0);
  store_v(lds[0], v0, kbeg);
  __syncthreads();
  {
    const char* qs = &lds[1][0] + (qb * 32 + ql) * C::QPITCH + h * 16;
#pragma unroll
    for (int t = 0; t < C::NT; ++t) {
      // rows past the segment (their scores are masked) keep a zero query
      const uint4 v = *reinterpret_cast<const uint4*>(qs + t * 32);
      qf[t] = row_ok ? v : make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();  // every wave has its q before tile 1 overwrites the buffer
  for (int i = 0; i < n_tiles; ++i) {
    const int kt = kbeg + i * kAttnTile;
    // lds[(i+1) & 1] is free (its last reader, tile i-1's compute, ended at the barrier).
    // Stores past the last tile fill a buffer nobody reads.
    store_k(lds[(i + 1) & 1], kh);
    __builtin_amdgcn_sched_barrier(0);  // the half's registers are free before its reload
    kh = load_k(kt + 2 * kAttnTile);
    compute(lds[i & 1], kt);
    store_v(lds[(i + 1) & 1], vh, kt + kAttnTile);
    __builtin_amdgcn_sched_barrier(0);
    vh = load_v(kt + 2 * kAttnTile);
    __syncthreads();  // lds[(i+1) & 1] holds tile i+1; lds[i & 1] is free
  }

  if (!(cell_max <= kF16Max)) atomicOr(range + it.seg, kRangeFlag);

  // ---- merge the key parts of each query block: waves kp > 0 hand (O, m, l) over
  // through LDS (the tile buffers are free after the last barrier); wave kp = 0 merges
  l_run += __shfl_xor(l_run, 32, 64);
  float* slot = reinterpret_cast<float*>(&lds[0][0]);  // [wave][ND*16 + 2][64 lanes]
  if (KP > 1) {
    if (wave_live && kp > 0) {
      float* my = slot + wave * C::SLOT;
#pragma unroll
      for (int u = 0; u < C::ND; ++u)
#pragma unroll
        for (int i = 0; i < 16; ++i) my[(u * 16 + i) * 64 + lane] = acc_o[u][i];
      my[(C::ND * 16) * 64 + lane] = m_ref;
      my[(C::ND * 16 + 1) * 64 + lane] = l_run;
    }
    __syncthreads();
  }
  if (!wave_live || kp != 0) return;
  float mm = m_ref;
  for (int p = 1; p < KP; ++p) mm = fmaxf(mm, slot[(qb + p * QBP) * C::SLOT + (C::ND * 16) * 64 + lane]);
  // a part that saw no key has m = -inf and weight 0; all empty keeps everything 0
  const float a0 = mm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_ref - mm);
  float L = a0 * l_run;
#pragma unroll
  for (int u = 0; u < C::ND; ++u) acc_o[u] *= a0;
  for (int p = 1; p < KP; ++p) {
    const float* o = slot + (qb + p * QBP) * C::SLOT;
    const float mp = o[(C::ND * 16) * 64 + lane];
    const float ap = mm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mp - mm);
    L += ap * o[(C::ND * 16 + 1) * 64 + lane];
#pragma unroll
    for (int u = 0; u < C::ND; ++u)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc_o[u][i] += ap * o[(u * 16 + i) * 64 + lane];
  }
  // the row's output normalized by its sum (0 where this key range held no visible key)
  const float inv = L > 0.f ? 1.f / L : 0.f;
  // The wave's 32 rows leave through its own merge slot (slot qb < QBP, never a merge
  // source), transposed there so that each store instruction writes whole rows.  LDS
  // operations of one wave complete in order: the fences only keep the compiler from
  // moving the reads above the writes.
  char* const tb = reinterpret_cast<char*>(slot + wave * C::SLOT);
  constexpr int LPR = DH / 8, RPI = 64 / LPR;  // 16-byte lanes per row, rows per store
  const int tc = lane % LPR, tr = lane / LPR;
  if (it.solo) {
    constexpr int FP = DH + 4;  // floats per staged row
    static_assert(32 * FP <= C::SLOT, "solo staging");
    float* const t = reinterpret_cast<float*>(tb);
#pragma unroll
    for (int u = 0; u < C::ND; ++u)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        // dims u*32 + 8 q4 + 4 h + 0..3 of this lane's query
        *reinterpret_cast<float4*>(t + ql * FP + u * 32 + 8 * q4 + 4 * h) =
            make_float4(acc_o[u][4 * q4] * inv, acc_o[u][4 * q4 + 1] * inv,
                        acc_o[u][4 * q4 + 2] * inv, acc_o[u][4 * q4 + 3] * inv);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < 32; i += RPI) {
      const int q = wrow0 + i + tr;  // the row this lane stores
      if (q >= R) continue;
      const float* src = t + (i + tr) * FP + tc * 8;
      const float4 a = *reinterpret_cast<const float4*>(src);
      const float4 b = *reinterpret_cast<const float4*>(src + 4);
      uint4 hi, lo;
      split_pair(a.x, a.y, hi.x, lo.x);
      split_pair(a.z, a.w, hi.y, lo.y);
      split_pair(b.x, b.y, hi.z, lo.z);
      split_pair(b.z, b.w, hi.w, lo.w);
      const int64_t o = ((int64_t)(sg.row0 + q / G) * s.n_q + it.kvh * G + q % G) * DH + tc * 8;
      *reinterpret_cast<uint4*>(out + o) = hi;
      *reinterpret_cast<uint4*>(out_lo + o) = lo;
    }
    return;
  }
  constexpr int HP = DH + 8;  // halves per staged row
  static_assert(32 * HP * 2 <= C::SLOT * 4, "partial staging");
  uint16_t* const t = reinterpret_cast<uint16_t*>(tb);
#pragma unroll
  for (int u = 0; u < C::ND; ++u)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4)
      *reinterpret_cast<uint2*>(t + ql * HP + u * 32 + 8 * q4 + 4 * h) =
          make_uint2(pack_f16(acc_o[u][4 * q4] * inv, acc_o[u][4 * q4 + 1] * inv),
                     pack_f16(acc_o[u][4 * q4 + 2] * inv, acc_o[u][4 * q4 + 3] * inv));
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // the item's partial rows: all 32 of the wave (rows past the segment hold zeros or
  // junk that the merge never reads; the item's slot has room for every row group row)
  const int64_t pbase = (int64_t)blockIdx.x * kAttnRowsH + (wrow0 - row0);
#pragma unroll
  for (int i = 0; i < 32; i += RPI)
    *reinterpret_cast<uint4*>(Opart + (pbase + i + tr) * DH + tc * 8) =
        *reinterpret_cast<const uint4*>(t + (i + tr) * HP + tc * 8);
  if (h == 0 && row_ok) MLpart[pbase + ql] = make_float2(mm, L);
}

// bf16 models: merge the key ranges of each query row of a (segment, kv head, row group)
// with more than one item, from the fp16 normalized outputs On_c and (m_c, l_c):
// out = sum_c w_c l_c On_c / sum_c w_c l_c, w_c = 2^(m_c - m), m the largest m_c, in range
// order.  DH/8 lanes per row, each owning 8 consecutive output dims (one 16-byte load per
// range); the ranges are taken 16 at a time with their loads in flight together.  The
// (m, l) pairs of a round are loaded once per row (lane i of the row takes range i), the
// row's maximum and the weights w_c l_c are formed across the row's lanes, and the
// weights reach every lane of the row through LDS.
template <int DH>
__global__ __launch_bounds__(64) void combine_kernel_h(Shape s, StepView sv,
                                                        const uint16_t* __restrict__ Opart,
                                                        const float2* __restrict__ MLpart,
                                                        bf16_t* out, bf16_t* out_lo) {
  constexpr int LPR = DH / 8;      // lanes per row
  constexpr int RPB = 64 / LPR;    // rows per block (one wave: many blocks per row group)
  constexpr int GRP = 16;          // key ranges per load round
  constexpr int PPL = GRP / LPR;   // (m, l) pairs per lane and round
  static_assert(GRP % LPR == 0 && (LPR & (LPR - 1)) == 0, "row lanes");
  __shared__ float wsh[RPB][GRP];  // the round's weights w_c l_c of each row
  const AttnGroup gr = sv.group[blockIdx.x];
  if (gr.n_items <= 1) return;     // its item wrote the output
  const Segment sg = gr.sg;
  const int G = s.n_q / s.n_kv;
  const int R = sg.len * G;
  const int sub = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int rl = blockIdx.y * RPB + sub;  // row within the group
  const int qr = gr.rowgrp * kAttnRowsH + rl;
  // (rows past the group still take part in the row-lane reductions; they store nothing)
  const bool live = rl < kAttnRowsH && qr < R;
  const int j = live ? qr / G : 0, head = gr.kvh * G + (live ? qr % G : 0);
  const int n = gr.n_items;
  const int64_t base = (int64_t)gr.first_item * kAttnRowsH + (live ? rl : 0);
  float mx = -INFINITY, L = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < n; c0 += GRP) {
    uint4 o[GRP];
#pragma unroll
    for (int u = 0; u < GRP; ++u)
      if (c0 + u < n)
        o[u] = *reinterpret_cast<const uint4*>(Opart + (base + (int64_t)(c0 + u) * kAttnRowsH) * DH +
                                               li * 8);
    float m_me[PPL], l_me[PPL];
    float gm = -INFINITY;
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      const int c = c0 + li + q * LPR;
      const float2 ml = c < n ? MLpart[base + (int64_t)c * kAttnRowsH] : make_float2(-INFINITY, 0.f);
      m_me[q] = ml.y > 0.f ? ml.x : -INFINITY;  // an empty range has weight 0
      l_me[q] = ml.y;
      gm = fmaxf(gm, m_me[q]);
    }
#pragma unroll
    for (int d = 1; d < LPR; d <<= 1) gm = fmaxf(gm, __shfl_xor(gm, d, 64));
    gm = fmaxf(gm, mx);
    if (gm > mx) {  // rescale what was merged so far to the new max
      const float a = __builtin_amdgcn_exp2f(mx - gm);  // mx = -inf gives 0
      L *= a;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] *= a;
      mx = gm;
    }
    float lsum = 0.f;
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      const float w = m_me[q] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_me[q] - mx) * l_me[q];
      wsh[sub][li + q * LPR] = w;
      lsum += w;
    }
#pragma unroll
    for (int d = 1; d < LPR; d <<= 1) lsum += __shfl_xor(lsum, d, 64);
    L += lsum;
    __syncthreads();  // (one wave) the round's weights are in LDS
#pragma unroll
    for (int u = 0; u < GRP; ++u)
      if (c0 + u < n) {
        const float w = wsh[sub][u];
        const f16x8 v = __builtin_bit_cast(f16x8, o[u]);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += w * (float)v[e];
      }
    __syncthreads();  // before the next round overwrites the weights
  }
  if (!live) return;
  const float inv = 1.f / L;
  const int64_t oo = ((int64_t)(sg.row0 + j) * s.n_q + head) * DH + li * 8;
  store_act4(out, out_lo, oo, make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv));
  store_act4(out, out_lo, oo + 4, make_float4(acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv));
}

// Merge the key ranges of each query row of a (segment, kv head, row group):
// out = sum_c 2^(m_c - m) O_c / sum_c 2^(m_c - m) l_c with m the largest m_c, in range
// order.  DH/4 lanes per row, each owning 4 consecutive output dims.  The ranges are
// taken 32 at a time, their (m, l) and O loads all in flight together, with the
// running max and sums rescaled when a later group raises the max.
template <typename T, int DH>
__global__ __launch_bounds__(128) void combine_kernel(Shape s, StepView sv,
                                                      const float* __restrict__ Opart,
                                                      const float2* __restrict__ MLpart, T* out,
                                                      T* out_lo) {
  constexpr int LPR = DH / 4;      // lanes per row
  constexpr int RPB = 128 / LPR;   // rows per block
  constexpr int GRP = 32;          // key ranges per load round
  const AttnGroup gr = sv.group[blockIdx.x];
  const Segment sg = gr.sg;
  const int G = s.n_q / s.n_kv;
  const int R = sg.len * G;
  const int sub = threadIdx.x / LPR, li = threadIdx.x % LPR;
  const int rl = blockIdx.y * RPB + sub;  // row within the group
  const int qr = gr.rowgrp * kAttnRows + rl;
  if (qr >= R) return;
  const int j = qr / G, head = gr.kvh * G + qr % G;
  const int n = gr.n_items;
  const int64_t base = (int64_t)gr.first_item * kAttnRows + rl;
  float mx = -INFINITY, L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int c0 = 0; c0 < n; c0 += GRP) {
    float2 ml[GRP];
    float4 o[GRP];
#pragma unroll
    for (int u = 0; u < GRP; ++u)
      if (c0 + u < n) {
        const int64_t prow = base + (int64_t)(c0 + u) * kAttnRows;
        ml[u] = MLpart[prow];
        o[u] = *reinterpret_cast<const float4*>(Opart + prow * DH + li * 4);
      }
    float gm = mx;
#pragma unroll
    for (int u = 0; u < GRP; ++u)
      if (c0 + u < n && ml[u].y > 0.f) gm = fmaxf(gm, ml[u].x);
    if (gm > mx) {  // rescale what was merged so far to the new max
      const float a = __builtin_amdgcn_exp2f(mx - gm);  // mx = -inf gives 0
      L *= a;
      acc.x *= a;
      acc.y *= a;
      acc.z *= a;
      acc.w *= a;
      mx = gm;
    }
#pragma unroll
    for (int u = 0; u < GRP; ++u)
      if (c0 + u < n && ml[u].y > 0.f) {
        const float w = __builtin_amdgcn_exp2f(ml[u].x - mx);
        L += w * ml[u].y;
        acc.x += w * o[u].x;
        acc.y += w * o[u].y;
        acc.z += w * o[u].z;
        acc.w += w * o[u].w;
      }
  }
  const float inv = 1.f / L;
  const int64_t o = ((int64_t)(sg.row0 + j) * s.n_q + head) * DH + li * 4;
  store_act4(out, out_lo, o, make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv));
}

template <typename T, int DH>
hipError_t launch_attn(const Shape& s, const StepView& dp, int n_items, int layer, const void* q,
                       const void* q_lo, void* o_part, float2* ml_part, void* out, void* out_lo,
                       uint32_t* range, hipStream_t st) {
  if constexpr (Elem<T>::kBytes == 2)
    SPP_LAUNCH((attn_kernel_h<DH>), dim3(n_items), dim3(64 * kAttnWaves), 0, st, s, dp,
                       layer, static_cast<const uint16_t*>(q), static_cast<uint16_t*>(o_part),
                       ml_part, static_cast<bf16_t*>(out), static_cast<bf16_t*>(out_lo), range);
  else
    SPP_LAUNCH((attn_kernel<T, DH>), dim3(n_items), dim3(64 * kAttnWaves), 0, st, s, dp,
                       layer, static_cast<const T*>(q), static_cast<const T*>(q_lo),
                       static_cast<float*>(o_part), ml_part);
  return hipGetLastError();
}

template <typename T, int DH>
hipError_t launch_combine(const Shape& s, const StepView& dp, int n_groups, const void* o_part,
                          const float2* ml_part, void* out, void* out_lo, hipStream_t st) {
  if constexpr (Elem<T>::kBytes == 2) {
    constexpr int RPB = 64 / (DH / 8);
    SPP_LAUNCH((combine_kernel_h<DH>), dim3(n_groups, kAttnRowsH / RPB), dim3(64), 0, st, s,
                       dp, static_cast<const uint16_t*>(o_part), ml_part, static_cast<bf16_t*>(out),
                       static_cast<bf16_t*>(out_lo));
  } else {
    constexpr int RPB = 128 / (DH / 4);
    SPP_LAUNCH((combine_kernel<T, DH>), dim3(n_groups, kAttnRows / RPB), dim3(128), 0, st, s,
                       dp, static_cast<const float*>(o_part), ml_part, static_cast<T*>(out),
                       static_cast<T*>(out_lo));
  }
  return hipGetLastError();
}

}  // namespace

namespace k {

hipError_t attention(const Shape& s, const StepView& dp, int n_items, int layer, const void* q,
                     const void* q_lo, void* o_part, float2* ml_part, void* out, void* out_lo,
                     uint32_t* range, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (s.bf16)
    return s.dh == 128 ? launch_attn<bf16_t, 128>(s, dp, n_items, layer, q, q_lo, o_part, ml_part,
                                                  out, out_lo, range, st)
                       : launch_attn<bf16_t, 64>(s, dp, n_items, layer, q, q_lo, o_part, ml_part,
                                                 out, out_lo, range, st);
  // fp32 models: head_dim 64 only (checked at model creation)
  return launch_attn<float, 64>(s, dp, n_items, layer, q, q_lo, o_part, ml_part, out, out_lo,
                                range, st);
}

hipError_t attention_combine(const Shape& s, const StepView& dp, int n_groups,
                             const void* o_part, const float2* ml_part, void* out, void* out_lo,
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
