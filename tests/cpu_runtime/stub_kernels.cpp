// Host stand-ins for the kernel launchers the runtime calls (the k:: interface of
// kernels.hpp), for the CPU build of the runtime under the sanitizers.  Test
// infrastructure only.
//
// The forward pass is not computed: the projections, norms and attention enqueue
// nothing but their place in the stream order.  What the runtime's own logic reads back
// is produced, with the meaning the kernels give it:
//   * the LM head writes a distribution with a planted maximum (token 7, margin 10) and
//     its summary (top-2, log-sum-exp, flags);
//   * the batched LM head's GEMM plants token 7 + row at margin 10 in its logits;
//   * the scan computes the top-2 (lowest index on ties), the set bit, the non-finite and
//     range flags, and publishes the sequence number in the done word last (release).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>

#include "kernels.hpp"

namespace spp {
namespace {

void summarize(const float* d, int V, const uint32_t* bitmap, bool lse, uint32_t extra_flags,
               ScanResult* out, uint32_t seq) {
  ScanResult r{};
  r.argmax = -1;
  r.second = -1;
  r.top1 = -std::numeric_limits<float>::infinity();
  r.top2 = r.top1;
  bool nonfinite = false;
  for (int v = 0; v < V; ++v) {
    const float x = d[v];
    if (!std::isfinite(x)) {
      nonfinite = true;
      continue;
    }
    if (x > r.top1) {
      r.top2 = r.top1;
      r.second = r.argmax;
      r.top1 = x;
      r.argmax = v;
    } else if (x > r.top2) {
      r.top2 = x;
      r.second = v;
    }
  }
  if (lse) {
    double s = 0.0;
    for (int v = 0; v < V; ++v)
      if (std::isfinite(d[v])) s += std::exp((double)d[v] - r.top1);
    r.lse = (float)(r.top1 + std::log(s));
  }
  r.flags = (nonfinite ? 1u : 0u) | (extra_flags & kRangeFlag);
  if (bitmap && r.argmax >= 0 && ((bitmap[r.argmax >> 5] >> (r.argmax & 31)) & 1u)) r.flags |= 2u;
  r.seq = seq;
  *out = r;
}

void plant(float* d, int V, int hot, const float* bias) {
  for (int v = 0; v < V; ++v) d[v] = 0.01f * (float)(v % 13) + (bias ? bias[v] : 0.f);
  d[hot % V] += 10.f;
}

hipError_t nothing(hipStream_t st) {
  stub::enqueue(st, [] {});
  return hipSuccess;
}

}  // namespace

namespace k {

int res_blocks(const Shape& s) { return (s.d + 1023) / 1024; }
int lmhead_blocks(const Shape&) { return 256; }
int scan_blocks(int, int n) { return std::max(4, std::min(64, 1024 / std::max(n, 1))); }

GemmPlan gemm_plan(const Shape&, int, int, int) { return GemmPlan{4, 2, 1, 2, 1, 2, 0}; }
GemmPlan gemm_plan_swiglu(const Shape&, int, int, int) { return GemmPlan{4, 2, 1, 2, 1, 2, 0}; }
GemmPlan gemm_plan_fp4(const Shape&, int, int, int) { return GemmPlan{4, 2, 1, 2, 1, 2, 0}; }
GemmPlan gemm_plan_swiglu_fp4(const Shape&, int, int, int) { return GemmPlan{4, 2, 1, 2, 1, 2, 0}; }
int pack_slab_steps(const Shape&, int, int K) { return std::max(1, K / 64); }
int pack_slab_steps_gateup(const Shape&, int, int K) { return std::max(1, K / 64); }
int pack_slab_steps_fp4(const Shape&, int, int K) { return std::max(1, K / 128); }
int pack_slab_steps_gateup_fp4(const Shape&, int, int K) { return std::max(1, K / 128); }

hipError_t embed(const Shape& s, const StepView& v, int, const void*, const void*, float*, void*,
                 void*, float*, float2*, uint32_t* range, hipStream_t st) {
  // the step's range words start clear, as the embedding kernel leaves them
  const StepParams* p = v.p;
  stub::enqueue(st, [p, range] {
    for (int i = 0; i < p->n_segments; ++i) range[i] = 0u;
  });
  (void)s;
  return hipSuccess;
}
hipError_t gemm(const Shape& s, const GemmPlan&, const void*, const void*, int M, int,
                const WeightCat&, int N, float* partials, hipStream_t st) {
  if (N == s.vocab)  // the batched LM head: one planted maximum per row
    stub::enqueue(st, [=] {
      for (int r = 0; r < M; ++r) plant(partials + (size_t)r * N, N, 7 + r, nullptr);
    });
  else
    stub::enqueue(st, [] {});
  return hipSuccess;
}
hipError_t gemm_swiglu(const Shape&, const GemmPlan&, const void*, const void*, int, int,
                       const WeightCat&, int, const float*, void*, void*, hipStream_t st) {
  return nothing(st);
}
hipError_t pack_weight(int, const void*, void*, int, int, int, hipStream_t st) { return nothing(st); }
hipError_t gemm_fp4(const Shape&, const GemmPlan&, const void*, const void*, int, int,
                    const WeightCat&, int, float*, hipStream_t st) {
  return nothing(st);
}
hipError_t gemm_swiglu_fp4(const Shape&, const GemmPlan&, const void*, const void*, int, int,
                           const WeightCat&, int, const float*, void*, void*, hipStream_t st) {
  return nothing(st);
}
hipError_t pack_weight_fp4(const void*, const void*, void*, void*, int, int, int, hipStream_t st) {
  return nothing(st);
}
hipError_t qkv_epilogue(const Shape&, const StepView&, int, int, const float*, int, const float*,
                        const float2*, void*, void*, uint32_t*, hipStream_t st) {
  return nothing(st);
}
hipError_t attention(const Shape&, const StepView&, int, int, const void*, const void*, void*,
                     float2*, void*, void*, uint32_t*, hipStream_t st) {
  return nothing(st);
}
hipError_t attention_combine(const Shape&, const StepView&, int, const void*, const float2*,
                             void*, void*, hipStream_t st) {
  return nothing(st);
}
hipError_t residual(const Shape&, int, const float*, int, float*, const void*, void*, void*,
                    float*, hipStream_t st) {
  return nothing(st);
}
hipError_t swiglu(const Shape&, int, const float*, int, const float*, void*, void*, hipStream_t st) {
  return nothing(st);
}
hipError_t lmhead_gemv(const Shape& s, const float*, const void*, const void*, const float* bias,
                       float* dist, const uint32_t* bitmap, ScanPartial*, ScanResult* result,
                       const uint32_t* range, hipStream_t st) {
  const int V = s.vocab;
  stub::enqueue(st, [=] {
    plant(dist, V, 7, bias);
    summarize(dist, V, bitmap, true, range ? *range : 0u, result, 0u);
  });
  return hipSuccess;
}
hipError_t final_norm_rows(const Shape&, const StepView&, int, const float*, const void*, void*,
                           void*, hipStream_t st) {
  return nothing(st);
}
hipError_t scan(const Shape& s, int n, const ScanJob& job, hipStream_t st) {
  const int V = s.vocab;
  const ScanJob j = job;  // the runtime's job record may be reused after the launch
  stub::enqueue(st, [=] {
    for (int b = 0; b < n; ++b) {
      float* d = j.dist[b];
      if (j.src) {
        for (int v = 0; v < V; ++v) {
          float x = j.bias ? j.bias[v] : 0.f;
          for (int sp = 0; sp < j.src_splits; ++sp) x += j.src[((size_t)sp * n + b) * V + v];
          d[v] = x;
        }
      }
      const uint32_t extra = j.flag_src[b] ? *j.flag_src[b] : 0u;
      summarize(d, V, j.bitmap[b], j.with_lse != 0, extra, j.result[b], j.seq);
    }
    if (j.done) __atomic_store_n(j.done, j.seq, __ATOMIC_RELEASE);
  });
  return hipSuccess;
}
hipError_t shift_cells(const Shape&, void*, int64_t, int, int, hipStream_t st) { return nothing(st); }
hipError_t copy_bytes(void* dst, const void* src, size_t n, hipStream_t st) {
  stub::enqueue(st, [=] { std::memcpy(dst, src, n); });
  return hipSuccess;
}

}  // namespace k
}  // namespace spp
