// Host runtime behind the C ABI (include/spp.h): models, sessions, the ready-
// distribution record with its epoch, the step scheduler that packs entries into
// one device pass, the gate's decision logic and the invalidation discipline.
#include "spp.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

#include "kernels.hpp"

using namespace spp;

namespace spp {

thread_local LaunchRecorder* launch_recorder = nullptr;

bool recorder_events(hipEvent_t* start, hipEvent_t* stop) {
  LaunchRecorder* r = launch_recorder;
  if (!r || r->cur < 0) return false;
  if (r->used == r->start.size()) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return false;
    if (hipEventCreate(&b) != hipSuccess) {
      hipEventDestroy(a);
      return false;
    }
    r->start.push_back(a);
    r->stop.push_back(b);
    r->cls.push_back(-1);
  }
  r->cls[r->used] = r->cur;
  *start = r->start[r->used];
  *stop = r->stop[r->used];
  ++r->used;
  return true;
}

}  // namespace spp

namespace {

thread_local std::string t_err;

spp_status fail(spp_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return st;
}

#define HIPCHK(expr)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess) return fail(SPP_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// A device buffer that grows on demand.  Growing frees the old block, so the caller
// must make sure no queued work still uses it.
struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
};

// Per-kernel timing for spp_profile_preposition (dispatch events, see LaunchRecorder).
using Prof = LaunchRecorder;

struct Model {
  spp_model_config cfg{};
  Shape s{};
  int device = 0;
  int n_cu = 256;                     // compute units of the device (attention work sizing)
  size_t elem = 2;
  const void* embed = nullptr;
  const void* final_norm = nullptr;
  const void* lm_head = nullptr;
  const float* lm_bias = nullptr;
  std::vector<const void*> attn_norm, wq, wk, wv, wo, mlp_norm, wg, wu, wd;  // wq..wd tiled
  bool fp4 = false;                   // wq..wd are MXFP4 codes (tiled), scales in wsc
  std::vector<const void*> wsc[7];    // tiled e8m0 scales per spp_weight_kind (MXFP4)
  std::vector<void*> owned;           // library-owned packed copies (weights_packed == 0)
  void* lm_tiled = nullptr;           // packed LM head for the batched path (max_sessions > 1)
  int slab[5] = {1, 1, 1, 1, 1};      // tiled-layout slab (K-steps) of QKV, O, gate/up, down, LM head
  // work buffers
  float* x = nullptr;
  void* h = nullptr;
  void* q = nullptr;
  void* att = nullptr;
  void* act = nullptr;
  float* part = nullptr;
  size_t part_elems = 0;              // floats of `part`
  float* ss = nullptr;                // row sums of squares [max_tokens][res_blocks]
  uint32_t* range = nullptr;          // the step's fp16 range word per segment [kMaxSegments]
  float2* rope = nullptr;
  void* z = nullptr;
  float* logits_rows = nullptr;
  ScanPartial* lm_parts = nullptr;   // lmhead: lmhead_blocks; batched: [64][scan_blocks]
  ScanPartial* gate_parts = nullptr; // [64][scan_blocks]
  ScanResult* gate_host = nullptr;   // pinned, device-mapped [64] results, then the done word
  ScanResult* gate_dev = nullptr;
  uint32_t gate_seq = 0;
  DevBuf o_part, ml_part, params_dev;
  char* params_host = nullptr;
  size_t params_host_bytes = 0;
  hipEvent_t params_free = nullptr;  // the last params upload has been consumed
  hipEvent_t step_done = nullptr;    // the last step has finished with the work buffers
  hipEvent_t chunk_end[2] = {};      // ends of the last two layer chunks of a yielding pass
  bool step_recorded = false;
  std::mutex mu;       // one step at a time per model (work buffers)
  std::mutex gate_mu;  // one gate scan at a time per model (gate buffers)
};

struct Session {
  Model* m = nullptr;
  int id = 0;
  int capacity = 0, cap_stride = 0, budget = 0;
  void* kv = nullptr;
  size_t kv_bytes = 0;
  std::mutex mu;
  int n_s = 0;
  std::vector<int32_t> entry;  // the pre-positioned entry (speculative cells n_s..)
  bool valid = false;
  uint64_t epoch = 0;
  int position = -1;
  float* dist = nullptr;
  hipEvent_t done = nullptr;
  uint64_t decoded_epoch = ~0ull;  // epoch whose device work was seen finished
  ScanResult* summary = nullptr;  // device slot written by the LM head
  // Released with the last reference: a gate that looked the session up by its id keeps
  // it alive until it returns, even when spp_session_destroy runs meanwhile.
  ~Session() {
    if (done) {
      hipEventSynchronize(done);
      hipEventDestroy(done);
    }
    if (summary) hipFree(summary);
  }
};

// Sessions by id.  Calls that take a ready handle (a value naming the session by id)
// hold a reference for their duration; spp_session_destroy drops the registry's.
std::mutex g_reg_mu;
std::unordered_map<int, std::shared_ptr<Session>> g_sessions;
int g_next_id = 1;

std::shared_ptr<Session> lookup(int id) {
  std::lock_guard<std::mutex> lk(g_reg_mu);
  auto it = g_sessions.find(id);
  return it == g_sessions.end() ? nullptr : it->second;
}

size_t layer_elems(const Model& m, int cap_stride) {
  return (size_t)2 * m.s.n_kv * cap_stride * m.s.dh;
}

// Grows a device buffer; waits for the last step first because a queued step may
// still read the old block.
spp_status ensure_dev(Model& m, DevBuf& b, size_t bytes) {
  if (b.bytes >= bytes) return SPP_OK;
  if (m.step_recorded) HIPCHK(hipEventSynchronize(m.step_done));
  if (b.p) HIPCHK(hipFree(b.p));
  b.p = nullptr;
  b.bytes = 0;
  const size_t nb = (size_t)round_up((int64_t)(bytes + bytes / 2), 4096);
  if (hipMalloc(&b.p, nb) != hipSuccess) return fail(SPP_E_NOMEM, "hipMalloc(%zu) failed", nb);
  b.bytes = nb;
  return SPP_OK;
}

struct SegReq {
  Session* s;
  const int32_t* tok;
  int len;
  int n_past;
  float* dist;
  const uint32_t* bitmap;
};

#define LAUNCH(cls, call)                                                                  \
  do {                                                                                     \
    if (prof) prof->cur = (cls);                                                           \
    hipError_t e_ = (call);                                                                \
    if (prof) prof->cur = -1;                                                              \
    if (e_ != hipSuccess) return fail(SPP_E_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

// Cooperative yield of an idle-window pass (Sec. 3.1): the layers are enqueued in chunks,
// at most two chunks ahead of the device, and before each chunk the caller's flag is read;
// once it is set, nothing more is enqueued and the pass ends when the device has drained.
struct YieldCtl {
  const volatile uint32_t* flag;
  int chunk;       // layers per chunk
  bool yielded;
};

// Before chunk c (c >= 1) of a yielding pass: mark the end of chunk c-1, then wait until
// chunk c-2 has finished (two chunks in flight keep the device busy while the host
// waits), watching the flag.  Returns true when the pass must stop.
bool chunk_gate(Model& m, YieldCtl& y, int c, hipStream_t st, spp_status* rc) {
  *rc = SPP_OK;
  if (hipEventRecord(m.chunk_end[(c - 1) & 1], st) != hipSuccess) {
    *rc = fail(SPP_E_HIP, "hipEventRecord failed");
    return true;
  }
  // acquire loads: the flag is written by another thread, the done word by the device
  bool stop = __atomic_load_n(y.flag, __ATOMIC_ACQUIRE) != 0;
  while (!stop && c >= 2) {
    const hipError_t q = hipEventQuery(m.chunk_end[c & 1]);
    if (q == hipSuccess) break;
    if (q != hipErrorNotReady) {
      *rc = fail(SPP_E_HIP, "chunk wait: %s", hipGetErrorString(q));
      return true;
    }
    stop = __atomic_load_n(y.flag, __ATOMIC_ACQUIRE) != 0;
    if (!stop) std::this_thread::yield();
  }
  if (!stop) return false;
  y.yielded = true;
  // the work already enqueued finishes; the next step of the model orders after it
  if (hipEventRecord(m.step_done, st) != hipSuccess ||
      hipEventSynchronize(m.chunk_end[(c - 1) & 1]) != hipSuccess)
    *rc = fail(SPP_E_HIP, "draining a yielded pass failed");
  return true;
}

// One device pass over the packed rows of `segs` (all of the same model).  With
// `logits`, also the LM head and reductions at each segment's last row.  With `y`, the
// pass yields as described at YieldCtl (then y->yielded is set and no logits are made).
// Caller holds m.mu and every session's mutex.
spp_status run_step(Model& m, const SegReq* segs, int nseg, bool logits, hipStream_t st,
                    Prof* prof, YieldCtl* y = nullptr) {
  const Shape& s = m.s;
  const int G = s.n_q / s.n_kv;
  int rows = 0;
  for (int i = 0; i < nseg; ++i) rows += segs[i].len;
  if (rows <= 0 || rows > m.cfg.max_tokens || nseg > kMaxSegments)
    return fail(SPP_E_INVALID_ARG, "step of %d rows / %d segments exceeds the model limits", rows, nseg);
  if (logits && nseg > k::kScanMax)
    return fail(SPP_E_INVALID_ARG, "at most %d decision points per pass", k::kScanMax);
  // several decision points in one pass take the tiled LM head and its partial logits,
  // sized at model creation for max_sessions rows
  if (logits && nseg > 1 && (nseg > m.cfg.max_sessions || !m.lm_tiled || !m.logits_rows))
    return fail(SPP_E_INVALID_ARG, "%d decision points in one pass exceed max_sessions %d", nseg,
                m.cfg.max_sessions);

  // ---- attention work list: units of (segment, kv head, row group of RG rows: 256 for
  // bf16 models, 128 for fp32), each cut into key ranges of whole 64-key blocks.  A unit
  // of S blocks gets S * target / total items, rounded (at least one, at most S), and its
  // blocks are dealt out evenly, so no item holds more than one block above the others of
  // its unit.  target = the compute units, so that a short list fits the chip once (one
  // work item per compute unit: an item holds most of a CU's LDS), or one item per ~64
  // blocks when the list is longer (many sessions of unequal lengths), dealt longest
  // first so that the launch ends on short items.  For the 64-session batch (U[1024,
  // 8192] cells) that measured best among 24-128 blocks per item: longer items carry less
  // of the per-item start-up and fewer partials for the merge, shorter ones end evenly.
  // segment i as the kernels see it (row0: its first packed row)
  std::vector<int> row0(nseg + 1, 0);
  for (int i = 0; i < nseg; ++i) row0[i + 1] = row0[i] + segs[i].len;
  auto seg_of = [&](int i) {
    return Segment{segs[i].s->kv, segs[i].s->cap_stride, segs[i].n_past, row0[i], segs[i].len};
  };
  std::vector<AttnItem> items;
  std::vector<AttnGroup> groups;
  const int RG = attn_rows(s);
  {
    int64_t total_blocks = 0;
    for (int i = 0; i < nseg; ++i) {
      const int R = segs[i].len * G;
      const int rgs = (R + RG - 1) / RG;
      for (int rg = 0; rg < rgs; ++rg) {
        const int last = std::min(rg * RG + RG, R) - 1;
        const int limit = segs[i].n_past + last / G + 1;
        total_blocks += (int64_t)s.n_kv * ((limit + kAttnSub - 1) / kAttnSub);
      }
    }
    struct Unit {
      int seg, kvh, rg, limit;
      int64_t nb, n;
    };
    std::vector<Unit> units;
    const int64_t target = std::max<int64_t>(m.n_cu, total_blocks / 64);
    for (int i = 0; i < nseg; ++i) {
      const int R = segs[i].len * G;
      const int rgs = (R + RG - 1) / RG;
      for (int kvh = 0; kvh < s.n_kv; ++kvh)
        for (int rg = 0; rg < rgs; ++rg) {
          const int last = std::min(rg * RG + RG, R) - 1;
          const int limit = segs[i].n_past + last / G + 1;
          const int64_t nb = (limit + kAttnSub - 1) / kAttnSub;
          // the item count nearest nb * target / total (rounded, not floored: a unit
          // just short of two items' blocks would otherwise make one item of twice the size)
          const int64_t n = std::min<int64_t>(
              nb, std::max<int64_t>(1, (2 * nb * target + total_blocks) / (2 * total_blocks)));
          units.push_back(Unit{i, kvh, rg, limit, nb, n});
        }
    }
    // longest items first (units of many sessions differ): the dispatcher starts workgroups
    // in index order, so the launch ends on the short ones; equal sizes keep their order
    std::stable_sort(units.begin(), units.end(), [](const Unit& a, const Unit& b) {
      return a.nb * b.n > b.nb * a.n;  // a.nb / a.n > b.nb / b.n
    });
    for (const Unit& u : units) {
      const int first = (int)items.size();
      for (int64_t j = 0; j < u.n; ++j) {
        const int b0 = (int)(j * u.nb / u.n), b1 = (int)((j + 1) * u.nb / u.n);
        items.push_back(AttnItem{seg_of(u.seg), u.seg, u.kvh, u.rg, b0 * kAttnSub,
                                 std::min(b1 * kAttnSub, u.limit), u.n == 1 ? 1 : 0});
      }
      // the merge's work list: a bf16 model's single-item group was written by its item
      if (!s.bf16 || u.n > 1)
        groups.push_back(AttnGroup{seg_of(u.seg), u.seg, u.kvh, u.rg, first,
                                   (int32_t)items.size() - first});
    }
  }

  // ---- step record: header, then the arrays, 16-byte aligned
  size_t off = round_up(sizeof(StepParams), 16);
  const size_t off_tok = off;
  off = round_up(off + 4 * (size_t)rows, 16);
  const size_t off_row = off;
  off = round_up(off + sizeof(RowInfo) * (size_t)rows, 16);
  const size_t off_it = off;
  off = round_up(off + sizeof(AttnItem) * items.size(), 16);
  const size_t off_gr = off;
  off = round_up(off + sizeof(AttnGroup) * groups.size(), 16);
  const size_t bytes = off;

  spp_status rc;
  if ((rc = ensure_dev(m, m.params_dev, bytes)) != SPP_OK) return rc;
  // attention partials: fp16 normalized outputs for bf16 models, fp32 sums for fp32 models
  if ((rc = ensure_dev(m, m.o_part, items.size() * RG * s.dh * (s.bf16 ? 2 : 4))) != SPP_OK) return rc;
  if ((rc = ensure_dev(m, m.ml_part, items.size() * RG * sizeof(float2))) != SPP_OK) return rc;

  // the pinned staging record is reused: wait until its last upload was consumed
  HIPCHK(hipEventSynchronize(m.params_free));
  if (m.params_host_bytes < bytes) {
    if (m.params_host) HIPCHK(hipHostFree(m.params_host));
    m.params_host = nullptr;
    const size_t nb = (size_t)round_up((int64_t)(bytes + bytes / 2), 4096);
    if (hipHostMalloc((void**)&m.params_host, nb, hipHostMallocDefault) != hipSuccess)
      return fail(SPP_E_NOMEM, "hipHostMalloc(%zu) failed", nb);
    m.params_host_bytes = nb;
  }
  StepParams* hp = reinterpret_cast<StepParams*>(m.params_host);
  memset(hp, 0, sizeof(StepParams));
  hp->n_rows = rows;
  hp->n_segments = nseg;
  hp->n_items = (int32_t)items.size();
  hp->n_groups = (int32_t)groups.size();
  hp->off_token = off_tok;
  hp->off_row = off_row;
  hp->off_item = off_it;
  hp->off_group = off_gr;
  int32_t* tok = reinterpret_cast<int32_t*>(m.params_host + off_tok);
  RowInfo* ri = reinterpret_cast<RowInfo*>(m.params_host + off_row);
  int r = 0;
  for (int i = 0; i < nseg; ++i) {
    hp->seg[i] = seg_of(i);
    for (int j = 0; j < segs[i].len; ++j, ++r) {
      tok[r] = segs[i].tok[j];
      ri[r] = RowInfo{segs[i].s->kv, segs[i].s->cap_stride, segs[i].n_past + j, i, 0};
    }
  }
  if (!items.empty()) memcpy(m.params_host + off_it, items.data(), sizeof(AttnItem) * items.size());
  if (!groups.empty()) memcpy(m.params_host + off_gr, groups.data(), sizeof(AttnGroup) * groups.size());

  // ---- order after the previous step of this model, whatever stream it ran on
  if (m.step_recorded) HIPCHK(hipStreamWaitEvent(st, m.step_done, 0));
  const StepView dp = step_view(static_cast<const StepParams*>(m.params_dev.p), hp);
  HIPCHK(hipMemcpyAsync(m.params_dev.p, m.params_host, bytes, hipMemcpyHostToDevice, st));
  HIPCHK(hipEventRecord(m.params_free, st));

  const int M = rows, d = s.d, F = s.ffn;
  const int nq = s.n_q * s.dh, nkv = s.n_kv * s.dh;
  // second halves (lo) of the split activations, right after the hi arrays
  const size_t Mx = (size_t)m.cfg.max_tokens;
  void* h_lo = static_cast<char*>(m.h) + Mx * d * m.elem;
  void* att_lo = static_cast<char*>(m.att) + Mx * nq * m.elem;
  void* act_lo = static_cast<char*>(m.act) + Mx * F * m.elem;
  void* z_lo = static_cast<char*>(m.z) + (size_t)k::kScanMax * d * m.elem;
  void* q_lo = static_cast<char*>(m.q) + Mx * nq * m.elem;
  const int n_items = (int)items.size(), n_groups = (int)groups.size();

  // h holds y = x * g of the next projection (RMSNorm factored; see k::res_blocks)
  LAUNCH(KC_EMBED, k::embed(s, dp, M, m.embed, m.attn_norm[0], m.x, m.h, h_lo, m.ss, m.rope, m.range,
                            st));
  const auto plan = m.fp4 ? k::gemm_plan_fp4 : k::gemm_plan;
  const auto gemm = m.fp4 ? k::gemm_fp4 : k::gemm;
  const k::GemmPlan p_qkv = plan(s, M, nq + 2 * nkv, d);
  const k::GemmPlan p_o = plan(s, M, d, nq);
  const k::GemmPlan p_gu = plan(s, M, 2 * F, d);
  // gate/up with the SwiGLU fused (no K-splits), where it applies
  const k::GemmPlan p_sw = m.fp4 ? k::gemm_plan_swiglu_fp4(s, M, F, d) : k::gemm_plan_swiglu(s, M, F, d);
  const auto gemm_sw = m.fp4 ? k::gemm_swiglu_fp4 : k::gemm_swiglu;
  const k::GemmPlan p_dn = plan(s, M, d, F);
  // every projection's split-K partials must fit the buffer sized at model creation
  for (const auto& pn : {std::make_pair(p_qkv, nq + 2 * nkv), std::make_pair(p_o, d),
                         std::make_pair(p_gu, 2 * F), std::make_pair(p_dn, d)})
    if ((size_t)pn.first.splits * M * pn.second > m.part_elems)
      return fail(SPP_E_INVALID_ARG, "partials of %d x %d rows exceed the work buffer", M, pn.second);
  auto sc = [&](int kind, int l) -> const void* { return m.fp4 ? m.wsc[kind][l] : nullptr; };
  for (int l = 0; l < s.n_layers; ++l) {
    if (y && l > 0 && l % y->chunk == 0) {
      spp_status yrc;
      if (chunk_gate(m, *y, l / y->chunk, st, &yrc)) {
        m.step_recorded = true;
        return yrc;
      }
    }
    WeightCat wqkv{{m.wq[l], m.wk[l], m.wv[l]}, {0, nq, nq + nkv, nq + 2 * nkv}, m.slab[0],
                   {sc(SPP_W_Q, l), sc(SPP_W_K, l), sc(SPP_W_V, l)}};
    LAUNCH(KC_GEMM_QKV, gemm(s, p_qkv, m.h, h_lo, M, d, wqkv, nq + 2 * nkv, m.part, st));
    LAUNCH(KC_QKV_EPI, k::qkv_epilogue(s, dp, M, l, m.part, p_qkv.splits, m.ss, m.rope, m.q, q_lo,
                                       m.range, st));
    LAUNCH(KC_ATTN, k::attention(s, dp, n_items, l, m.q, q_lo, m.o_part.p,
                                 static_cast<float2*>(m.ml_part.p), m.att, att_lo, m.range, st));
    LAUNCH(KC_ATTN_COMBINE, k::attention_combine(s, dp, n_groups, m.o_part.p,
                                                 static_cast<float2*>(m.ml_part.p), m.att, att_lo,
                                                 st));
    WeightCat wo{{m.wo[l], nullptr, nullptr}, {0, d, d, d}, m.slab[1], {sc(SPP_W_O, l), nullptr, nullptr}};
    LAUNCH(KC_GEMM_O, gemm(s, p_o, m.att, att_lo, M, nq, wo, d, m.part, st));
    LAUNCH(KC_RESID_NORM, k::residual(s, M, m.part, p_o.splits, m.x, m.mlp_norm[l], m.h, h_lo, m.ss,
                                      st));
    WeightCat wgu{{m.wg[l], m.wu[l], nullptr}, {0, F, 2 * F, 2 * F}, m.slab[2],
                  {sc(SPP_W_GATE, l), sc(SPP_W_UP, l), nullptr}};
    if (p_sw.splits == 1) {
      LAUNCH(KC_GEMM_GATEUP, gemm_sw(s, p_sw, m.h, h_lo, M, d, wgu, F, m.ss, m.act, act_lo, st));
    } else {
      LAUNCH(KC_GEMM_GATEUP, gemm(s, p_gu, m.h, h_lo, M, d, wgu, 2 * F, m.part, st));
      LAUNCH(KC_SWIGLU, k::swiglu(s, M, m.part, p_gu.splits, m.ss, m.act, act_lo, st));
    }
    WeightCat wdn{{m.wd[l], nullptr, nullptr}, {0, d, d, d}, m.slab[3], {sc(SPP_W_DOWN, l), nullptr, nullptr}};
    LAUNCH(KC_GEMM_DOWN, gemm(s, p_dn, m.act, act_lo, M, F, wdn, d, m.part, st));
    const void* g_next = l + 1 < s.n_layers ? m.attn_norm[l + 1] : nullptr;
    LAUNCH(KC_RESID_NORM, k::residual(s, M, m.part, p_dn.splits, m.x, g_next, m.h, h_lo, m.ss, st));
  }

  if (logits) {
    if (nseg == 1) {
      const float* xr = m.x + (int64_t)(segs[0].len - 1) * d;
      LAUNCH(KC_LMHEAD, k::lmhead_gemv(s, xr, m.final_norm, m.lm_head, m.lm_bias, segs[0].dist,
                                       segs[0].bitmap, m.lm_parts, segs[0].s->summary, m.range,
                                       st));
    } else {
      LAUNCH(KC_LMHEAD, k::final_norm_rows(s, dp, nseg, m.x, m.final_norm, m.z, z_lo, st));
      const k::GemmPlan p_lm = k::gemm_plan(s, nseg, s.vocab, d);
      WeightCat wl{{m.lm_tiled, nullptr, nullptr}, {0, s.vocab, s.vocab, s.vocab}, m.slab[4], {}};
      LAUNCH(KC_LMHEAD, k::gemm(s, p_lm, m.z, z_lo, nseg, d, wl, s.vocab, m.logits_rows, st));
      k::ScanJob job{};
      for (int i = 0; i < nseg; ++i) {
        job.dist[i] = segs[i].dist;
        job.bitmap[i] = segs[i].bitmap;
        job.result[i] = segs[i].s->summary;
        job.flag_src[i] = m.range + i;
      }
      job.src = m.logits_rows;
      job.src_splits = p_lm.splits;
      job.bias = m.lm_bias;
      job.parts = m.lm_parts;
      job.seq = 1;
      job.with_lse = 1;
      LAUNCH(KC_SCAN, k::scan(s, nseg, job, st));
    }
  }
  HIPCHK(hipEventRecord(m.step_done, st));
  m.step_recorded = true;
  return SPP_OK;
}

spp_status check_tokens(const Model& m, const int32_t* t, int n) {
  if (!t) return fail(SPP_E_INVALID_ARG, "null token array");
  for (int i = 0; i < n; ++i)
    if (t[i] < 0 || t[i] >= m.s.vocab)
      return fail(SPP_E_INVALID_ARG, "token %d at %d outside [0, %d)", t[i], i, m.s.vocab);
  return SPP_OK;
}

void invalidate(Session& s) {  // Sec. 3.6: flags cleared in the same step as the mutation
  s.valid = false;
  s.entry.clear();
  ++s.epoch;
}

void fill_summary(const ScanResult& r, int position, spp_summary* out) {
  out->argmax = r.argmax;
  out->top1 = r.top1;
  out->top2 = r.top2;
  out->gap = r.top1 - r.top2;
  out->lse = r.lse;
  out->position = position;
  out->flags = r.flags & 7u;
}

spp_gate_outcome decide(const ScanResult& r, float tau, int32_t* token) {
  *token = -1;
  // non-finite logits, or a distribution whose fp16 attention saw an input beyond range
  if (r.flags & (1u | kRangeFlag)) return SPP_FALL_NONFINITE;
  const float gap = r.top1 - r.top2;
  if (!(gap > tau)) return SPP_FALL_GAP;  // Eq. (gate): strict
  if (!(r.flags & 2u)) return SPP_FALL_NOT_IN_SET;
  *token = r.argmax;
  return SPP_SERVED;
}

// Whether the device work of the session's current record has finished (Alg. 2 serves
// only a decoded distribution).  Events complete once and a new record bumps the epoch,
// so a completion seen for this epoch is remembered and the event is not queried again.
// Caller holds s.mu.  Returns SPP_OK and sets *done, or an error.
spp_status decoded(Session& s, bool* done) {
  *done = false;
  if (s.decoded_epoch == s.epoch) {
    *done = true;
    return SPP_OK;
  }
  const hipError_t q = hipEventQuery(s.done);
  if (q == hipErrorNotReady) return SPP_OK;
  if (q != hipSuccess) return fail(SPP_E_HIP, "hipEventQuery: %s", hipGetErrorString(q));
  s.decoded_epoch = s.epoch;
  *done = true;
  return SPP_OK;
}

// The done word after the scan results in the pinned gate block.
volatile uint32_t* gate_done_host(Model& m) {
  return reinterpret_cast<volatile uint32_t*>(m.gate_host + k::kScanMax);
}
uint32_t* gate_done_dev(Model& m) { return reinterpret_cast<uint32_t*>(m.gate_dev + k::kScanMax); }

// Waits until the scan has published `seq` in the done word (written after every result
// of the batch is visible).  Falls back to the stream's completion; never waits forever.
spp_status wait_done(Model& m, uint32_t seq, hipStream_t st) {
  volatile uint32_t* w = gate_done_host(m);
  const auto t0 = std::chrono::steady_clock::now();
  for (uint64_t it = 0;; ++it) {
    if (__atomic_load_n(w, __ATOMIC_ACQUIRE) == seq) return SPP_OK;
    if ((it & 1023) == 1023) {
      const hipError_t q = hipStreamQuery(st);
      if (q == hipSuccess) {
        if (__atomic_load_n(w, __ATOMIC_ACQUIRE) == seq) return SPP_OK;
        return fail(SPP_E_HIP, "gate scan finished without publishing its result");
      }
      if (q != hipErrorNotReady) return fail(SPP_E_HIP, "gate scan: %s", hipGetErrorString(q));
      if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(20))
        return fail(SPP_E_HIP, "gate scan did not finish within 20 s");
    }
  }
}

}  // namespace

struct spp_model_s : Model {};
struct spp_session_s : Session {};

extern "C" {

const char* spp_last_error(void) { return t_err.c_str(); }

}  // extern "C"

namespace {

// Shape checks shared by model creation and weight packing.
spp_status check_config(const spp_model_config& c) {
  const bool bf16 = c.dtype == SPP_DTYPE_BF16;
  if (c.dtype != SPP_DTYPE_BF16 && c.dtype != SPP_DTYPE_F32) return fail(SPP_E_INVALID_ARG, "dtype");
  if (c.n_layers < 1 || c.d_model < 1 || c.n_q_heads < 1 || c.n_kv_heads < 1 || c.ffn_dim < 1 ||
      c.vocab < 2 || c.n_q_heads % c.n_kv_heads)
    return fail(SPP_E_INVALID_ARG, "bad model shape");
  if (bf16 ? (c.head_dim != 64 && c.head_dim != 128) : c.head_dim != 64)
    return fail(SPP_E_INVALID_ARG, "head_dim must be 64 or 128 (bf16) / 64 (fp32)");
  const int kmul = bf16 ? 64 : 32;
  if (c.d_model % kmul || c.ffn_dim % kmul || (c.n_q_heads * c.head_dim) % kmul)
    return fail(SPP_E_INVALID_ARG, "d_model, ffn_dim and n_q_heads*head_dim must be multiples of %d", kmul);
  {
    const int E = bf16 ? 8 : 4;
    const int nc = (c.d_model + 64 * E - 1) / (64 * E);
    if (c.d_model % E || !(nc == 1 || nc == 2 || nc == 4 || nc == 8 || nc == 10 || nc == 16))
      return fail(SPP_E_INVALID_ARG, "d_model %d not supported by the LM head kernel", c.d_model);
  }
  if (c.max_sessions > 1 && c.vocab % 16)
    return fail(SPP_E_INVALID_ARG, "batched models need vocab %% 16 == 0");
  if (c.max_tokens < 1 || c.max_sessions < 1 || c.max_sessions > k::kScanMax)
    return fail(SPP_E_INVALID_ARG, "max_tokens >= 1 and 1 <= max_sessions <= %d", k::kScanMax);
  if (!(c.rope_base > 0) || !(c.rms_eps >= 0)) return fail(SPP_E_INVALID_ARG, "rope_base / rms_eps");
  if (c.weight_format != SPP_WFMT_DTYPE && c.weight_format != SPP_WFMT_MXFP4)
    return fail(SPP_E_INVALID_ARG, "unknown weight_format %d", c.weight_format);
  if (c.weight_format == SPP_WFMT_MXFP4 &&
      (!bf16 || c.d_model % 128 || c.ffn_dim % 128 || (c.n_q_heads * c.head_dim) % 128))
    return fail(SPP_E_INVALID_ARG,
                "MXFP4 weights need a bf16 model with d_model, ffn_dim and n_q_heads*head_dim "
                "multiples of 128");
  return SPP_OK;
}

// Rows and columns of projection `which`, and the (N, K) of the launch that streams it
// (the QKV and gate/up matrices are streamed together).
bool projection_dims(const Shape& s, int which, int* rows, int* cols, int* N, int* K) {
  const int nq = s.n_q * s.dh, nkv = s.n_kv * s.dh;
  switch (which) {
    case SPP_W_Q: *rows = nq; *cols = s.d; *N = nq + 2 * nkv; *K = s.d; return true;
    case SPP_W_K:
    case SPP_W_V: *rows = nkv; *cols = s.d; *N = nq + 2 * nkv; *K = s.d; return true;
    case SPP_W_O: *rows = s.d; *cols = nq; *N = s.d; *K = nq; return true;
    case SPP_W_GATE:
    case SPP_W_UP: *rows = s.ffn; *cols = s.d; *N = 2 * s.ffn; *K = s.d; return true;
    case SPP_W_DOWN: *rows = s.d; *cols = s.ffn; *N = s.d; *K = s.ffn; return true;
    default: return false;
  }
}

// Slab of an MXFP4 projection's tiled layout: that of the fused gate/up + SwiGLU for the
// gate and up matrices, that of the split-K projection otherwise.
int fp4_slab(const Shape& s, int which) {
  int rows, cols, N, K;
  projection_dims(s, which, &rows, &cols, &N, &K);
  return which == SPP_W_GATE || which == SPP_W_UP ? k::pack_slab_steps_gateup_fp4(s, s.ffn, s.d)
                                                  : k::pack_slab_steps_fp4(s, N, K);
}

Shape shape_of(const spp_model_config& c) {
  return Shape{c.n_layers, c.d_model, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn_dim, c.vocab,
               c.rms_eps, c.rope_base, c.dtype == SPP_DTYPE_BF16 ? 1 : 0};
}

}  // namespace

extern "C" {

spp_status spp_model_create(const spp_model_config* cfg, const spp_weights* w, spp_model_t* out) {
  if (!cfg || !w || !out) return fail(SPP_E_INVALID_ARG, "null argument");
  *out = nullptr;
  const spp_model_config& c = *cfg;
  const bool bf16 = c.dtype == SPP_DTYPE_BF16;
  if (const spp_status rc = check_config(c); rc != SPP_OK) return rc;
  if (!w->embed || !w->final_norm || !w->lm_head || !w->attn_norm || !w->wq || !w->wk || !w->wv ||
      !w->wo || !w->mlp_norm || !w->w_gate || !w->w_up || !w->w_down)
    return fail(SPP_E_INVALID_ARG, "null weight pointer");
  for (int l = 0; l < c.n_layers; ++l)
    if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] || !w->mlp_norm[l] ||
        !w->w_gate[l] || !w->w_up[l] || !w->w_down[l])
      return fail(SPP_E_INVALID_ARG, "null weight pointer in layer %d", l);

  spp_model_s* m = new spp_model_s();
  m->cfg = c;
  m->s = Shape{c.n_layers, c.d_model, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn_dim, c.vocab,
               c.rms_eps, c.rope_base, bf16 ? 1 : 0};
  m->elem = bf16 ? 2 : 4;
  {
    const Shape& s = m->s;
    const int nq = s.n_q * s.dh, nkv = s.n_kv * s.dh;
    const auto slab_of = c.weight_format == SPP_WFMT_MXFP4 ? k::pack_slab_steps_fp4
                                                            : k::pack_slab_steps;
    m->slab[0] = slab_of(s, nq + 2 * nkv, s.d);
    m->slab[1] = slab_of(s, s.d, nq);
    m->slab[2] = c.weight_format == SPP_WFMT_MXFP4 ? k::pack_slab_steps_gateup_fp4(s, s.ffn, s.d)
                                                   : k::pack_slab_steps_gateup(s, s.ffn, s.d);
    m->slab[3] = slab_of(s, s.d, s.ffn);
    m->slab[4] = k::pack_slab_steps(s, s.vocab, s.d);  // the LM head stays bf16
  }
  hipGetDevice(&m->device);
  {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, m->device) == hipSuccess &&
        cu > 0)
      m->n_cu = cu;
  }
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  m->lm_head = w->lm_head;
  m->lm_bias = w->lm_bias;
  for (int l = 0; l < c.n_layers; ++l) {
    m->attn_norm.push_back(w->attn_norm[l]);
    m->wq.push_back(w->wq[l]);
    m->wk.push_back(w->wk[l]);
    m->wv.push_back(w->wv[l]);
    m->wo.push_back(w->wo[l]);
    m->mlp_norm.push_back(w->mlp_norm[l]);
    m->wg.push_back(w->w_gate[l]);
    m->wu.push_back(w->w_up[l]);
    m->wd.push_back(w->w_down[l]);
  }
  m->fp4 = c.weight_format == SPP_WFMT_MXFP4;
  if (m->fp4) {
    for (int kind = 0; kind < 7; ++kind) {
      if (!w->scales[kind]) {
        spp_model_destroy(m);
        return fail(SPP_E_INVALID_ARG, "null MXFP4 scale array for projection %d", kind);
      }
      for (int l = 0; l < c.n_layers; ++l) {
        if (!w->scales[kind][l]) {
          spp_model_destroy(m);
          return fail(SPP_E_INVALID_ARG, "null MXFP4 scales of projection %d, layer %d", kind, l);
        }
        m->wsc[kind].push_back(w->scales[kind][l]);
      }
    }
  }
  const Shape& s = m->s;
  const int nq = s.n_q * s.dh, nkv = s.n_kv * s.dh;
  const size_t Mx = (size_t)c.max_tokens;
  // split-K partials: the largest of every projection's plan at every row count up to
  // max_tokens (the split count falls with the row count in places, so no single row
  // count bounds the product)
  size_t part_elems = 0;
  for (int M = 1; M <= c.max_tokens; ++M) {
    const int shapes[4][2] = {{nq + 2 * nkv, s.d}, {s.d, nq}, {2 * s.ffn, s.d}, {s.d, s.ffn}};
    for (auto& sh : shapes)
      part_elems = std::max(part_elems, (size_t)(m->fp4 ? k::gemm_plan_fp4 : k::gemm_plan)(
                                                    s, M, sh[0], sh[1]).splits * M * sh[0]);
  }
  m->part_elems = part_elems;
  // batched LM head partials: the largest split count at any session count
  int lm_splits = 1;
  for (int n = 2; n <= c.max_sessions; ++n)
    lm_splits = std::max(lm_splits, k::gemm_plan(s, n, s.vocab, s.d).splits);
  const int sb = k::kScanMaxBlocks;
  bool ok = true;
  auto dmal = [&](void** p, size_t b) {
    if (ok && hipMalloc(p, b) != hipSuccess) ok = false;
  };
  dmal((void**)&m->x, Mx * s.d * 4);
  dmal(&m->h, 2 * Mx * s.d * m->elem);      // hi, lo
  dmal(&m->q, 2 * Mx * nq * m->elem);       // hi, lo
  dmal(&m->att, 2 * Mx * nq * m->elem);     // hi, lo
  dmal(&m->act, 2 * Mx * s.ffn * m->elem);  // hi, lo
  dmal((void**)&m->part, part_elems * 4);
  dmal((void**)&m->ss, Mx * k::res_blocks(s) * 4);
  dmal((void**)&m->range, kMaxSegments * sizeof(uint32_t));
  dmal((void**)&m->rope, Mx * (s.dh / 2) * sizeof(float2));
  dmal(&m->z, 2 * (size_t)k::kScanMax * s.d * m->elem);  // hi, lo
  if (c.max_sessions > 1) {
    dmal((void**)&m->logits_rows, (size_t)lm_splits * c.max_sessions * s.vocab * 4);
    dmal(&m->lm_tiled, (size_t)s.vocab * s.d * m->elem);
    if (ok && k::pack_weight((int)m->elem, w->lm_head, m->lm_tiled, s.vocab, s.d, m->slab[4],
                             nullptr) != hipSuccess)
      ok = false;
  }
  if (!c.weights_packed && m->fp4) {  // keep tiled copies of the MXFP4 codes and scales
    std::vector<const void*>* lists[7] = {&m->wq, &m->wk, &m->wv, &m->wo, &m->wg, &m->wu, &m->wd};
    for (int kind = 0; kind < 7 && ok; ++kind) {
      int rows, cols, N, K;
      projection_dims(s, kind, &rows, &cols, &N, &K);
      const int slab = fp4_slab(s, kind);
      for (int l = 0; l < s.n_layers && ok; ++l) {
        void *cd = nullptr, *sd = nullptr;
        dmal(&cd, (size_t)rows * cols / 2);
        dmal(&sd, (size_t)rows * cols / 32);
        if (!ok) break;
        m->owned.push_back(cd);
        m->owned.push_back(sd);
        if (k::pack_weight_fp4((*lists[kind])[l], m->wsc[kind][l], cd, sd, rows, cols, slab,
                               nullptr) != hipSuccess)
          ok = false;
        (*lists[kind])[l] = cd;
        m->wsc[kind][l] = sd;
      }
    }
  } else if (!c.weights_packed) {  // keep packed copies of the projection weights
    const int rows[9] = {0, nq, nkv, nkv, s.d, 0, s.ffn, s.ffn, s.d};
    const int cols[9] = {0, s.d, s.d, s.d, nq, 0, s.d, s.d, s.ffn};
    const int slab[9] = {0, m->slab[0], m->slab[0], m->slab[0], m->slab[1], 0, m->slab[2],
                         m->slab[2], m->slab[3]};
    std::vector<const void*>* lists[9] = {nullptr, &m->wq, &m->wk, &m->wv, &m->wo, nullptr,
                                          &m->wg, &m->wu, &m->wd};
    for (int kind = 0; kind < 9 && ok; ++kind) {
      if (!lists[kind]) continue;
      for (int l = 0; l < s.n_layers && ok; ++l) {
        void* dst = nullptr;
        dmal(&dst, (size_t)rows[kind] * cols[kind] * m->elem);
        if (!ok) break;
        m->owned.push_back(dst);
        if (k::pack_weight((int)m->elem, (*lists[kind])[l], dst, rows[kind], cols[kind],
                           slab[kind], nullptr) != hipSuccess)
          ok = false;
        (*lists[kind])[l] = dst;
      }
    }
  }
  const size_t lm_parts = std::max((size_t)k::lmhead_blocks(s), (size_t)k::kScanMax * sb);
  dmal((void**)&m->lm_parts, lm_parts * sizeof(ScanPartial));
  dmal((void**)&m->gate_parts, (size_t)k::kScanMax * sb * sizeof(ScanPartial));
  if (ok && hipHostMalloc((void**)&m->gate_host, (k::kScanMax + 1) * sizeof(ScanResult),
                          hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess)
    ok = false;
  if (ok && hipHostGetDevicePointer((void**)&m->gate_dev, m->gate_host, 0) != hipSuccess) ok = false;
  if (ok && hipEventCreateWithFlags(&m->params_free, hipEventDisableTiming) != hipSuccess) ok = false;
  if (ok && hipEventCreateWithFlags(&m->step_done, hipEventDisableTiming) != hipSuccess) ok = false;
  for (int i = 0; i < 2 && ok; ++i)
    if (hipEventCreateWithFlags(&m->chunk_end[i], hipEventDisableTiming) != hipSuccess) ok = false;
  if (ok) memset(m->gate_host, 0, (k::kScanMax + 1) * sizeof(ScanResult));
  if (ok && hipDeviceSynchronize() != hipSuccess) ok = false;
  if (!ok) {
    spp_model_destroy(m);
    return fail(SPP_E_NOMEM, "could not allocate the model work buffers");
  }
  *out = m;
  return SPP_OK;
}

spp_status spp_model_destroy(spp_model_t m) {
  if (!m) return SPP_OK;
  hipDeviceSynchronize();
  void* bufs[] = {m->x, m->h, m->q, m->att, m->act, m->part, m->rope, m->z, m->logits_rows,
                  m->lm_parts, m->gate_parts, m->o_part.p,
                  m->ml_part.p, m->params_dev.p, m->lm_tiled, m->ss, m->range};
  for (void* p : bufs)
    if (p) hipFree(p);
  for (void* p : m->owned) hipFree(p);
  if (m->gate_host) hipHostFree(m->gate_host);
  if (m->params_host) hipHostFree(m->params_host);
  if (m->params_free) hipEventDestroy(m->params_free);
  if (m->step_done) hipEventDestroy(m->step_done);
  for (hipEvent_t e : m->chunk_end)
    if (e) hipEventDestroy(e);
  delete m;
  return SPP_OK;
}

size_t spp_session_kv_bytes(spp_model_t m, int32_t capacity) {
  if (!m || capacity < 1) return 0;
  return layer_elems(*m, (int)round_up(capacity, 64)) * m->s.n_layers * m->elem;
}

spp_status spp_session_kv_layout(spp_model_t m, int32_t capacity, int32_t layer, spp_kv_layout* out) {
  if (!m || !out || capacity < 1 || layer < 0 || layer >= m->s.n_layers)
    return fail(SPP_E_INVALID_ARG, "bad layout query");
  const int64_t cs = round_up(capacity, 64), dh = m->s.dh;
  const int64_t base = (int64_t)layer * layer_elems(*m, (int)cs);
  out->elem_bytes = (int32_t)m->elem;
  out->k_offset = base * m->elem;
  out->k_stride[0] = cs * dh;
  out->k_stride[1] = dh;
  out->k_stride[2] = 1;
  out->v_offset = (base + (int64_t)m->s.n_kv * cs * dh) * m->elem;
  out->v_stride[0] = dh * cs;
  out->v_stride[1] = 1;
  out->v_stride[2] = cs;
  return SPP_OK;
}

spp_status spp_session_create(spp_model_t m, const spp_session_config* cfg, void* kv_dev,
                              size_t kv_bytes, spp_session_t* out) {
  if (!m || !cfg || !kv_dev || !out) return fail(SPP_E_INVALID_ARG, "null argument");
  *out = nullptr;
  if (cfg->capacity < 1 || cfg->capacity > SPP_MAX_CAPACITY || cfg->budget < 0 ||
      cfg->budget > cfg->capacity)
    return fail(SPP_E_INVALID_ARG, "1 <= capacity <= %d and 0 <= budget <= capacity",
                SPP_MAX_CAPACITY);
  if (kv_bytes < spp_session_kv_bytes(m, cfg->capacity))
    return fail(SPP_E_INVALID_ARG, "KV buffer of %zu bytes, need %zu", kv_bytes,
                spp_session_kv_bytes(m, cfg->capacity));
  if (reinterpret_cast<uintptr_t>(kv_dev) % 16) return fail(SPP_E_INVALID_ARG, "KV buffer not 16-byte aligned");
  std::shared_ptr<spp_session_s> sp = std::make_shared<spp_session_s>();
  spp_session_s* s = sp.get();
  s->m = m;
  s->capacity = cfg->capacity;
  s->cap_stride = (int)round_up(cfg->capacity, 64);
  s->budget = cfg->budget ? cfg->budget : cfg->capacity;
  s->kv = kv_dev;
  s->kv_bytes = kv_bytes;
  if (hipEventCreateWithFlags(&s->done, hipEventDisableTiming) != hipSuccess ||
      hipMalloc((void**)&s->summary, sizeof(ScanResult)) != hipSuccess)
    return fail(SPP_E_NOMEM, "session resources");  // (released with sp)
  {
    std::lock_guard<std::mutex> lk(g_reg_mu);
    s->id = g_next_id++;
    g_sessions[s->id] = sp;
  }
  *out = s;
  return SPP_OK;
}

spp_status spp_session_destroy(spp_session_t s) {
  if (!s) return SPP_OK;
  std::shared_ptr<Session> keep;
  {
    std::lock_guard<std::mutex> lk(g_reg_mu);
    auto it = g_sessions.find(s->id);
    if (it == g_sessions.end() || it->second.get() != s)
      return fail(SPP_E_INVALID_ARG, "unknown or already destroyed session");
    keep = std::move(it->second);
    g_sessions.erase(it);
  }
  {
    // a call already inside the session finishes first; one that still holds a
    // reference afterwards finds no valid record (a stale handle falls through)
    std::lock_guard<std::mutex> lk(keep->mu);
    invalidate(*keep);
  }
  keep.reset();  // the session is freed here or by the last call still holding it
  return SPP_OK;
}

int32_t spp_session_id(spp_session_t s) { return s ? s->id : -1; }

spp_status spp_session_restore(spp_session_t s, int32_t n) {
  if (!s || n < 0 || n > s->capacity) return fail(SPP_E_INVALID_ARG, "restore length");
  std::lock_guard<std::mutex> lk(s->mu);
  invalidate(*s);
  s->n_s = n;
  return SPP_OK;
}

spp_status spp_kv_append_delta(spp_session_t s, const int32_t* tokens, int32_t n, void* stream) {
  if (!s || n < 1) return fail(SPP_E_INVALID_ARG, "session and n >= 1 required");
  Model& m = *s->m;
  spp_status rc = check_tokens(m, tokens, n);
  if (rc != SPP_OK) return rc;
  std::lock_guard<std::mutex> lk(s->mu);
  if ((int64_t)s->n_s + n > s->capacity)
    return fail(SPP_E_CAPACITY, "n_s %d + %d exceeds capacity %d", s->n_s, n, s->capacity);
  invalidate(*s);  // drops the speculative entry cells too
  hipSetDevice(m.device);
  std::lock_guard<std::mutex> mk(m.mu);
  for (int off = 0; off < n; off += m.cfg.max_tokens) {
    const int len = std::min(n - off, m.cfg.max_tokens);
    SegReq r{s, tokens + off, len, s->n_s + off, nullptr, nullptr};
    rc = run_step(m, &r, 1, false, static_cast<hipStream_t>(stream), nullptr);
    if (rc != SPP_OK) return rc;
  }
  s->n_s += n;
  return SPP_OK;
}

static spp_status preposition_impl(spp_session_t s, const int32_t* entry, int32_t L, float* dist,
                                   const uint32_t* bitmap, void* stream, spp_ready_t* out,
                                   Prof* prof, YieldCtl* y = nullptr) {
  if (!s || !dist || !out || L < 1) return fail(SPP_E_INVALID_ARG, "null argument or L_entry < 1");
  Model& m = *s->m;
  if (L > m.cfg.max_tokens) return fail(SPP_E_INVALID_ARG, "L_entry %d > max_tokens %d", L, m.cfg.max_tokens);
  spp_status rc = check_tokens(m, entry, L);
  if (rc != SPP_OK) return rc;
  std::lock_guard<std::mutex> lk(s->mu);
  out->session_id = s->id;
  out->reserved = 0;
  // Alg. 1: skip without touching any cell when the entry exceeds the headroom B
  const int B = s->budget - s->n_s;
  if (L > B) {
    invalidate(*s);
    out->epoch = s->epoch;
    return SPP_SKIPPED_BUDGET;
  }
  invalidate(*s);  // the previous ready record (if any) is replaced
  if (y && __atomic_load_n(y->flag, __ATOMIC_ACQUIRE)) {  // a request is already waiting: nothing is enqueued
    out->epoch = s->epoch;
    return SPP_YIELDED;
  }
  hipSetDevice(m.device);
  {
    std::lock_guard<std::mutex> mk(m.mu);
    SegReq r{s, entry, L, s->n_s, dist, bitmap};
    rc = run_step(m, &r, 1, true, static_cast<hipStream_t>(stream), prof, y);
    if (rc != SPP_OK) return rc;
    if (y && y->yielded) {  // the entry cells written so far stay uncommitted
      out->epoch = s->epoch;
      return SPP_YIELDED;
    }
    const hipError_t e = hipEventRecord(s->done, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(SPP_E_HIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  s->entry.assign(entry, entry + L);
  s->position = s->n_s + L;  // decision point, Eq. (decision-point)
  s->dist = dist;
  s->valid = true;
  out->epoch = s->epoch;
  return SPP_OK;
}

spp_status spp_preposition(spp_session_t s, const int32_t* entry, int32_t L, float* dist,
                           const uint32_t* bitmap, void* stream, spp_ready_t* out) {
  return preposition_impl(s, entry, L, dist, bitmap, stream, out, nullptr);
}

spp_status spp_preposition_idle(spp_session_t s, const int32_t* entry, int32_t L, float* dist,
                                const uint32_t* bitmap, const volatile uint32_t* yield_flag,
                                int32_t chunk_layers, void* stream, spp_ready_t* out) {
  if (!yield_flag || chunk_layers < 1) return fail(SPP_E_INVALID_ARG, "null yield flag or chunk_layers < 1");
  YieldCtl y{yield_flag, chunk_layers, false};
  spp_status rc = preposition_impl(s, entry, L, dist, bitmap, stream, out, nullptr, &y);
  if (rc != SPP_OK) return rc;
  // the pass has been enqueued in full: wait for it, still watching nothing (the last
  // chunks and the LM head run to the end; the ready record is already in place)
  const hipError_t e = hipEventSynchronize(s->done);
  if (e != hipSuccess) return fail(SPP_E_HIP, "hipEventSynchronize: %s", hipGetErrorString(e));
  return SPP_OK;
}

// Eq. (fallthrough), Sec. 3.5: the entry cells stay where the pre-position wrote them (the
// constant-time restore) and are committed with the delta; only the delta is processed.
spp_status spp_resume(spp_session_t s, const int32_t* delta, int32_t n, float* dist,
                      const uint32_t* bitmap, void* stream, spp_ready_t* out) {
  if (!s || !dist || !out || n < 1) return fail(SPP_E_INVALID_ARG, "null argument or n < 1");
  Model& m = *s->m;
  spp_status rc = check_tokens(m, delta, n);
  if (rc != SPP_OK) return rc;
  std::lock_guard<std::mutex> lk(s->mu);
  const int live = s->n_s + (int)s->entry.size();
  if ((int64_t)live + n > s->capacity)
    return fail(SPP_E_CAPACITY, "%d live cells + %d exceed capacity %d", live, n, s->capacity);
  invalidate(*s);  // the entry's record is consumed (its cells are kept)
  s->n_s = live;
  hipSetDevice(m.device);
  {
    std::lock_guard<std::mutex> mk(m.mu);
    hipStream_t st = static_cast<hipStream_t>(stream);
    for (int off = 0; off < n; off += m.cfg.max_tokens) {
      const int len = std::min(n - off, m.cfg.max_tokens);
      const bool last = off + len == n;
      SegReq r{s, delta + off, len, s->n_s + off, last ? dist : nullptr, last ? bitmap : nullptr};
      rc = run_step(m, &r, 1, last, st, nullptr);
      if (rc != SPP_OK) {
        s->n_s += off;  // the chunks already written stay committed
        return rc;
      }
    }
    const hipError_t e = hipEventRecord(s->done, st);
    if (e != hipSuccess) return fail(SPP_E_HIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  s->n_s += n;
  s->position = s->n_s;
  s->dist = dist;
  s->valid = true;
  out->session_id = s->id;
  out->reserved = 0;
  out->epoch = s->epoch;
  return SPP_OK;
}

spp_status spp_ready_summary(spp_ready_t ready, spp_summary* out) {
  if (!out) return fail(SPP_E_INVALID_ARG, "null summary");
  const std::shared_ptr<Session> s = lookup(ready.session_id);
  if (!s) return fail(SPP_E_STATE, "no session %d", ready.session_id);
  std::lock_guard<std::mutex> lk(s->mu);
  if (!s->valid || s->epoch != ready.epoch) return fail(SPP_E_STATE, "stale ready handle");
  HIPCHK(hipEventSynchronize(s->done));
  ScanResult r;
  HIPCHK(hipMemcpy(&r, s->summary, sizeof(r), hipMemcpyDeviceToHost));
  fill_summary(r, s->position, out);
  return SPP_OK;
}

spp_status spp_gate(spp_ready_t ready, float tau, const uint32_t* bitmap,
                    const int32_t* realized, int32_t n_realized, void* stream, int32_t* token_out,
                    spp_gate_outcome* outcome, spp_summary* scan_out) {
  if (!token_out || !outcome) return fail(SPP_E_INVALID_ARG, "null output");
  *token_out = -1;
  *outcome = SPP_FALL_INVALID;
  if (!(tau >= 0.f)) return fail(SPP_E_INVALID_ARG, "tau must be >= 0 (got %g)", (double)tau);
  if (realized && n_realized < 0) return fail(SPP_E_INVALID_ARG, "n_realized < 0");
  const std::shared_ptr<Session> s = lookup(ready.session_id);
  if (!s) return SPP_OK;  // unknown session: nothing valid to serve
  std::lock_guard<std::mutex> lk(s->mu);
  // Alg. 2: eligibility first
  if (!s->valid || s->epoch != ready.epoch) return SPP_OK;
  bool done = false;
  if (const spp_status rc = decoded(*s, &done); rc != SPP_OK) return rc;
  if (!done) return SPP_OK;  // not decoded yet: fall through
  if (realized && ((size_t)n_realized != s->entry.size() ||
                   memcmp(realized, s->entry.data(), s->entry.size() * 4) != 0)) {
    *outcome = SPP_FALL_INELIGIBLE;
    return SPP_OK;
  }
  Model& m = *s->m;
  hipSetDevice(m.device);
  std::lock_guard<std::mutex> gk(m.gate_mu);
  const uint32_t seq = ++m.gate_seq;
  k::ScanJob job{};
  job.dist[0] = s->dist;
  job.bitmap[0] = bitmap;
  job.result[0] = m.gate_dev;
  job.parts = m.gate_parts;
  job.flag_src[0] = &s->summary->flags;
  job.done = gate_done_dev(m);
  job.seq = seq;
  job.with_lse = 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e = k::scan(m.s, 1, job, st);
  if (e != hipSuccess) return fail(SPP_E_HIP, "gate scan launch: %s", hipGetErrorString(e));
  spp_status rc = wait_done(m, seq, st);
  if (rc != SPP_OK) return rc;
  const ScanResult r = *const_cast<const ScanResult*>(m.gate_host);
  *outcome = decide(r, tau, token_out);
  if (scan_out) fill_summary(r, s->position, scan_out);
  return SPP_OK;
}

}  // extern "C"

namespace {

// Where a batched gate's scan keeps its partials and results.  kModel: the model's work
// buffers, results published to its pinned, host-mapped block (one wait on the done
// word).  kStatic: the library's static device scratch of this device (results copied
// back on the stream, then the stream is synchronized).
enum class GateScratch { kModel, kStatic };

spp_status gate_batch_impl(int32_t n, const spp_ready_t* ready, const float* taus,
                           const uint32_t* const* bitmaps, hipStream_t st, int32_t* tokens_out,
                           spp_gate_outcome* outcomes, GateScratch where, char* scratch) {
  std::vector<std::shared_ptr<Session>> ss;
  std::vector<Session*> order;
  for (int base = 0; base < n; base += k::kScanMax) {
    const int cnt = std::min(n - base, k::kScanMax);
    // every handle of the chunk resolved under one registry lock
    ss.assign(cnt, nullptr);
    {
      std::lock_guard<std::mutex> lk(g_reg_mu);
      for (int i = 0; i < cnt; ++i) {
        tokens_out[base + i] = -1;
        outcomes[base + i] = SPP_FALL_INVALID;
        auto it = g_sessions.find(ready[base + i].session_id);
        if (it != g_sessions.end()) ss[i] = it->second;
      }
    }
    // lock the distinct sessions in id order (a session may appear more than once)
    order.clear();
    for (const auto& sp : ss)
      if (sp) order.push_back(sp.get());
    std::sort(order.begin(), order.end(), [](Session* a, Session* b) { return a->id < b->id; });
    order.erase(std::unique(order.begin(), order.end()), order.end());
    for (Session* sp : order) sp->mu.lock();
    std::vector<int> scan_of(cnt, -1);
    k::ScanJob job{};
    int ns = 0;
    Model* mp = nullptr;
    spp_status rc = SPP_OK;
    for (int i = 0; i < cnt && rc == SPP_OK; ++i) {
      Session* s = ss[i].get();
      if (!s || !s->valid || s->epoch != ready[base + i].epoch) continue;
      bool done = false;
      rc = decoded(*s, &done);
      if (rc != SPP_OK || !done) continue;
      if (mp && mp != s->m) {
        rc = fail(SPP_E_INVALID_ARG, "handles of different models in one batch");
        break;
      }
      mp = s->m;
      scan_of[i] = ns;
      job.dist[ns] = s->dist;
      job.bitmap[ns] = bitmaps ? bitmaps[base + i] : nullptr;
      job.flag_src[ns] = &s->summary->flags;
      ++ns;
    }
    if (rc == SPP_OK && ns > 0) {
      Model& m = *mp;
      hipSetDevice(m.device);
      ScanResult res[k::kScanMax];
      job.with_lse = 0;
      if (where == GateScratch::kModel) {
        std::lock_guard<std::mutex> gk(m.gate_mu);
        const uint32_t seq = ++m.gate_seq;
        for (int j = 0; j < ns; ++j) job.result[j] = m.gate_dev + j;
        job.parts = m.gate_parts;
        job.done = gate_done_dev(m);
        job.seq = seq;
        const hipError_t e = k::scan(m.s, ns, job, st);
        if (e != hipSuccess) rc = fail(SPP_E_HIP, "gate scan launch: %s", hipGetErrorString(e));
        if (rc == SPP_OK) rc = wait_done(m, seq, st);
        for (int j = 0; j < ns && rc == SPP_OK; ++j) res[j] = *const_cast<const ScanResult*>(m.gate_host + j);
      } else {
        // [kScanMax results][kScanMax * kScanMaxBlocks partials]; the partials of every
        // used block and the results read back are written by the scan itself, so
        // nothing has to start cleared
        ScanResult* rdev = reinterpret_cast<ScanResult*>(scratch);
        for (int j = 0; j < ns; ++j) job.result[j] = rdev + j;
        job.parts = reinterpret_cast<ScanPartial*>(scratch + k::kScanMax * sizeof(ScanResult));
        job.done = nullptr;
        job.seq = 1;
        hipError_t e = k::scan(m.s, ns, job, st);
        if (e == hipSuccess) e = hipMemcpyAsync(res, rdev, ns * sizeof(ScanResult), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) rc = fail(SPP_E_HIP, "gate scan: %s", hipGetErrorString(e));
      }
      for (int i = 0; i < cnt && rc == SPP_OK; ++i)
        if (scan_of[i] >= 0) outcomes[base + i] = decide(res[scan_of[i]], taus[base + i], tokens_out + base + i);
    }
    for (Session* sp : order) sp->mu.unlock();
    if (rc != SPP_OK) return rc;
  }
  return SPP_OK;
}

}  // namespace

// Static scratch of spp_gate_batch_noalloc: the results and first-phase partials of one
// scan of at most kScanMax distributions.  Each device holds its own copy of this array
// for the life of the process; host code takes its address per device through
// hipGetSymbolAddress (the name itself is a host-side stand-in, not a device address).
constexpr size_t kNoallocScratchBytes =
    k::kScanMax * sizeof(ScanResult) + (size_t)k::kScanMax * k::kScanMaxBlocks * sizeof(ScanPartial);
static __device__ __align__(256) char scratch[kNoallocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu[kMaxDevices];   // one no-alloc gate at a time per device
char* g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch` per device (set once)

// The device address of `scratch` on `dev`, resolved on the first call there (with that
// device current).  Caller holds g_scratch_mu[dev].
spp_status scratch_of(int dev, char** out) {
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SPP_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return SPP_OK;
}

spp_status check_gate_batch_args(int32_t n, const spp_ready_t* ready, const float* taus,
                                 int32_t* tokens_out, spp_gate_outcome* outcomes) {
  if (n < 0 || (n > 0 && (!ready || !taus || !tokens_out || !outcomes)))
    return fail(SPP_E_INVALID_ARG, "null argument");
  for (int i = 0; i < n; ++i)
    if (!(taus[i] >= 0.f)) return fail(SPP_E_INVALID_ARG, "tau[%d] must be >= 0", i);
  return SPP_OK;
}

}  // namespace

extern "C" {

spp_status spp_gate_batch(int32_t n, const spp_ready_t* ready, const float* taus,
                          const uint32_t* const* bitmaps, void* stream, int32_t* tokens_out,
                          spp_gate_outcome* outcomes) {
  if (const spp_status rc = check_gate_batch_args(n, ready, taus, tokens_out, outcomes); rc != SPP_OK)
    return rc;
  return gate_batch_impl(n, ready, taus, bitmaps, static_cast<hipStream_t>(stream), tokens_out,
                         outcomes, GateScratch::kModel, nullptr);
}

spp_status spp_gate_batch_noalloc(int32_t n, const spp_ready_t* ready, const float* taus,
                                  const uint32_t* const* bitmaps, void* stream,
                                  int32_t* tokens_out, spp_gate_outcome* outcomes) {
  // the count first: a call beyond the limit is rejected before its arrays are read
  if (n > k::kScanMax)
    return fail(SPP_E_INVALID_ARG,
                "spp_gate_batch_noalloc takes at most %d handles per call (got %d): its static "
                "scratch holds one scan of %d distributions",
                k::kScanMax, n, k::kScanMax);
  if (const spp_status rc = check_gate_batch_args(n, ready, taus, tokens_out, outcomes); rc != SPP_OK)
    return rc;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(SPP_E_HIP, "no usable current device");
  std::lock_guard<std::mutex> lk(g_scratch_mu[dev]);
  char* scr = nullptr;
  if (const spp_status rc = scratch_of(dev, &scr); rc != SPP_OK) return rc;
  // the handles' model must live on this device, whose copy of the scratch the scan uses
  for (int i = 0; i < n; ++i) {
    const std::shared_ptr<Session> s = lookup(ready[i].session_id);
    if (s && s->m->device != dev)
      return fail(SPP_E_INVALID_ARG, "handle %d belongs to device %d, current device is %d", i,
                  s->m->device, dev);
  }
  return gate_batch_impl(n, ready, taus, bitmaps, static_cast<hipStream_t>(stream), tokens_out,
                         outcomes, GateScratch::kStatic, scr);
}

spp_status spp_invalidate_on_mutation(spp_session_t s, spp_mutation kind, int32_t arg) {
  if (!s) return fail(SPP_E_INVALID_ARG, "null session");
  if (kind != SPP_MUT_SHIFT && kind != SPP_MUT_ROLLBACK && kind != SPP_MUT_UPDATE)
    return fail(SPP_E_INVALID_ARG, "unknown mutation %d", (int)kind);
  if (kind == SPP_MUT_ROLLBACK && arg < 0) return fail(SPP_E_INVALID_ARG, "rollback length < 0");
  std::lock_guard<std::mutex> lk(s->mu);
  invalidate(*s);
  if (kind == SPP_MUT_ROLLBACK) s->n_s = std::min(s->n_s, (int)arg);
  return SPP_OK;
}

spp_status spp_shift(spp_session_t s, int32_t delta, void* stream) {
  if (!s) return fail(SPP_E_INVALID_ARG, "null session");
  Model& m = *s->m;
  std::lock_guard<std::mutex> lk(s->mu);
  if (delta < 1 || delta > s->n_s)
    return fail(SPP_E_INVALID_ARG, "shift by %d outside [1, n_s = %d]", delta, s->n_s);
  invalidate(*s);  // Sec. 3.6: in the same call as the mutation (drops the entry cells too)
  const int n_new = s->n_s - delta;
  hipSetDevice(m.device);
  {
    std::lock_guard<std::mutex> mk(m.mu);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    // ordered after the model's last step on whatever stream it ran, and before the next
    if (m.step_recorded) HIPCHK(hipStreamWaitEvent(st, m.step_done, 0));
    const hipError_t e = k::shift_cells(m.s, s->kv, s->cap_stride, n_new, delta, st);
    if (e != hipSuccess) return fail(SPP_E_HIP, "shift: %s", hipGetErrorString(e));
    HIPCHK(hipEventRecord(m.step_done, st));
    m.step_recorded = true;
  }
  s->n_s = n_new;
  return SPP_OK;
}

// Wilson score interval of k successes in n trials at normal quantile z.
static void wilson(int64_t k, int64_t n, double z, double* lo, double* hi) {
  if (n <= 0) {
    *lo = 0.0;
    *hi = 1.0;
    return;
  }
  const double p = (double)k / n, z2 = z * z;
  const double den = 1.0 + z2 / n;
  const double mid = (p + z2 / (2.0 * n)) / den;
  const double half = z / den * std::sqrt(p * (1.0 - p) / n + z2 / (4.0 * n * (double)n));
  *lo = std::max(0.0, mid - half);
  *hi = std::min(1.0, mid + half);
}

spp_status spp_gate_calibrate(int32_t n, const float* gaps, const uint8_t* in_set,
                              const uint8_t* correct, double r_max, double z, int32_t n_taus,
                              const float* taus, spp_gate_point* curve, int32_t curve_cap,
                              int32_t* n_points, float* tau_star) {
  if (n < 1 || !gaps || !in_set || !correct || !n_points || !tau_star || (n_taus > 0 && !taus) ||
      n_taus < 0 || !(r_max >= 0.0) || !(z > 0.0))
    return fail(SPP_E_INVALID_ARG, "bad calibration arguments");
  // candidate thresholds: the given ones, or 0 and every distinct nonnegative gap (the
  // accepted set, hence coverage and risk, changes only where tau crosses a gap)
  std::vector<float> cand;
  if (n_taus > 0) {
    for (int i = 0; i < n_taus; ++i) {
      if (!(taus[i] >= 0.0f)) return fail(SPP_E_INVALID_ARG, "tau %d is negative or NaN", i);
      cand.push_back(taus[i]);
    }
  } else {
    cand.push_back(0.0f);
    for (int i = 0; i < n; ++i)
      if (gaps[i] >= 0.0f) cand.push_back(gaps[i]);  // NaN gaps never qualify
  }
  std::sort(cand.begin(), cand.end());
  cand.erase(std::unique(cand.begin(), cand.end()), cand.end());
  if (curve && curve_cap < (int)cand.size())
    return fail(SPP_E_INVALID_ARG, "curve holds %d points, %zu needed", curve_cap, cand.size());
  *n_points = (int32_t)cand.size();
  *tau_star = INFINITY;
  for (size_t c = 0; c < cand.size(); ++c) {
    const float tau = cand[c];
    int64_t served = 0, wrong = 0;
    for (int i = 0; i < n; ++i)
      if (gaps[i] > tau && in_set[i]) {  // Eq. (gate): strictly above tau, argmax in the set
        ++served;
        if (!correct[i]) ++wrong;
      }
    const double risk = served ? (double)wrong / served : NAN;  // undefined with none served
    if (curve) {
      spp_gate_point& pt = curve[c];
      pt.tau = tau;
      pt.served = (int32_t)served;
      pt.wrong = (int32_t)wrong;
      pt.coverage = (double)served / n;
      pt.risk = risk;
      wilson(served, n, z, &pt.coverage_lo, &pt.coverage_hi);
      wilson(wrong, served, z, &pt.risk_lo, &pt.risk_hi);
    }
    // the smallest threshold whose risk is within the budget (coverage is largest there)
    if (served && risk <= r_max && *tau_star == INFINITY) *tau_star = tau;
  }
  return SPP_OK;
}

spp_status spp_session_info(spp_session_t s, spp_session_info_t* out) {
  if (!s || !out) return fail(SPP_E_INVALID_ARG, "null argument");
  std::lock_guard<std::mutex> lk(s->mu);
  out->n_committed = s->n_s;
  out->used_cells = s->n_s + (int)s->entry.size();
  out->capacity = s->capacity;
  out->budget = s->budget;
  out->position = s->position;
  out->valid = s->valid ? 1 : 0;
  bool done = false;
  if (s->valid && decoded(*s, &done) != SPP_OK) done = false;
  out->decoded = done ? 1 : 0;
  out->entry_len = (int)s->entry.size();
  out->epoch = s->epoch;
  return SPP_OK;
}

spp_status spp_session_info_get(spp_session_t s, spp_session_info_t* out) {
  return spp_session_info(s, out);
}

}  // extern "C"

static spp_status preposition_batch_impl(int32_t n, const spp_session_t* sessions,
                                         const int32_t* const* entries, const int32_t* lengths,
                                         float* const* dists, void* stream,
                                         spp_ready_t* out_ready, spp_status* out_status,
                                         Prof* prof) {
  if (n < 1 || !sessions || !entries || !lengths || !dists || !out_ready || !out_status)
    return fail(SPP_E_INVALID_ARG, "null argument or n < 1");
  Model* mp = sessions[0] ? sessions[0]->m : nullptr;
  if (!mp) return fail(SPP_E_INVALID_ARG, "null session");
  Model& m = *mp;
  std::vector<std::pair<int, Session*>> order;
  for (int i = 0; i < n; ++i) {
    Session* s = sessions[i];
    if (!s || s->m != mp) return fail(SPP_E_INVALID_ARG, "session %d null or of another model", i);
    if (!dists[i] || lengths[i] < 1 || lengths[i] > m.cfg.max_tokens)
      return fail(SPP_E_INVALID_ARG, "entry %d: null dist or length outside [1, max_tokens]", i);
    spp_status rc = check_tokens(m, entries[i], lengths[i]);
    if (rc != SPP_OK) return rc;
    order.push_back({s->id, s});
  }
  std::sort(order.begin(), order.end());
  for (size_t i = 1; i < order.size(); ++i)
    if (order[i].first == order[i - 1].first) return fail(SPP_E_INVALID_ARG, "a session appears twice");
  for (auto& p : order) p.second->mu.lock();
  spp_status rc = SPP_OK;
  std::vector<SegReq> reqs;
  std::vector<int> req_of;
  for (int i = 0; i < n; ++i) {
    Session* s = sessions[i];
    out_ready[i].session_id = s->id;
    out_ready[i].reserved = 0;
    invalidate(*s);
    out_ready[i].epoch = s->epoch;
    if (lengths[i] > s->budget - s->n_s) {
      out_status[i] = SPP_SKIPPED_BUDGET;
      continue;
    }
    out_status[i] = SPP_OK;
    reqs.push_back(SegReq{s, entries[i], lengths[i], s->n_s, dists[i], nullptr});
    req_of.push_back(i);
  }
  hipSetDevice(m.device);
  hipStream_t st = static_cast<hipStream_t>(stream);
  {
    std::lock_guard<std::mutex> mk(m.mu);
    size_t b = 0;
    while (b < reqs.size() && rc == SPP_OK) {  // passes of <= max_tokens rows, <= max_sessions segments
      size_t e = b;
      int rows = 0;
      const int per_pass = std::min(k::kScanMax, m.cfg.max_sessions);
      while (e < reqs.size() && (int)(e - b) < per_pass && rows + reqs[e].len <= m.cfg.max_tokens)
        rows += reqs[e++].len;
      rc = run_step(m, reqs.data() + b, (int)(e - b), true, st, prof);
      b = e;
    }
  }
  for (size_t j = 0; j < reqs.size() && rc == SPP_OK; ++j) {
    Session* s = reqs[j].s;
    if (hipEventRecord(s->done, st) != hipSuccess) {
      rc = fail(SPP_E_HIP, "hipEventRecord failed");
      break;
    }
    s->entry.assign(reqs[j].tok, reqs[j].tok + reqs[j].len);
    s->position = s->n_s + reqs[j].len;
    s->dist = reqs[j].dist;
    s->valid = true;
  }
  for (auto& p : order) p.second->mu.unlock();
  return rc;
}

extern "C" {

spp_status spp_preposition_batch(int32_t n, const spp_session_t* sessions,
                                 const int32_t* const* entries, const int32_t* lengths,
                                 float* const* dists, void* stream, spp_ready_t* out_ready,
                                 spp_status* out_status) {
  return preposition_batch_impl(n, sessions, entries, lengths, dists, stream, out_ready, out_status,
                                nullptr);
}

// Sums the recorded kernel times per class (after the stream has finished).
static void collect_profile(const Prof& prof, int32_t n_classes, float* times_us, int32_t* counts) {
  for (int k = 0; k < n_classes; ++k) {
    times_us[k] = 0.f;
    counts[k] = 0;
  }
  for (size_t i = 0; i < prof.used; ++i) {
    const int c = prof.cls[i];
    float ms = 0.f;
    if (c >= 0 && c < n_classes && hipEventElapsedTime(&ms, prof.start[i], prof.stop[i]) == hipSuccess) {
      times_us[c] += ms * 1000.f;
      counts[c] += 1;
    }
  }
}

int32_t spp_profile_preposition_batch(int32_t n, const spp_session_t* sessions,
                                      const int32_t* const* entries, const int32_t* lengths,
                                      float* const* dists, void* stream, spp_ready_t* out_ready,
                                      spp_status* out_status, int32_t n_classes, float* times_us,
                                      int32_t* counts) {
  if (!times_us || !counts || n_classes < 1) {
    fail(SPP_E_INVALID_ARG, "null argument");
    return -1;
  }
  Prof prof;
  launch_recorder = &prof;
  const spp_status rc = preposition_batch_impl(n, sessions, entries, lengths, dists, stream,
                                               out_ready, out_status, &prof);
  launch_recorder = nullptr;
  hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (rc == SPP_OK) collect_profile(prof, n_classes, times_us, counts);
  for (hipEvent_t e : prof.start) hipEventDestroy(e);
  for (hipEvent_t e : prof.stop) hipEventDestroy(e);
  return rc == SPP_OK ? KC_COUNT : -1;
}

int32_t spp_profile_preposition(spp_session_t s, const int32_t* entry, int32_t L, float* dist,
                                void* stream, int32_t n_classes, float* times_us, int32_t* counts) {
  if (!s || !times_us || !counts || n_classes < 1) {
    fail(SPP_E_INVALID_ARG, "null argument");
    return -1;
  }
  Prof prof;
  auto release = [&prof] {
    for (hipEvent_t e : prof.start) hipEventDestroy(e);
    for (hipEvent_t e : prof.stop) hipEventDestroy(e);
  };
  spp_ready_t r;
  launch_recorder = &prof;
  const spp_status rc = preposition_impl(s, entry, L, dist, nullptr, stream, &r, &prof);
  launch_recorder = nullptr;
  if (rc != SPP_OK) {
    hipStreamSynchronize(static_cast<hipStream_t>(stream));
    release();
    if (rc == SPP_SKIPPED_BUDGET)  // not an error of the pass itself: say why nothing ran
      fail(SPP_E_STATE, "profiling pass skipped: the entry exceeds the session's headroom");
    return -1;
  }
  hipStreamSynchronize(static_cast<hipStream_t>(stream));
  collect_profile(prof, n_classes, times_us, counts);
  release();
  return KC_COUNT;
}

const char* spp_kernel_class_name(int32_t k) {
  static const char* names[KC_COUNT] = {"embed_norm", "gemm_qkv", "qkv_epilogue", "attention",
                                        "attention_combine", "gemm_o", "residual_norm",
                                        "gemm_gate_up", "swiglu", "gemm_down", "lm_head", "scan"};
  return (k >= 0 && k < KC_COUNT) ? names[k] : "";
}

spp_status spp_pack_weight_mxfp4(const spp_model_config* cfg, int32_t which,
                                 const void* codes_src, const void* scales_src, void* codes_dst,
                                 void* scales_dst, void* stream) {
  if (!cfg || !codes_src || !scales_src || !codes_dst || !scales_dst)
    return fail(SPP_E_INVALID_ARG, "null pointer");
  if (const spp_status rc = check_config(*cfg); rc != SPP_OK) return rc;
  if (cfg->weight_format != SPP_WFMT_MXFP4)
    return fail(SPP_E_INVALID_ARG, "spp_pack_weight_mxfp4 needs weight_format SPP_WFMT_MXFP4");
  const Shape s = shape_of(*cfg);
  int rows, cols, N, K;
  if (!projection_dims(s, which, &rows, &cols, &N, &K))
    return fail(SPP_E_INVALID_ARG, "unknown projection weight %d", which);
  const hipError_t e = k::pack_weight_fp4(codes_src, scales_src, codes_dst, scales_dst, rows, cols,
                                          fp4_slab(s, which), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SPP_E_HIP, "pack: %s", hipGetErrorString(e));
  return SPP_OK;
}

spp_status spp_pack_weight(const spp_model_config* cfg, int32_t which, const void* src, void* dst,
                           void* stream) {
  if (!cfg || !src || !dst) return fail(SPP_E_INVALID_ARG, "null pointer");
  if (const spp_status rc = check_config(*cfg); rc != SPP_OK) return rc;
  if (cfg->weight_format != SPP_WFMT_DTYPE)
    return fail(SPP_E_INVALID_ARG, "MXFP4 weights are packed by spp_pack_weight_mxfp4");
  const spp_model_config& c = *cfg;
  const Shape s{c.n_layers, c.d_model, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn_dim, c.vocab,
                c.rms_eps, c.rope_base, c.dtype == SPP_DTYPE_BF16 ? 1 : 0};
  const int nq = s.n_q * s.dh, nkv = s.n_kv * s.dh;
  int rows, cols, slab;
  switch (which) {
    case SPP_W_Q: rows = nq; cols = s.d; slab = k::pack_slab_steps(s, nq + 2 * nkv, s.d); break;
    case SPP_W_K:
    case SPP_W_V: rows = nkv; cols = s.d; slab = k::pack_slab_steps(s, nq + 2 * nkv, s.d); break;
    case SPP_W_O: rows = s.d; cols = nq; slab = k::pack_slab_steps(s, s.d, nq); break;
    case SPP_W_GATE:
    case SPP_W_UP: rows = s.ffn; cols = s.d; slab = k::pack_slab_steps_gateup(s, s.ffn, s.d); break;
    case SPP_W_DOWN: rows = s.d; cols = s.ffn; slab = k::pack_slab_steps(s, s.d, s.ffn); break;
    default: return fail(SPP_E_INVALID_ARG, "unknown projection weight %d", which);
  }
  const hipError_t e = k::pack_weight(s.bf16 ? 2 : 4, src, dst, rows, cols, slab,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SPP_E_HIP, "pack: %s", hipGetErrorString(e));
  return SPP_OK;
}

spp_status spp_copy_reference(void* dst, const void* src, size_t n, void* stream) {
  if (!dst || !src) return fail(SPP_E_INVALID_ARG, "null pointer");
  const hipError_t e = k::copy_bytes(dst, src, n, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SPP_E_HIP, "copy: %s", hipGetErrorString(e));
  return SPP_OK;
}

}  // extern "C"
