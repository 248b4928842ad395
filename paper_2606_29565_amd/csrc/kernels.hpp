// Internal interface between the host runtime and the gfx950 kernels.
//
// One pre-position (or committed delta) step processes a PACKED batch of rows:
// the new tokens of one or more sessions ("segments"), each appended at its own
// live end.  Every row carries its token id and absolute position; every
// segment carries its session's KV buffer.  The host fills a StepParams record
// per step and copies it to the device; the kernels read it from there, through a
// StepView of its arrays' device addresses resolved on the host (a kernel argument, so
// the first load of a kernel is the entry it needs, not an offset to it).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

namespace spp {

// Dispatch timing.  While a recorder with a class set is installed on the calling thread,
// every kernel of a step is launched with a start and a stop event carried by its own
// dispatch (hipExtLaunchKernelGGL): the time between the two is the kernel's execution on
// the device, without the launch gap that events recorded around the launch would add.
struct LaunchRecorder {
  std::vector<hipEvent_t> start, stop;
  std::vector<int> cls;
  size_t used = 0;  // event pairs handed out
  int cur = -1;     // class of the launches being issued; -1 records nothing
};
extern thread_local LaunchRecorder* launch_recorder;
// Hands out the next event pair of the installed recorder (creating it on first use);
// false when nothing is to be recorded.
bool recorder_events(hipEvent_t* start, hipEvent_t* stop);

#define SPP_LAUNCH(kern, grid, block, shm, st, ...)                                  \
  do {                                                                               \
    hipEvent_t ev_a_, ev_b_;                                                         \
    if (::spp::recorder_events(&ev_a_, &ev_b_))                                      \
      hipExtLaunchKernelGGL(kern, grid, block, shm, st, ev_a_, ev_b_, 0, __VA_ARGS__); \
    else                                                                             \
      hipLaunchKernelGGL(kern, grid, block, shm, st, __VA_ARGS__);                   \
  } while (0)

constexpr int kMaxSegments = 256;
// Value a step's per-segment range word takes when the fp16 attention of a bf16 model
// meets a scaled query or a K/V cell of magnitude above 65504 (the largest finite fp16):
// the segment's distribution is then flagged (ScanResult flag bit 2) and never served.
constexpr uint32_t kRangeFlag = 4u;
constexpr float kF16Max = 65504.f;
constexpr int kAttnWaves = 8;                 // waves per attention work item
constexpr int kAttnRows = 16 * kAttnWaves;    // query rows per attention work item (fp32)
constexpr int kAttnRowsH = 256;               // query rows per work item of bf16 models
constexpr int kAttnTile = 128;                // keys staged in LDS per iteration
constexpr int kAttnSub = 64;                  // keys per matrix-core pass over a stage

struct Segment {
  void* kv;          // session KV buffer: per layer K [Hkv][cap][dh] then V^T [Hkv][dh][cap]
  int32_t cap;       // cells per layer
  int32_t n_past;    // committed cells before this step (n_s)
  int32_t row0;      // first packed row of the segment
  int32_t len;       // rows (tokens) of the segment
};

// One attention work item: query rows [rowgrp*RG, +RG) of the segment's (token,
// head-in-group) rows of kv head `kvh` (RG = attn_rows: 256 for bf16 models, 128 for
// fp32), against keys [k0, k1) (k0 a multiple of kAttnSub); the causal limit of each row
// cuts the range further.  `solo`: the item is its row group's only one (bf16 models then
// write the attention output directly, with no key-range merge).
// Items and groups carry a copy of their segment, so that one load gives a kernel all
// it needs to start.
struct AttnItem {
  Segment sg;
  int32_t seg, kvh, rowgrp, k0, k1, solo;
};

// Items of one (segment, kv head, row group) are consecutive, chunk 0 first.  The merge's
// work list holds every group of an fp32 model and, for a bf16 model, the groups of more
// than one item (a single item writes the attention output itself).
struct AttnGroup {
  Segment sg;
  int32_t seg, kvh, rowgrp;
  int32_t first_item, n_items;
};

// One packed row: its session's KV buffer and cells per layer, its absolute position and
// its segment.
struct RowInfo {
  void* kv;
  int32_t cap, pos, seg, pad;
};

struct StepParams {
  int32_t n_rows, n_segments, n_items, n_groups;
  Segment seg[kMaxSegments];
  // variable-length arrays follow in the same allocation (offsets in bytes from the
  // start of the record): int32 token[n_rows], RowInfo row[n_rows], AttnItem
  // item[n_items], AttnGroup group[n_groups]
  int64_t off_token, off_row, off_item, off_group;
};

// Device addresses of one step record and its arrays.
struct StepView {
  const StepParams* p;
  const int32_t* token;
  const RowInfo* row;
  const AttnItem* item;
  const AttnGroup* group;
};

// The view of a record at device address `dev` whose host copy is `host`.
inline StepView step_view(const StepParams* dev, const StepParams* host) {
  const char* b = reinterpret_cast<const char*>(dev);
  return StepView{dev, reinterpret_cast<const int32_t*>(b + host->off_token),
                  reinterpret_cast<const RowInfo*>(b + host->off_row),
                  reinterpret_cast<const AttnItem*>(b + host->off_item),
                  reinterpret_cast<const AttnGroup*>(b + host->off_group)};
}

struct Shape {
  int32_t n_layers, d, n_q, n_kv, dh, ffn, vocab;
  float eps;
  double rope_base;
  int32_t bf16;
};

// Query rows per attention row group of a model.
inline int attn_rows(const Shape& s) { return s.bf16 ? kAttnRowsH : kAttnRows; }

// Up to three weight matrices concatenated along the output dimension:
// output column n in [nbeg[i], nbeg[i+1]) is row (n - nbeg[i]) of mat[i].  The matrices
// are in the tiled layout with `slab` K-steps per slab (see pack_weight).
// MXFP4 matrices (gemm_fp4) also carry their tiled e8m0 scales in `scale`.
struct WeightCat {
  const void* mat[3];
  int32_t nbeg[4];
  int32_t slab;
  const void* scale[3];
};

// Result of a reduction over one distribution (32 bytes).
struct ScanResult {
  int32_t argmax, second;
  float top1, top2, lse;
  uint32_t flags;    // bit 0 nonfinite, bit 1 argmax in the bitmap, bit 2 the fp16
                     // attention saw an input beyond its range (see kRangeFlag)
  uint32_t seq;      // sequence number written last (host polling)
  uint32_t pad;
};

static_assert(sizeof(ScanResult) == 32, "results are stored as two 16-byte halves");

// Per-workgroup partial of a scan.
struct ScanPartial {
  float v1, v2;
  int32_t i1, i2;
  float m, s;        // running max and sum of exp(x - m) over finite values
  uint32_t nonfinite;
  uint32_t pad;
};

// Kernel classes (for per-class device timing).
enum KernelClass {
  KC_EMBED = 0, KC_GEMM_QKV, KC_QKV_EPI, KC_ATTN, KC_ATTN_COMBINE, KC_GEMM_O, KC_RESID_NORM,
  KC_GEMM_GATEUP, KC_SWIGLU, KC_GEMM_DOWN, KC_LMHEAD, KC_SCAN, KC_COUNT
};

namespace k {

// Matrix-core inputs (h, attention output, SwiGLU output, final-norm rows) are written
// as a (hi, lo) pair of arrays in bf16 models (lo = bf16 rounding remainder; the GEMM
// multiplies both); fp32 models use hi alone.

// RMSNorm is factored: (RMSNorm(x) * g) W = inv * ((x * g) W), inv[r] = 1/sqrt(mean(x[r]^2)
// + eps).  Producers of x write y = x * g (the projection input) and ss[r][b], the sums of
// squares of row r over its res_blocks(s) 1024-column blocks; consumers of the split sums
// scale row r by inv[r].
int res_blocks(const Shape& s);

// x[r] = E[token[r]], y[r] = x[r] * g, ss; rope table rows (cos, sin).
// range[0 .. n_segments) is cleared (the step's fp16 range words, see kRangeFlag).
hipError_t embed(const Shape& s, const StepView& v, int n_rows, const void* embed, const void* g,
                 float* x, void* y, void* y_lo, float* ss, float2* rope, uint32_t* range,
                 hipStream_t st);

// Launch shape of one projection GEMM: NW waves x CB column blocks of 16 per workgroup,
// slices of STEPS K-steps, ITERS pipelined slices per workgroup, MT 16-row tiles.
// A workgroup covers STEPS * ITERS K-steps.  row_tiles = 0: each workgroup runs every
// row in passes of 16*MT; row_tiles > 0 (many rows): each workgroup runs one tile of
// 16*MT rows, the tiles of one (split, column group) dealt to one XCD in turn.
struct GemmPlan {
  int nw, steps, iters, mt, splits, cb;
  int row_tiles;
};
GemmPlan gemm_plan(const Shape& s, int M, int N, int K);

// K-steps per slab of the tiled layout of a projection with N outputs (all its
// matrices together) and K inputs: the K-range one workgroup covers at M = 32, so that
// at every moment the workgroups of that launch read one compact window.
int pack_slab_steps(const Shape& s, int N, int K);

// partials[split][M][N] = X[M][K] (row-major, ld = K) times W^T over the K-range of
// `split`; W are up to three TILED matrices (see pack_weight) concatenated along N.
hipError_t gemm(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                const WeightCat& w, int N, float* partials, hipStream_t st);

// The MLP gate/up projection with the SwiGLU fused: act[r][f] = silu(inv g) * (inv u) from
// the gate (w.mat[0]) and up (w.mat[1]) matrices of F rows each (w.nbeg = {0, F, 2F, ...}),
// inv = the row's 1/RMS from ss.  gemm_plan_swiglu returns splits = 0 where the fused
// variant does not apply (then gemm + swiglu).  pack_slab_steps_gateup is the slab of the
// gate and up matrices' tiled layout.
GemmPlan gemm_plan_swiglu(const Shape& s, int M, int F, int K);
hipError_t gemm_swiglu(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M,
                       int K, const WeightCat& w, int F, const float* ss, void* act, void* act_lo,
                       hipStream_t st);
int pack_slab_steps_gateup(const Shape& s, int F, int K);

// Rearranges a row-major [N][K] matrix into the tiled layout the GEMM streams.  Blocks
// of 16 rows x one 128-byte K-step (2 KB: two 1 KB fragments in lane order) are ordered
// time-major: block (row block cb, K-step ks) goes to position
//   ((ks % slab) * (KS / slab) + ks / slab) * (N / 16) + cb,   KS = K-steps per row,
// so the workgroups of a launch whose K-range is `slab` steps, all at their t-th step,
// read adjacent blocks.  slab divides KS.
hipError_t pack_weight(int elem_bytes, const void* src, void* dst, int N, int K, int slab,
                       hipStream_t st);

// MXFP4 projections (4-bit e2m1 weights, one e8m0 scale per 32 along K; bf16 models):
// the same partials as gemm() from the tiled codes and scales of pack_weight_fp4.  K is
// a multiple of 128 (one step); `slab` counts steps.
GemmPlan gemm_plan_fp4(const Shape& s, int M, int N, int K);
int pack_slab_steps_fp4(const Shape& s, int N, int K);
hipError_t gemm_fp4(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M, int K,
                    const WeightCat& w, int N, float* partials, hipStream_t st);
// The fused gate/up + SwiGLU over MXFP4 gate and up matrices (as gemm_swiglu).
GemmPlan gemm_plan_swiglu_fp4(const Shape& s, int M, int F, int K);
hipError_t gemm_swiglu_fp4(const Shape& s, const GemmPlan& p, const void* X, const void* Xlo, int M,
                           int K, const WeightCat& w, int F, const float* ss, void* act,
                           void* act_lo, hipStream_t st);
int pack_slab_steps_gateup_fp4(const Shape& s, int F, int K);
// Row-major codes [N][K/2] (even k in the low nibble) and scales [N][K/32] into the tiled
// layout: per 16 rows x 128 columns a 1 KB code block (lane order of the MFMA B
// fragments) and a 64-byte scale block, ordered time-major with `slab` steps per slab.
hipError_t pack_weight_fp4(const void* codes_src, const void* scales_src, void* codes_dst,
                           void* scales_dst, int N, int K, int slab, hipStream_t st);

// Split-K sums of the QKV projection times inv[r] (ss of its input rows), RoPE, q out
// (scaled for the base-2 softmax), K and V appended to the sessions' caches.  bf16
// models: a scaled query beyond the fp16 range sets range[segment] = kRangeFlag.
hipError_t qkv_epilogue(const Shape& s, const StepView& v, int n_rows, int layer,
                        const float* partials, int splits, const float* ss, const float2* rope,
                        void* q_out, void* q_lo, uint32_t* range, hipStream_t st);

// Delta attention over the step's work items.  Partials per item and row: the output
// (bf16 models: normalized by its own sum, fp16 [items][256][dh]; fp32 models: the
// unnormalized fp32 sum [items][128][dh]) and (max, sum) in ml_part.  bf16 models: an
// item alone in its row group writes the output (hi, lo) to out / out_lo directly, and a
// K/V cell beyond the fp16 range sets range[segment] = kRangeFlag.
hipError_t attention(const Shape& s, const StepView& v, int n_items, int layer, const void* q,
                     const void* q_lo, void* o_part, float2* ml_part, void* out, void* out_lo,
                     uint32_t* range, hipStream_t st);
// Merges the key ranges of every row group with more than one item into out / out_lo.
hipError_t attention_combine(const Shape& s, const StepView& v, int n_groups,
                             const void* o_part, const float2* ml_part, void* out, void* out_lo,
                             hipStream_t st);

// x[r] += sum_split partials; if g: y[r] = x[r] * g; ss of the new x.
hipError_t residual(const Shape& s, int n_rows, const float* partials, int splits, float* x,
                    const void* g, void* y, void* y_lo, float* ss, hipStream_t st);
// act = silu(inv * gate) * (inv * up) from the gate/up split sums (ss of their input rows).
hipError_t swiglu(const Shape& s, int n_rows, const float* partials, int splits, const float* ss,
                  void* act, void* act_lo, hipStream_t st);

// LM head for one row with the fused vocabulary reductions (GEMV).
// range (nullable): the step's range word of the row's segment, ORed into the flags.
hipError_t lmhead_gemv(const Shape& s, const float* x_row, const void* g_final, const void* w_lm,
                       const float* bias, float* dist, const uint32_t* bitmap,
                       ScanPartial* parts, ScanResult* result, const uint32_t* range,
                       hipStream_t st);
int lmhead_blocks(const Shape& s);

// Final norm of the rows `rows` of x into z (model dtype), for the batched LM head.
hipError_t final_norm_rows(const Shape& s, const StepView& v, int n_segs, const float* x,
                           const void* g_final, void* z, void* z_lo, hipStream_t st);

// Scan of n distributions: top-2, optional log-sum-exp, bitmap bit of the argmax.  With
// `src`: dist[b][v] = sum_split src[split][b][v] + bias[v] is formed first.
constexpr int kScanMax = 64;        // distributions per scan launch
constexpr int kScanMaxBlocks = 64;  // first-phase blocks per distribution
struct ScanJob {
  float* dist[kScanMax];
  const uint32_t* bitmap[kScanMax];  // entries may be null (empty set)
  ScanResult* result[kScanMax];      // may point into host-mapped memory
  const float* src;            // optional [src_splits][n][V] partial logits: summed,
  int src_splits;              //   plus the bias, then written to dist[b]
  const float* bias;           // optional [V]
  ScanPartial* parts;          // [n][scan_blocks(V, n)]
  const uint32_t* flag_src[kScanMax];  // optional words: their bit 2 is ORed into the flags
  uint32_t* done;              // optional: receives seq once every result is visible
  uint32_t seq;
  int with_lse;
};
hipError_t scan(const Shape& s, int n, const ScanJob& job, hipStream_t st);
int scan_blocks(int vocab, int n);

// Sliding-window shift of a session's cells (every layer): cells [delta, delta + n_new)
// move to [0, n_new), keys turned back by delta positions (RoPE), values unchanged.
hipError_t shift_cells(const Shape& s, void* kv, int64_t cap, int n_new, int delta,
                       hipStream_t st);

hipError_t copy_bytes(void* dst, const void* src, size_t n, hipStream_t st);

}  // namespace k
}  // namespace spp
