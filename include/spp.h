/* spp.h -- speculative pre-positioning on one MI355X (gfx950): the C ABI.
 *
 * A stateful session keeps a persistent KV cache of n_s committed tokens
 * (Sec. 2 of the paper).  In the idle window after a state update the caller
 * runs a PRE-POSITION step (Alg. 1): the entry tokens (query prefix plus
 * assistant header, or a post-tool-call envelope) are appended at the live end
 * n_s and one forward pass runs over the entry only, against the resident
 * cells.  The logits at the last entry token -- the decision point
 * p = n_s + L_entry of Eq. (decision-point) -- are the READY DISTRIBUTION
 * (Sec. 2.1, Sec. 3.3).  When a request arrives, the GATE (Alg. 2, Eq. (gate))
 * scans that cached distribution: it serves the argmax token iff the top-1 to
 * top-2 logit gap (Eq. (gap)) is strictly greater than tau and the token is in
 * the fast-answer set; otherwise the request falls through.  Any mutation of
 * the state invalidates the cached distribution in the same call (Sec. 3.6).
 *
 * Conventions for every entry point:
 *   - Return value: spp_status.  0 = SPP_OK, > 0 = an informational outcome,
 *     < 0 = an error; spp_last_error() then describes it (thread-local string).
 *     No C++ exception crosses this boundary.
 *   - Device memory holding weights, KV cells, distributions and fast-answer
 *     bitmaps is allocated and owned by the caller and must outlive every model
 *     and session that points at it.  The library owns its own work buffers
 *     (allocated at model creation) and the opaque model / session objects.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Device work is
 *     enqueued on it in order; calls marked "asynchronous" return before the
 *     device finishes.
 *   - Matrices are row-major.  A projection weight W of a layer y = x W^T is
 *     stored [out_features][in_features].  Element type is the model dtype:
 *     SPP_DTYPE_BF16 (16-bit bf16 patterns) or SPP_DTYPE_F32.
 *   - One thread at a time per session for mutating calls; spp_gate may run
 *     concurrently with a pending pre-position of the same session.
 */
#ifndef SPP_H
#define SPP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPP_OK = 0,
  SPP_SKIPPED_BUDGET = 1,   /* Alg. 1: L_entry > cell-budget headroom B; nothing touched  */
  SPP_YIELDED = 2,          /* Sec. 3.1: an idle-window pass gave way to a request       */
  SPP_E_INVALID_ARG = -1,   /* null pointer, bad size, token outside [0, vocab), tau < 0 */
  SPP_E_CAPACITY = -2,      /* committed tokens would exceed the session's KV capacity  */
  SPP_E_HIP = -3,           /* a HIP runtime call failed                                 */
  SPP_E_STATE = -4,         /* call not allowed in the current state                     */
  SPP_E_NOMEM = -5          /* the library could not allocate its work buffers          */
} spp_status;

/* Alg. 2 outcomes.  The paper's "fall through" is split by its cause. */
typedef enum {
  SPP_SERVED = 0,           /* gate fired: *token_out is the cached argmax                */
  SPP_FALL_INVALID = 1,     /* no valid ready distribution, stale handle, or not decoded */
  SPP_FALL_INELIGIBLE = 2,  /* realized entry differs from the pre-positioned entry      */
  SPP_FALL_GAP = 3,         /* gap <= tau                                                */
  SPP_FALL_NOT_IN_SET = 4,  /* argmax not in the fast-answer set                         */
  SPP_FALL_NONFINITE = 5    /* the distribution holds NaN or +-inf (never served)        */
} spp_gate_outcome;

/* State mutations of Sec. 3.6. */
typedef enum {
  SPP_MUT_SHIFT = 0,        /* sliding-window shift done by the caller: invalidates only
                               (spp_shift relocates the cells itself)                    */
  SPP_MUT_ROLLBACK = 1,     /* discard committed tokens: n_s <- min(arg, n_s)            */
  SPP_MUT_UPDATE = 2        /* a fresh update was committed elsewhere: invalidate only   */
} spp_mutation;

typedef enum { SPP_DTYPE_F32 = 0, SPP_DTYPE_BF16 = 1 } spp_dtype;

/* Storage of the projection weights wq..w_down.  MXFP4 is the OCP microscaling format
 * (the 4-bit weight-only variant of the 70B-class headline model, Sec. 4): every weight
 * is a 4-bit e2m1 code (bit 3 sign, bits 2..1 exponent, bit 0 mantissa: magnitudes
 * 0, 0.5, 1, 1.5, 2, 3, 4, 6), and every 32 consecutive weights of a row share one
 * 8-bit e8m0 scale E, w = 2^(E - 127) * e2m1(code), E in [1, 254].  Row-major storage:
 * codes [rows][cols/2] bytes with the even column in the low nibble, scales
 * [rows][cols/32] bytes.  Activations, KV cells, embedding and LM head stay bf16. */
typedef enum { SPP_WFMT_DTYPE = 0, SPP_WFMT_MXFP4 = 1 } spp_weight_format;

typedef struct spp_model_s* spp_model_t;
typedef struct spp_session_s* spp_session_t;

/* Decoder shape.  Pre-norm decoder: RMSNorm (rms_eps), rotate-half RoPE
 * (rope_base), grouped-query attention where q head h reads kv head
 * h / (n_q_heads / n_kv_heads), SwiGLU MLP, untied LM head with optional bias. */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rms_eps;
  double rope_base;
  int32_t dtype;            /* spp_dtype of weights, KV cells and matrix-core operands  */
  int32_t max_tokens;       /* most tokens one call processes (sizes the work buffers)  */
  int32_t max_sessions;     /* most sessions one batched call covers (1..64)            */
  int32_t weights_packed;   /* 1: wq..w_down are already in the tiled layout written by
                               spp_pack_weight; 0: they are row-major and the library keeps
                               tiled copies (it does not read the caller's projection
                               weights after spp_model_create returns)                    */
  int32_t weight_format;    /* spp_weight_format of wq..w_down (MXFP4: bf16 models only)  */
} spp_model_config;

/* Device pointers to the weights (caller-owned).  The per-layer members are HOST
 * arrays of n_layers device pointers; the library copies the arrays.  The projection
 * weights wq..w_down are row-major or tiled (spp_model_config.weights_packed); the
 * embedding, norms and LM head are always row-major. */
typedef struct {
  const void* embed;                 /* [vocab][d_model]                               */
  const void* final_norm;            /* [d_model]                                      */
  const void* lm_head;               /* [vocab][d_model]                               */
  const float* lm_bias;              /* [vocab] fp32, or NULL for no bias              */
  const void* const* attn_norm;      /* [d_model]                                      */
  const void* const* wq;             /* [n_q_heads*head_dim][d_model]                  */
  const void* const* wk;             /* [n_kv_heads*head_dim][d_model]                 */
  const void* const* wv;             /* [n_kv_heads*head_dim][d_model]                 */
  const void* const* wo;             /* [d_model][n_q_heads*head_dim]                  */
  const void* const* mlp_norm;       /* [d_model]                                      */
  const void* const* w_gate;         /* [ffn_dim][d_model]                             */
  const void* const* w_up;           /* [ffn_dim][d_model]                             */
  const void* const* w_down;         /* [d_model][ffn_dim]                             */
  /* MXFP4 models only (else ignored): scales[kind], kind an spp_weight_kind, is a HOST
   * array of n_layers device pointers to that projection's e8m0 scales -- row-major
   * [rows][cols/32] bytes, or tiled by spp_pack_weight_mxfp4 when weights_packed = 1.
   * The projection members above then point at the 4-bit codes. */
  const void* const* scales[7];
} spp_weights;

typedef struct {
  int32_t capacity;         /* KV cells the caller's buffer holds per layer              */
  int32_t budget;           /* the session's cell budget (0 = capacity): pre-positions
                               need L_entry <= budget - n_s (Alg. 1's headroom B)         */
} spp_session_config;

/* Where cell (head, position, dim) of layer `layer` lives inside a session's KV
 * buffer: byte offset of K element = k_offset + (head*k_stride[0] +
 * position*k_stride[1] + dim*k_stride[2]) * elem_bytes, likewise for V. */
typedef struct {
  int64_t k_offset, v_offset;        /* bytes                                          */
  int64_t k_stride[3], v_stride[3];  /* elements, for (head, position, dim)            */
  int32_t elem_bytes;
} spp_kv_layout;

/* Handle to a ready distribution: a value, nothing to free.  It names the
 * session and the epoch of the pre-position; once any mutation (or a newer
 * pre-position) bumps the session's epoch, the handle is stale and the gate
 * returns SPP_FALL_INVALID (Sec. 3.6: a stale answer is never served). */
typedef struct {
  int32_t session_id;
  int32_t reserved;
  uint64_t epoch;
} spp_ready_t;

/* The reductions over a ready distribution (Eq. (gap)): argmax (ties -> lowest
 * index), the two largest logits (a duplicated maximum gives gap 0), the gap,
 * log-sum-exp (NaN when any logit is NaN or +-inf), and the flags.
 *
 * Flag bit 2 (bf16 models): the forward pass met an attention input outside the range
 * of fp16, in which the attention of bf16 models multiplies -- a query scaled by
 * log2(e)/sqrt(head_dim), or a K or V cell, of magnitude above 65504.  Precondition of
 * the bf16 path: every K/V cell and every scaled query stays within +-65504 (magnitudes
 * below 2^-14 are kept to fp16's absolute resolution, 2^-24).  A flagged distribution
 * is never served: the gate answers SPP_FALL_NONFINITE. */
typedef struct {
  int32_t argmax;
  float top1, top2, gap, lse;
  int32_t position;         /* decision point p = n_s + L_entry                         */
  uint32_t flags;           /* bit 0: nonfinite logits; bit 1: argmax in the default set;
                               bit 2: an attention input beyond the fp16 range          */
} spp_summary;

/* The fields Alg. 1 records on the session (decision-point position, a decoded flag and
 * a validity flag for the cached distribution), with the cell accounting behind its
 * budget check and the epoch that invalidation bumps (Sec. 3.6). */
typedef struct {
  int32_t n_committed;      /* n_s                                                      */
  int32_t used_cells;       /* n_s + entry cells of the current pre-position            */
  int32_t capacity, budget;
  int32_t position;         /* last recorded decision point (-1 = none)                 */
  int32_t valid;            /* 1 while the ready distribution is current               */
  int32_t decoded;          /* 1 once the pre-position's device work has finished      */
  int32_t entry_len;
  uint64_t epoch;
} spp_session_info_t;

/* ---- models ---------------------------------------------------------------------- */

/* The target model whose single forward pass over the entry is Alg. 1's Forward(E) (the
 * paper's engine serves one decoder on one accelerator, Sec. 4; its architecture is not
 * given there and follows spp_model_config).
 * Validates the shape (head_dim 64 or 128 for bf16, 64 for fp32; n_q_heads a multiple of
 * n_kv_heads; d_model, ffn_dim and n_q_heads*head_dim multiples of 64 (bf16) or 32
 * (fp32); d_model a width the LM-head kernel covers: ceil(d_model / 512) (bf16) or
 * ceil(d_model / 256) (fp32) in {1, 2, 4, 8, 10, 16}; with MXFP4 weights also d_model,
 * ffn_dim and n_q_heads*head_dim multiples of 128), copies the weight pointers and
 * allocates the work buffers on the current HIP device.  SPP_E_INVALID_ARG on a bad
 * shape or null pointer. */
spp_status spp_model_create(const spp_model_config* cfg, const spp_weights* weights,
                            spp_model_t* out);
spp_status spp_model_destroy(spp_model_t model);

/* Which projection weight of a layer spp_pack_weight rearranges; the shape follows
 * from the model configuration. */
typedef enum {
  SPP_W_Q = 0,     /* [n_q_heads*head_dim][d_model]  */
  SPP_W_K = 1,     /* [n_kv_heads*head_dim][d_model] */
  SPP_W_V = 2,     /* [n_kv_heads*head_dim][d_model] */
  SPP_W_O = 3,     /* [d_model][n_q_heads*head_dim]  */
  SPP_W_GATE = 4,  /* [ffn_dim][d_model]             */
  SPP_W_UP = 5,    /* [ffn_dim][d_model]             */
  SPP_W_DOWN = 6   /* [d_model][ffn_dim]             */
} spp_weight_kind;

/* Rearranges one row-major projection weight of a model with configuration `cfg`
 * (device memory, model dtype) into the tiled layout the projection kernels stream:
 * every 16 rows x 128 bytes of columns become one 2 KB block in the order a 64-lane
 * wave loads it, and the blocks are ordered so that the workgroups of a projection
 * launch read adjacent blocks at the same moment (the order depends on the projection
 * and the configuration, hence both arguments).  src and dst are distinct device
 * buffers of rows*cols elements.  The result is what spp_model_create expects with
 * weights_packed = 1 for the same configuration.  Asynchronous on `stream`.
 * SPP_E_INVALID_ARG for a bad configuration, unknown `which` or null pointer. */
spp_status spp_pack_weight(const spp_model_config* cfg, int32_t which, const void* src, void* dst,
                           void* stream);

/* MXFP4 counterpart of spp_pack_weight: rearranges one projection's row-major codes
 * ([rows][cols/2] bytes) and scales ([rows][cols/32] bytes) into the tiled layout of the
 * 4-bit projection kernels: per 16 rows x 128 columns, a 1 KB code block in the order
 * the 64 lanes of a wave feed the matrix cores and a 64-byte scale block, ordered like
 * the bf16 tiles.  cfg->weight_format must be SPP_WFMT_MXFP4 and cols a multiple of 128.
 * Destinations are distinct device buffers of the same sizes as the sources.
 * Asynchronous on `stream`.  SPP_E_INVALID_ARG for a bad configuration, unknown `which`
 * or null pointer. */
spp_status spp_pack_weight_mxfp4(const spp_model_config* cfg, int32_t which,
                                 const void* codes_src, const void* scales_src, void* codes_dst,
                                 void* scales_dst, void* stream);

/* ---- sessions -------------------------------------------------------------------- */

/* Largest KV capacity of a session in cells per layer (2^24 - 64: the attention kernels
 * address one kv head's keys and values with 32-bit byte offsets). */
#define SPP_MAX_CAPACITY (16777216 - 64)

/* Bytes of device memory a session of `capacity` cells needs for its KV buffer. */
size_t spp_session_kv_bytes(spp_model_t model, int32_t capacity);
spp_status spp_session_kv_layout(spp_model_t model, int32_t capacity, int32_t layer,
                                 spp_kv_layout* out);

/* A stateful session (Sec. 2: one persistent KV cache of n_s accumulated tokens that
 * survives across requests and advances incrementally) over a caller-owned KV buffer of
 * kv_bytes >= spp_session_kv_bytes(), 16-byte aligned, laid out as
 * spp_session_kv_layout describes.  cfg->capacity is the cells per layer the buffer
 * holds, at most SPP_MAX_CAPACITY; cfg->budget (0 = capacity) bounds n_s plus the entry
 * of a pre-position, the cell budget of Alg. 1.  Starts with n_s = 0 and no ready
 * distribution.  SPP_E_INVALID_ARG on a null pointer, capacity outside
 * [1, SPP_MAX_CAPACITY], budget outside [0, capacity], a short or misaligned buffer; SPP_E_NOMEM if the session's small device record cannot
 * be allocated.  The session is named by a process-unique id (spp_session_id), which
 * ready handles carry. */
spp_status spp_session_create(spp_model_t model, const spp_session_config* cfg, void* kv_dev,
                              size_t kv_bytes, spp_session_t* out);
/* Removes the session from the id registry and invalidates its record: a gate still
 * holding a handle of it falls through as SPP_FALL_INVALID; a gate or summary already
 * inside the session finishes first, and the session's resources are released when the
 * last such call returns.  SPP_E_INVALID_ARG for a session destroyed before. */
spp_status spp_session_destroy(spp_session_t session);
int32_t spp_session_id(spp_session_t session);

/* Metadata-only restore (the paper's constant-time T_restore): declare that cells
 * [0, n_tokens) of every layer already hold committed state the caller wrote (see
 * spp_session_kv_layout).  Invalidates any ready distribution. */
spp_status spp_session_restore(spp_session_t session, int32_t n_tokens);

/* Commit a delta (a data batch, a tool result): drops the speculative entry cells,
 * invalidates the ready distribution (Sec. 3.6), then appends `n` tokens (host
 * array) at n_s with one forward pass and advances n_s.  Asynchronous.
 * SPP_E_CAPACITY if n_s + n > capacity; SPP_E_INVALID_ARG on a token outside
 * [0, vocab) or n outside [1, max_tokens]. */
spp_status spp_kv_append_delta(spp_session_t session, const int32_t* tokens, int32_t n,
                               void* stream);

/* Alg. 1.  If L_entry > B (B = budget - n_s): invalidates, touches no cell and
 * returns SPP_SKIPPED_BUDGET.  Otherwise appends the entry (host array) at n_s, runs
 * one forward pass over it, writes the fp32 logits of the last entry token to
 * dist_dev[vocab] (caller-owned device memory), records p = n_s + L_entry, bumps
 * the epoch, marks the session valid, and returns the handle in *out.  The entry
 * cells stay speculative (n_s does not move).  `default_bitmap_dev` (nullable,
 * ceil(vocab/32) words, bit t&31 of word t>>5) sets summary flag bit 1.
 * Asynchronous: the gate treats the distribution as not decoded until the device
 * work has finished. */
spp_status spp_preposition(spp_session_t session, const int32_t* entry, int32_t L_entry,
                           float* dist_dev, const uint32_t* default_bitmap_dev, void* stream,
                           spp_ready_t* out);

/* The idle-window pre-position (Sec. 3.1: speculative work runs only while the session
 * is idle and gives way at once to an arriving request; Alg. 1).  Computes what
 * spp_preposition computes, but enqueues the forward pass in chunks of `chunk_layers`
 * layers, at most two chunks ahead of the device, and reads *yield_flag (caller-owned
 * host memory; a serving thread sets it nonzero when a request arrives) before each
 * chunk.  Blocking: returns when the pass has finished (SPP_OK: the ready record is in
 * place and decoded) or, once the flag is seen set, when the chunks already enqueued
 * have drained (SPP_YIELDED: nothing more was enqueued, no logits were made, the
 * session has no ready record and n_s is unchanged; the entry cells written so far are
 * uncommitted).  A flag already set at the call yields before any device work.  The
 * wait after a set flag is bounded by two chunks of layers (plus the LM head if the
 * last chunk was already enqueued).  Stream priorities are not used: the yield is the
 * library's own.  While the pass runs it holds the model's step lock, so a forward pass
 * of any session of the same model (resume, append, another pre-position) waits for it:
 * a serving thread sets the flag first, then makes its call.  Gates of other sessions
 * do not wait; a gate of this session waits for the yield and then falls through as
 * SPP_FALL_INVALID.  Budget, argument errors and the handle as in
 * spp_preposition; SPP_E_INVALID_ARG for a null flag or chunk_layers < 1. */
spp_status spp_preposition_idle(spp_session_t session, const int32_t* entry, int32_t L_entry,
                                float* dist_dev, const uint32_t* default_bitmap_dev,
                                const volatile uint32_t* yield_flag, int32_t chunk_layers,
                                void* stream, spp_ready_t* out);

/* Fall-through resume (Eq. (fallthrough); Sec. 3.5): the arriving request extends the
 * pre-positioned entry by `delta` (n >= 1 tokens, host array).  The entry's cells stay
 * where the pre-position wrote them (the constant-time restore) and are committed
 * together with the delta: n_s <- n_s + L_entry + n.  Forward passes over the delta
 * alone (max_tokens rows each) write its cells, and the last one writes the fp32 logits
 * at the new end to dist_dev[vocab], recorded as the session's new ready state (position
 * n_s, epoch bumped, so earlier handles go stale; entry_len 0, so only the relaxed gate
 * with realized = NULL can serve it).  With no entry present (never pre-positioned,
 * skipped, or dropped by a mutation) the delta is appended after the committed cells,
 * which is the cold path.  A one-token delta is one decode step.  Unlike a pre-position,
 * a resume is on the critical path: it is bounded by the session's capacity, not by its
 * idle-window budget, and SPP_E_CAPACITY (nothing changed) if the cells do not fit.
 * Asynchronous on `stream`; default_bitmap_dev as in spp_preposition. */
spp_status spp_resume(spp_session_t session, const int32_t* delta, int32_t n, float* dist_dev,
                      const uint32_t* default_bitmap_dev, void* stream, spp_ready_t* out);

/* The reductions the LM head computed over the ready distribution of `ready` (Eq. (gap):
 * argmax, top-1 and top-2 logits, their gap; Sec. 3.3: under the gate the cache may
 * hold only the argmax and the gap), with the log-sum-exp and the flags.  Blocks until
 * the pre-position behind `ready` has finished.  SPP_E_STATE if the handle is stale or
 * its session is gone; SPP_E_INVALID_ARG for a null `out`. */
spp_status spp_ready_summary(spp_ready_t ready, spp_summary* out);

/* Alg. 2.  Checks, in this order: handle current and session valid and device work
 * finished (else SPP_FALL_INVALID); the realized entry (host array, NULL = relaxed
 * streaming mode of Sec. 3.4) equal to the pre-positioned entry (else
 * SPP_FALL_INELIGIBLE).  Then one scan of the cached distribution on `stream`
 * computes the argmax, the two largest logits and the set bit; the call waits for
 * it and decides: nonfinite -> SPP_FALL_NONFINITE; gap > tau is false ->
 * SPP_FALL_GAP; argmax not in the set (fast_bitmap_dev, device, ceil(vocab/32)
 * words; NULL = empty set) -> SPP_FALL_NOT_IN_SET; else SPP_SERVED with
 * *token_out = argmax (otherwise *token_out = -1).  Synchronous.  Read-only: the
 * distribution keeps serving repeated requests.  SPP_E_INVALID_ARG for tau < 0 or
 * NaN.  `scan_out` (nullable) receives the scan's summary. */
spp_status spp_gate(spp_ready_t ready, float tau, const uint32_t* fast_bitmap_dev,
                    const int32_t* realized_entry, int32_t n_realized, void* stream,
                    int32_t* token_out, spp_gate_outcome* outcome, spp_summary* scan_out);

/* Sec. 3.6: clears the valid and decoded flags and bumps the epoch in the same call
 * as the mutation.  SPP_MUT_ROLLBACK sets n_s <- min(arg, n_s) (arg >= 0). */
spp_status spp_invalidate_on_mutation(spp_session_t session, spp_mutation kind, int32_t arg);

/* Sliding-window shift (Sec. 3.6, the mutation that relocates positions): drops the
 * oldest `delta` committed cells and moves the others down by delta positions in every
 * layer -- cell p goes to p - delta, its key turned back by delta positions (rotate-half
 * RoPE: the pair (k_i, k_{i+dh/2}) rotated by the angle -delta * rope_base^(-2i/dh)),
 * its value unchanged -- so n_s <- n_s - delta.  Invalidates the ready distribution and
 * drops the speculative entry in the same call.  Asynchronous on `stream`, ordered after
 * the session's earlier device work.  SPP_E_INVALID_ARG unless 1 <= delta <= n_s (then
 * nothing changes). */
spp_status spp_shift(spp_session_t session, int32_t delta, void* stream);

/* The fields of spp_session_info_t (Alg. 1's recorded position, decoded and valid
 * flags; the cell accounting; the epoch).  Reading `decoded` queries the device work's
 * completion, nothing else.  SPP_E_INVALID_ARG on a null pointer. */
spp_status spp_session_info(spp_session_t session, spp_session_info_t* out);
/* The same call under its earlier name. */
spp_status spp_session_info_get(spp_session_t session, spp_session_info_t* out);

/* ---- batched (many sessions of one model in one pass) ------------------------------ */

/* Alg. 1 for `n` sessions at once: the entries are packed into one pass so every
 * weight is read once for all of them.  Arrays of length n: sessions, entries (host
 * arrays), lengths, dists (device fp32[vocab] each).  Per-session results go to
 * out_status[i] (SPP_OK or SPP_SKIPPED_BUDGET) and out_ready[i].  A pass packs at most
 * the model's max_sessions entries (and max_tokens rows); more sessions take further
 * passes.  The return value is an error if any argument is invalid (then nothing ran):
 * a null pointer, a session of another model or listed twice, a length outside
 * [1, max_tokens], a token outside [0, vocab).  Asynchronous. */
spp_status spp_preposition_batch(int32_t n, const spp_session_t* sessions,
                                 const int32_t* const* entries, const int32_t* lengths,
                                 float* const* dists, void* stream, spp_ready_t* out_ready,
                                 spp_status* out_status);

/* Alg. 2 for n handles, as spp_gate in the relaxed mode (no realized entry): one scan
 * launch per 64 handles, one wait for all of them.  bitmaps (nullable) holds a device
 * bitmap or NULL per handle; taus[i] >= 0.  tokens_out[i] and outcomes[i] as in
 * spp_gate.  Handles of one call belong to one model.  Synchronous. */
spp_status spp_gate_batch(int32_t n, const spp_ready_t* ready, const float* taus,
                          const uint32_t* const* bitmaps, void* stream, int32_t* tokens_out,
                          spp_gate_outcome* outcomes);

/* For callers that cannot allocate memory -- code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation: spp_gate_batch with the scan's partials and
 * results in a static device array of the library (about 130 KB, one copy per device for
 * the life of the process) instead of the model's buffers.  Allocates nothing: no
 * hipMalloc, hipFree or allocating library call.  The results come back through one
 * device-to-host copy on `stream`, which is then synchronized.  At most 64 handles per
 * call (SPP_E_INVALID_ARG beyond, nothing run), all of models on the current device.
 * Outcomes and tokens as spp_gate_batch.  Every call on a device shares that device's
 * array: the library serializes such calls per device (a call waits for the previous
 * one's results), so overlapping calls do not race; nothing in the array has to start
 * cleared, since each call writes every partial and result it reads. */
spp_status spp_gate_batch_noalloc(int32_t n, const spp_ready_t* ready, const float* taus,
                                  const uint32_t* const* bitmaps, void* stream,
                                  int32_t* tokens_out, spp_gate_outcome* outcomes);

/* ---- gate calibration ------------------------------------------------------------- */

/* One threshold of the gate's risk-coverage curve (Sec. 2.4, Eqs. (coverage), (risk)):
 * `served` of the n decision points pass the gate (gap > tau and argmax in the set),
 * `wrong` of those disagree with the full-path output; coverage = served / n, risk =
 * wrong / served (NaN when nothing is served); Wilson score intervals for both. */
typedef struct {
  float tau;
  int32_t served, wrong;
  double coverage, coverage_lo, coverage_hi;
  double risk, risk_lo, risk_hi;
} spp_gate_point;

/* Host-side calibration of the gate threshold from n measured decision points (Sec. 2.4:
 * the smallest tau with r(tau) <= r_max, which maximizes coverage at bounded risk).
 * gaps[i]: the top-1 minus top-2 logit gap of decision point i's ready distribution;
 * in_set[i]: 1 if its argmax is in the fast-answer set; correct[i]: 1 if that argmax
 * equals the model's full-path output for the request.  Candidate thresholds are the
 * n_taus values in `taus` (each >= 0), or with n_taus = 0 every distinct gap >= 0 plus
 * 0 (coverage and risk change only where tau crosses a gap).  curve (nullable, curve_cap
 * points) receives the curve in ascending tau, *n_points its length; *tau_star the
 * smallest candidate with at least one point served and risk <= r_max, or +inf if none
 * qualifies (then the gate should not fire).  z: the normal quantile of the intervals
 * (1.959964 for 95%).  No device work.  SPP_E_INVALID_ARG on null pointers, n < 1, a
 * negative or NaN tau, r_max < 0, z <= 0, or a curve too short for the candidates. */
spp_status spp_gate_calibrate(int32_t n, const float* gaps, const uint8_t* in_set,
                              const uint8_t* correct, double r_max, double z, int32_t n_taus,
                              const float* taus, spp_gate_point* curve, int32_t curve_cap,
                              int32_t* n_points, float* tau_star);

/* ---- diagnostics ------------------------------------------------------------------- */

const char* spp_last_error(void);

/* Device time of the kernels of one pre-position step, measured with a start and a
 * stop HIP event carried by each kernel's own dispatch on `stream` (the kernel's
 * execution, without the launch gaps between kernels; a profiling run: it performs a
 * real pre-position with the same effects as spp_preposition, then waits).
 * times_us[k] receives the summed time of kernel class k over the step and counts[k]
 * its kernel launches, for k < n_classes (see spp_kernel_class_name).  Returns the
 * number of classes, or -1 on error (spp_last_error; an entry beyond the session's
 * headroom, which spp_preposition answers with SPP_SKIPPED_BUDGET, is an error here). */
int32_t spp_profile_preposition(spp_session_t session, const int32_t* entry, int32_t L_entry,
                                float* dist_dev, void* stream, int32_t n_classes,
                                float* times_us, int32_t* counts);
const char* spp_kernel_class_name(int32_t k);

/* spp_preposition_batch measured the same way: the same effects, then a wait; times_us[k]
 * and counts[k] summed over every pass of the batch.  Returns the number of classes, or
 * -1 on error (spp_last_error). */
int32_t spp_profile_preposition_batch(int32_t n, const spp_session_t* sessions,
                                      const int32_t* const* entries, const int32_t* lengths,
                                      float* const* dists, void* stream, spp_ready_t* out_ready,
                                      spp_status* out_status, int32_t n_classes, float* times_us,
                                      int32_t* counts);

/* Plain device copy of n bytes (both device pointers): the traffic reference the
 * HBM counters are calibrated against.  Asynchronous. */
spp_status spp_copy_reference(void* dst, const void* src, size_t n, void* stream);

#ifdef __cplusplus
}
#endif
#endif
