/* CPU oracle for the pre-position step and the confidence gate.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call
 * this code; it exists so that tests, the smoke check and the bench's CPU
 * baseline can compare the HIP path against a plain, slow, obviously correct
 * definition.  It shares no code, header, table or constant with the HIP path.
 *
 * Arithmetic is fp64 throughout (the paper fixes no precision).  Weights and
 * KV cells arrive as float arrays holding exactly the stored values (fp32, or
 * bf16 widened); KV cells written by the oracle are rounded to the cache
 * format, because the cache format is part of the session state.
 *
 * What is computed (speculative pre-positioning, Sec. 2.1 and 3.2):
 * the pre-position step is one forward pass of the decoder over the entry
 * tokens only, appended at the session's live end n_s (Alg. 1, "Append(E) at
 * end position n_s" and "Forward(E)"), against the resident KV cells; the
 * ready distribution is the logit vector at the last entry token, the
 * decision point p = n_s + L_entry of Eq. (decision-point).  The decoder itself
 * is not described by the paper: it is the standard pre-norm decoder of the
 * workloads (RMSNorm, rotate-half RoPE, grouped-query attention with
 * contiguous head groups, SwiGLU MLP, untied LM head with an optional bias).
 */
#ifndef SPP_ORACLE_H
#define SPP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t d_model, n_q, n_kv, head_dim, ffn, vocab;
  double eps, rope_base;
  int32_t cache_bf16; /* 1: KV cells stored as bf16, 0: as fp32 */
} orc_shape;

typedef struct {
  const float *attn_norm, *wq, *wk, *wv, *wo, *mlp_norm, *wg, *wu, *wd;
} orc_layer_weights;

typedef struct {
  int32_t argmax;      /* index of the largest logit; ties -> lowest index      */
  int32_t second;      /* index of the runner-up under the same order           */
  double top1, top2;   /* l(1), l(2): the two largest values (duplicates count) */
  double gap;          /* gamma = l(1) - l(2), Eq. (gap)                         */
  double lse;          /* log sum exp of the logits (NaN when nonfinite)         */
  int32_t nonfinite;   /* any NaN or +-inf among the logits                      */
} orc_summary;

/* Decoder pieces.  x, h: [M][d] row-major.  W: [N][K] row-major (y = x W^T). */
void orc_rmsnorm(int M, int d, const double* x, const float* g, double eps, double* out);
void orc_linear(int M, int N, int K, const double* x, const float* W, double* y);
void orc_rope(int M, int H, int dh, double* u, int64_t pos0, double base);
void orc_attention(int M, int Hq, int Hkv, int dh, const double* q, const float* Kc,
                   const float* Vc, int64_t cap, int64_t n_past, double* out);
void orc_swiglu(int M, int F, const double* gate, const double* up, double* out);
double orc_round_bf16(double v);
void orc_embed(int M, int d, const int32_t* tokens, const float* E, double* x);

/* One decoder layer over M tokens at positions n_past .. n_past+M-1.  Writes their
 * K and V cells into Kc/Vc ([n_kv][cap][head_dim]) and updates x in place. */
int orc_layer(const orc_shape* s, const orc_layer_weights* w, float* Kc, float* Vc,
              int64_t cap, int64_t n_past, int M, double* x);

/* orc_layer for a final layer whose later use reads the last row only: every row's K
 * and V cells are appended, the rest runs for row M-1 alone (same arithmetic). */
int orc_layer_last(const orc_shape* s, const orc_layer_weights* w, float* Kc, float* Vc,
                   int64_t cap, int64_t n_past, int M, double* x);

/* Ready distribution at the last row: RMSNorm(x_last) g_f W_lm^T + bias (bias may be NULL). */
void orc_logits(const orc_shape* s, const double* x_last, const float* g_final,
                const float* w_lm, const float* bias, double* logits);

/* Sliding-window shift of the cells of one layer: cells [delta, n_s) move to
 * [0, n_s - delta), keys turned back by delta positions (RoPE at position -delta, then
 * rounded to the cache format), values unchanged.  Returns nonzero on bad arguments. */
int orc_shift_cells(int n_kv, int64_t cap, int dh, float* Kc, float* Vc, int64_t n_s,
                    int64_t delta, double rope_base, int cache_bf16);

/* Top-2 by a full sort (value descending, index ascending; NaN last), log-sum-exp. */
void orc_summary_of(int V, const double* logits, orc_summary* out);

/* Gate outcome, Alg. 2 with Eq. (gate):
 *   0 SERVED, 1 FALL_INVALID, 2 FALL_INELIGIBLE, 3 FALL_GAP, 4 FALL_NOT_IN_SET,
 *   5 FALL_NONFINITE.  Checked in that precedence: invalid, ineligible,
 *   nonfinite, gap > tau (strict), argmax in the fast-answer set. */
int orc_gate(int valid, int eligible, int nonfinite, double gap, double tau, int in_set);

#ifdef __cplusplus
}
#endif
#endif
