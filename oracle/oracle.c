/* CPU oracle: plain fp64 definitions of the pre-position step and the gate.
 * TEST INFRASTRUCTURE ONLY (see oracle.h).  Every sum runs in ascending index
 * order, one output element at a time, so results do not depend on the number
 * of OpenMP threads and a row's result does not depend on the other rows. */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* RMSNorm: out = x / sqrt(mean(x^2) + eps) * g, per row. */
void orc_rmsnorm(int M, int d, const double* x, const float* g, double eps, double* out) {
  for (int m = 0; m < M; ++m) {
    const double* r = x + (int64_t)m * d;
    double ss = 0.0;
    for (int i = 0; i < d; ++i) ss += r[i] * r[i];
    const double inv = 1.0 / sqrt(ss / d + eps);
    for (int i = 0; i < d; ++i) out[(int64_t)m * d + i] = r[i] * inv * (double)g[i];
  }
}

/* y[m][n] = sum_k x[m][k] * W[n][k]   (W holds one output feature per row) */
void orc_linear(int M, int N, int K, const double* x, const float* W, double* y) {
#pragma omp parallel for schedule(static)
  for (int n = 0; n < N; ++n) {
    const float* w = W + (int64_t)n * K;
    for (int m = 0; m < M; ++m) {
      const double* xr = x + (int64_t)m * K;
      double acc = 0.0;
      for (int k = 0; k < K; ++k) acc += xr[k] * (double)w[k];
      y[(int64_t)m * N + n] = acc;
    }
  }
}

/* Rotary position embedding, rotate-half pairing (i, i + dh/2), applied to
 * u[M][H][dh] for the token at position pos0 + m:
 *   theta_i = P * base^(-2i/dh),
 *   (a, b) <- (a cos theta_i - b sin theta_i, a sin theta_i + b cos theta_i). */
void orc_rope(int M, int H, int dh, double* u, int64_t pos0, double base) {
  const int half = dh / 2;
  for (int m = 0; m < M; ++m) {
    const double P = (double)(pos0 + m);
    for (int i = 0; i < half; ++i) {
      const double th = P * pow(base, -2.0 * i / dh);
      const double c = cos(th), s = sin(th);
      for (int h = 0; h < H; ++h) {
        double* v = u + ((int64_t)m * H + h) * dh;
        const double a = v[i], b = v[i + half];
        v[i] = a * c - b * s;
        v[i + half] = a * s + b * c;
      }
    }
  }
}

/* Causal grouped-query attention of M new queries (positions n_past + m) against
 * cached cells 0 .. n_past + m.  q head h reads kv head h / (Hq / Hkv).
 *   s_i = q . K_i / sqrt(dh),  o = sum_i softmax(s)_i V_i. */
void orc_attention(int M, int Hq, int Hkv, int dh, const double* q, const float* Kc,
                   const float* Vc, int64_t cap, int64_t n_past, double* out) {
  const int G = Hq / Hkv;
  const double scale = 1.0 / sqrt((double)dh);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int m = 0; m < M; ++m) {
    for (int h = 0; h < Hq; ++h) {
      const int64_t P = n_past + m;
      const int c = h / G;
      const double* qv = q + ((int64_t)m * Hq + h) * dh;
      const float* K = Kc + (int64_t)c * cap * dh;
      const float* V = Vc + (int64_t)c * cap * dh;
      double* s = (double*)malloc(sizeof(double) * (size_t)(P + 1));
      double mx = -INFINITY;
      for (int64_t i = 0; i <= P; ++i) {
        double acc = 0.0;
        for (int t = 0; t < dh; ++t) acc += qv[t] * (double)K[i * dh + t];
        s[i] = acc * scale;
        if (s[i] > mx) mx = s[i];
      }
      double Z = 0.0;
      for (int64_t i = 0; i <= P; ++i) {
        s[i] = exp(s[i] - mx);
        Z += s[i];
      }
      double* o = out + ((int64_t)m * Hq + h) * dh;
      for (int t = 0; t < dh; ++t) {
        double acc = 0.0;
        for (int64_t i = 0; i <= P; ++i) acc += s[i] * (double)V[i * dh + t];
        o[t] = acc / Z;
      }
      free(s);
    }
  }
}

/* SwiGLU: out = silu(gate) * up with silu(z) = z / (1 + e^-z). */
void orc_swiglu(int M, int F, const double* gate, const double* up, double* out) {
  for (int64_t i = 0; i < (int64_t)M * F; ++i) out[i] = gate[i] / (1.0 + exp(-gate[i])) * up[i];
}

/* Round to the nearest bf16 value (8 significant bits), ties to even, straight
 * from the double (no intermediate fp32 rounding). */
double orc_round_bf16(double v) {
  if (v == 0.0 || !isfinite(v)) return v;
  int e;
  frexp(v, &e);                     /* |v| in [2^(e-1), 2^e) */
  int ulp_exp = e - 8;              /* spacing of 8-bit significands */
  if (ulp_exp < -133) ulp_exp = -133; /* bf16 subnormal spacing 2^-133 */
  const double q = ldexp(v, -ulp_exp);
  const double r = nearbyint(q);    /* default rounding mode: nearest, ties to even */
  const double out = ldexp(r, ulp_exp);
  if (fabs(out) > 3.3895313892515355e38) return v > 0 ? INFINITY : -INFINITY;
  return out;
}

void orc_embed(int M, int d, const int32_t* tokens, const float* E, double* x) {
  for (int m = 0; m < M; ++m)
    for (int i = 0; i < d; ++i) x[(int64_t)m * d + i] = (double)E[(int64_t)tokens[m] * d + i];
}

static double to_cache(double v, int bf16) { return bf16 ? orc_round_bf16(v) : (double)(float)v; }

int orc_layer(const orc_shape* s, const orc_layer_weights* w, float* Kc, float* Vc,
              int64_t cap, int64_t n_past, int M, double* x) {
  const int d = s->d_model, dh = s->head_dim, Hq = s->n_q, Hkv = s->n_kv, F = s->ffn;
  const int nq = Hq * dh, nkv = Hkv * dh;
  if (n_past + M > cap || Hq % Hkv) return -1;
  double* h = (double*)malloc(sizeof(double) * (size_t)M * d);
  double* q = (double*)malloc(sizeof(double) * (size_t)M * nq);
  double* k = (double*)malloc(sizeof(double) * (size_t)M * nkv);
  double* v = (double*)malloc(sizeof(double) * (size_t)M * nkv);
  double* a = (double*)malloc(sizeof(double) * (size_t)M * nq);
  double* y = (double*)malloc(sizeof(double) * (size_t)M * d);
  double* g = (double*)malloc(sizeof(double) * (size_t)M * F);
  double* u = (double*)malloc(sizeof(double) * (size_t)M * F);

  /* attention block */
  orc_rmsnorm(M, d, x, w->attn_norm, s->eps, h);
  orc_linear(M, nq, d, h, w->wq, q);
  orc_linear(M, nkv, d, h, w->wk, k);
  orc_linear(M, nkv, d, h, w->wv, v);
  orc_rope(M, Hq, dh, q, n_past, s->rope_base);
  orc_rope(M, Hkv, dh, k, n_past, s->rope_base);
  for (int m = 0; m < M; ++m)          /* append the new cells at positions n_past + m */
    for (int c = 0; c < Hkv; ++c)
      for (int t = 0; t < dh; ++t) {
        const int64_t dst = ((int64_t)c * cap + n_past + m) * dh + t;
        Kc[dst] = (float)to_cache(k[((int64_t)m * Hkv + c) * dh + t], s->cache_bf16);
        Vc[dst] = (float)to_cache(v[((int64_t)m * Hkv + c) * dh + t], s->cache_bf16);
      }
  orc_attention(M, Hq, Hkv, dh, q, Kc, Vc, cap, n_past, a);
  orc_linear(M, d, nq, a, w->wo, y);
  for (int64_t i = 0; i < (int64_t)M * d; ++i) x[i] += y[i];

  /* MLP block */
  orc_rmsnorm(M, d, x, w->mlp_norm, s->eps, h);
  orc_linear(M, F, d, h, w->wg, g);
  orc_linear(M, F, d, h, w->wu, u);
  orc_swiglu(M, F, g, u, g);
  orc_linear(M, d, F, g, w->wd, y);
  for (int64_t i = 0; i < (int64_t)M * d; ++i) x[i] += y[i];

  free(h); free(q); free(k); free(v); free(a); free(y); free(g); free(u);
  return 0;
}

/* The same layer when only the LAST row's output is needed afterwards (the final layer
 * of a pre-position: the ready distribution reads the last row alone).  The K and V
 * cells of every row are still computed and appended, since the last row attends to
 * them; queries, attention, projections and the MLP run for the last row only, with
 * exactly the arithmetic of orc_layer.  Rows 0 .. M-2 of x are left unchanged. */
int orc_layer_last(const orc_shape* s, const orc_layer_weights* w, float* Kc, float* Vc,
                   int64_t cap, int64_t n_past, int M, double* x) {
  const int d = s->d_model, dh = s->head_dim, Hq = s->n_q, Hkv = s->n_kv, F = s->ffn;
  const int nq = Hq * dh, nkv = Hkv * dh;
  if (n_past + M > cap || Hq % Hkv || M < 1) return -1;
  double* h = (double*)malloc(sizeof(double) * (size_t)M * d);
  double* k = (double*)malloc(sizeof(double) * (size_t)M * nkv);
  double* v = (double*)malloc(sizeof(double) * (size_t)M * nkv);
  double* q = (double*)malloc(sizeof(double) * (size_t)nq);
  double* a = (double*)malloc(sizeof(double) * (size_t)nq);
  double* y = (double*)malloc(sizeof(double) * (size_t)d);
  double* g = (double*)malloc(sizeof(double) * (size_t)F);
  double* u = (double*)malloc(sizeof(double) * (size_t)F);
  double* xl = x + (int64_t)(M - 1) * d;
  const double* hl;

  orc_rmsnorm(M, d, x, w->attn_norm, s->eps, h);
  orc_linear(M, nkv, d, h, w->wk, k);
  orc_linear(M, nkv, d, h, w->wv, v);
  orc_rope(M, Hkv, dh, k, n_past, s->rope_base);
  for (int m = 0; m < M; ++m)
    for (int c = 0; c < Hkv; ++c)
      for (int t = 0; t < dh; ++t) {
        const int64_t dst = ((int64_t)c * cap + n_past + m) * dh + t;
        Kc[dst] = (float)to_cache(k[((int64_t)m * Hkv + c) * dh + t], s->cache_bf16);
        Vc[dst] = (float)to_cache(v[((int64_t)m * Hkv + c) * dh + t], s->cache_bf16);
      }
  hl = h + (int64_t)(M - 1) * d;
  orc_linear(1, nq, d, hl, w->wq, q);
  orc_rope(1, Hq, dh, q, n_past + M - 1, s->rope_base);
  orc_attention(1, Hq, Hkv, dh, q, Kc, Vc, cap, n_past + M - 1, a);
  orc_linear(1, d, nq, a, w->wo, y);
  for (int i = 0; i < d; ++i) xl[i] += y[i];
  orc_rmsnorm(1, d, xl, w->mlp_norm, s->eps, h);
  orc_linear(1, F, d, h, w->wg, g);
  orc_linear(1, F, d, h, w->wu, u);
  orc_swiglu(1, F, g, u, g);
  orc_linear(1, d, F, g, w->wd, y);
  for (int i = 0; i < d; ++i) xl[i] += y[i];
  free(h); free(k); free(v); free(q); free(a); free(y); free(g); free(u);
  return 0;
}

void orc_logits(const orc_shape* s, const double* x_last, const float* g_final,
                const float* w_lm, const float* bias, double* logits) {
  const int d = s->d_model;
  double* z = (double*)malloc(sizeof(double) * (size_t)d);
  orc_rmsnorm(1, d, x_last, g_final, s->eps, z);
  orc_linear(1, s->vocab, d, z, w_lm, logits);
  if (bias)
    for (int i = 0; i < s->vocab; ++i) logits[i] += (double)bias[i];
  free(z);
}

/* ---- summary: a full sort, the plainest top-2 there is ---- */
static const double* g_sort_vals;
static int cmp_desc(const void* pa, const void* pb) {
  const int a = *(const int*)pa, b = *(const int*)pb;
  const double va = g_sort_vals[a], vb = g_sort_vals[b];
  const int na = isnan(va), nb = isnan(vb);
  if (na != nb) return na - nb; /* NaN sorts last */
  if (!na) {
    if (va > vb) return -1;
    if (va < vb) return 1;
  }
  return (a > b) - (a < b);     /* equal values: ascending index */
}

void orc_summary_of(int V, const double* logits, orc_summary* out) {
  int* idx = (int*)malloc(sizeof(int) * (size_t)V);
  for (int i = 0; i < V; ++i) idx[i] = i;
  g_sort_vals = logits;
  qsort(idx, (size_t)V, sizeof(int), cmp_desc);
  memset(out, 0, sizeof(*out));
  out->argmax = idx[0];
  out->second = V > 1 ? idx[1] : -1;
  out->top1 = logits[idx[0]];
  out->top2 = V > 1 ? logits[idx[1]] : -INFINITY;
  out->gap = out->top1 - out->top2;
  int nonfinite = 0;
  for (int i = 0; i < V; ++i) nonfinite |= !isfinite(logits[i]);
  out->nonfinite = nonfinite;
  if (nonfinite) {
    out->lse = NAN;
  } else {
    const double mx = out->top1;
    double z = 0.0;
    for (int i = 0; i < V; ++i) z += exp(logits[i] - mx);
    out->lse = mx + log(z);
  }
  free(idx);
}

int orc_gate(int valid, int eligible, int nonfinite, double gap, double tau, int in_set) {
  if (!valid) return 1;
  if (!eligible) return 2;
  if (nonfinite) return 5;
  if (!(gap > tau)) return 3;
  if (!in_set) return 4;
  return 0;
}

/* Sliding-window shift (Sec. 3.6: a mutation that relocates positions).  The oldest
 * `delta` of the n_s cached cells are dropped and cell p moves to p - delta.  A cached
 * key is RoPE(k, p); at its new position it must be RoPE(k, p - delta), which is the
 * key rotated once more at position -delta (rotations compose by adding angles), so the
 * key is turned by orc_rope at position -delta and rounded to the cache format; the value
 * moves unchanged.  Kc, Vc: [n_kv][cap][dh].  Cells at n_s - delta and above keep
 * their old contents (they lie past the new n_s). */
int orc_shift_cells(int n_kv, int64_t cap, int dh, float* Kc, float* Vc, int64_t n_s,
                    int64_t delta, double rope_base, int cache_bf16) {
  if (delta < 1 || delta > n_s || n_s > cap) return 1;
  const int64_t n_new = n_s - delta;
  double* u = (double*)malloc(sizeof(double) * dh);
  if (!u) return 2;
  for (int c = 0; c < n_kv; ++c)
    for (int64_t i = 0; i < n_new; ++i) {  /* ascending: sources lie above destinations */
      const int64_t src = ((int64_t)c * cap + i + delta) * dh, dst = ((int64_t)c * cap + i) * dh;
      for (int t = 0; t < dh; ++t) u[t] = Kc[src + t];
      orc_rope(1, 1, dh, u, -delta, rope_base);
      for (int t = 0; t < dh; ++t) {
        Kc[dst + t] = (float)to_cache(u[t], cache_bf16);
        Vc[dst + t] = Vc[src + t];
      }
    }
  free(u);
  return 0;
}
