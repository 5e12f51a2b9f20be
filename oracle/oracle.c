/*
 * CPU oracle for the FastMTP greedy speculative-decode step.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, obviously
 * correct reference used by the tests, the smoke check and the CPU
 * baseline of the benchmark.  The GPU library never links, loads or
 * calls it, and it shares no code with the GPU library.
 *
 * What it computes (paper sections cited per function):
 *   - the verifier: a DeepSeekMoE decoder (Table "Model specification":
 *     12 layers, d = 1280, 64 routed + 2 shared experts, top-6, RoPE);
 *   - the FastMTP draft block of the state-shift equation (Section
 *     "Draft-head architecture"): z = P([N_e(e); N_h(a)]),
 *     u = N_o(B(z; pos = p)), logits = W_lm u;
 *   - greedy verification (the acceptance equation) lives in the Python
 *     half of the oracle (oracle/__init__.py).
 *
 * Precision: values are kept at the model's storage points -- float32 for
 * the residual stream, projections, RoPE, scores, softmax, router, gate
 * weights, post-norm states and logits, and (bf16 models) bfloat16 for
 * weights, embeddings, vision rows, the KV cache and every matrix-product
 * input.  Inside one operation (a dot product, a softmax sum, a norm) the
 * arithmetic is float64 and rounds once to the storage type.
 *
 * Row invariance: every row's result is computed by the same sequence of
 * operations whatever other rows share the call, so a row evaluated in a
 * batch equals the same row evaluated alone, bit for bit.  OpenMP only
 * splits independent outputs; it never splits a sum.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t n_layers, hidden, n_heads, head_dim, n_routed, top_k, n_shared, moe_inter,
      draft_inter, vocab, tie_lm_head, bf16;
  double rope_theta, rms_eps;
} orc_dims;

/* Host weights.  Matrices are [out][in] row-major, stored as bf16 bit
 * patterns (bf16 models) or float32.  Norm gains and router bias are float32. */
typedef struct {
  const void *embed, *lm_head; /* [V][H]; lm_head NULL when tied to embed */
  const float* final_norm;     /* [H] */
  const float *attn_norm, *ffn_norm; /* [L][H] */
  const void *wqkv, *wo;       /* [L][3*nh*dh][H], [L][H][nh*dh] */
  const void* router;          /* [L][E][H] */
  const void *exp_gu, *exp_down; /* [L][E][2I][H], [L][E][H][I] */
  const void *sh_gu, *sh_down; /* [L][2*S*I][H], [L][H][S*I] */
  const float* router_bias;    /* [L][E] */
  const float *d_enorm, *d_hnorm, *d_attn_norm, *d_ffn_norm; /* [H] */
  const void *d_eh_proj, *d_wqkv, *d_wo, *d_gu, *d_down;
} orc_weights;

/* ---------------------------------------------------------------- */
/* storage types                                                     */
/* ---------------------------------------------------------------- */

/* Sensitivity-measurement switch (never set for reference values): when
 * nonzero, every sum the oracle forms in float64 -- weight dot products,
 * norm sums of squares, attention scores, softmax sums and the weighted
 * value sum, the router softmax -- is formed in float32 instead, by
 * pairwise summation (each product rounded to float32, halves summed
 * recursively down to blocks of 8 summed in order), and each elementwise
 * step (SwiGLU, RoPE, the MoE combine) rounds to float32.  That is a
 * different but equally valid float32 evaluation of the same model at the
 * same storage points, with about as many roundings in a chain as a
 * blocked or tree-shaped reduction; the distance between the two shows
 * how far summation order alone moves each output. */
static int g_sum32 = 0;
void orc_set_sum32(int on) { g_sum32 = on; }

/* pairwise float32 sum of v[0..n) */
static float psum32(const float* v, int n) {
  if (n <= 8) {
    float s = 0.f;
    for (int i = 0; i < n; ++i) s += v[i];
    return s;
  }
  const int h = n / 2;
  return psum32(v, h) + psum32(v + h, n - h);
}

/* bfloat16 round-to-nearest-even of a float32 value, returned widened */
static float bf16_round(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return f;
  u += 0x7fffu + ((u >> 16) & 1u);
  u &= 0xffff0000u;
  float r;
  memcpy(&r, &u, 4);
  return r;
}

float orc_bf16_round(float f) { return bf16_round(f); }

/* value at a matrix-product input: float32, then bf16 for bf16 models */
static inline float st_in(const orc_dims* d, double x) {
  float f = (float)x;
  return d->bf16 ? bf16_round(f) : f;
}

static inline float wload(const orc_dims* d, const void* base, size_t i) {
  if (d->bf16) {
    uint32_t u = (uint32_t)((const uint16_t*)base)[i] << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
  }
  return ((const float*)base)[i];
}

static inline size_t wsize(const orc_dims* d) { return d->bf16 ? 2 : 4; }

static inline const void* woff(const orc_dims* d, const void* base, size_t elems) {
  return (const char*)base + elems * wsize(d);
}

static double wdot32(const orc_dims* d, const void* w, const float* x, int n) {
  float* t = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
  for (int k = 0; k < n; ++k) t[k] = wload(d, w, (size_t)k) * x[k];
  const float s = psum32(t, n);
  free(t);
  return s;
}

/* dot product of weight row w[0..n) with float vector x, in float64
 * with four interleaved partial sums combined in a fixed order. */
static double wdot(const orc_dims* d, const void* w, const float* x, int n) {
  if (g_sum32) return wdot32(d, w, x, n);
  double s0 = 0, s1 = 0, s2 = 0, s3 = 0;
  int k = 0;
  if (d->bf16) {
    const uint16_t* p = (const uint16_t*)w;
    for (; k + 4 <= n; k += 4) {
      uint32_t u0 = (uint32_t)p[k] << 16, u1 = (uint32_t)p[k + 1] << 16;
      uint32_t u2 = (uint32_t)p[k + 2] << 16, u3 = (uint32_t)p[k + 3] << 16;
      float f0, f1, f2, f3;
      memcpy(&f0, &u0, 4); memcpy(&f1, &u1, 4); memcpy(&f2, &u2, 4); memcpy(&f3, &u3, 4);
      s0 += (double)f0 * x[k];
      s1 += (double)f1 * x[k + 1];
      s2 += (double)f2 * x[k + 2];
      s3 += (double)f3 * x[k + 3];
    }
  } else {
    const float* p = (const float*)w;
    for (; k + 4 <= n; k += 4) {
      s0 += (double)p[k] * x[k];
      s1 += (double)p[k + 1] * x[k + 1];
      s2 += (double)p[k + 2] * x[k + 2];
      s3 += (double)p[k + 3] * x[k + 3];
    }
  }
  for (; k < n; ++k) s0 += (double)wload(d, w, (size_t)k) * x[k];
  return (s0 + s1) + (s2 + s3);
}

/* Y[r][o] = float(W[o][:] . X[r][:]) for r < nr, o < no.  X rows are
 * already at the product-input precision. */
static void linear(const orc_dims* d, const void* W, int no, int ni, const float* X, int nr,
                   float* Y) {
#pragma omp parallel for schedule(static)
  for (int o = 0; o < no; ++o) {
    const void* wr = woff(d, W, (size_t)o * ni);
    for (int r = 0; r < nr; ++r) Y[(size_t)r * no + o] = (float)wdot(d, wr, X + (size_t)r * ni, ni);
  }
}

/* ---------------------------------------------------------------- */
/* building blocks                                                   */
/* ---------------------------------------------------------------- */

/* RMSNorm: out_i = x_i / sqrt(mean(x^2) + eps) * g_i (float32 result). */
void orc_rmsnorm(const float* x, const float* g, int n, double eps, float* out) {
  if (g_sum32) {
    float* t = (float*)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
    for (int i = 0; i < n; ++i) t[i] = x[i] * x[i];
    const float r = 1.0f / sqrtf(psum32(t, n) / (float)n + (float)eps);
    free(t);
    for (int i = 0; i < n; ++i) out[i] = x[i] * r * g[i];
    return;
  }
  double ss = 0;
  for (int i = 0; i < n; ++i) ss += (double)x[i] * x[i];
  double r = 1.0 / sqrt(ss / n + eps);
  for (int i = 0; i < n; ++i) out[i] = (float)((double)x[i] * r * g[i]);
}

/* Rotary embedding (Su et al.), rotate-half pairing: for i < dh/2 the
 * pair (x_i, x_{i+dh/2}) is rotated by angle pos * theta^(-2i/dh).
 * cos/sin come from float64 and are rounded to float32; the rotation
 * itself is float32 arithmetic (one rounding per output). */
void orc_rope(float* x, int dh, int pos, double theta) {
  int half = dh / 2;
  for (int i = 0; i < half; ++i) {
    double inv = pow(theta, -2.0 * i / dh);
    double ang = (double)pos * inv;
    float c = (float)cos(ang), s = (float)sin(ang);
    float a = x[i], b = x[i + half];
    if (g_sum32) {
      x[i] = a * c - b * s;
      x[i + half] = b * c + a * s;
      continue;
    }
    x[i] = (float)((double)a * c - (double)b * s);
    x[i + half] = (float)((double)b * c + (double)a * s);
  }
}

/* One attention head of one query row: scores s_j = (q . k_j) / sqrt(dh)
 * for j < n_keys (rows of K/V with stride dh), softmax, o = sum_j p_j v_j. */
static void attend32(const float* q, const float* K, const float* V, int n_keys, int dh,
                     float* o) {
  const float scale = 1.0f / sqrtf((float)dh);
  const size_t nk = (size_t)(n_keys > 0 ? n_keys : 1);
  float* s = (float*)malloc(sizeof(float) * nk);
  float* t = (float*)malloc(sizeof(float) * (nk > (size_t)dh ? nk : (size_t)dh));
  float m = -INFINITY;
  for (int j = 0; j < n_keys; ++j) {
    for (int c = 0; c < dh; ++c) t[c] = q[c] * K[(size_t)j * dh + c];
    s[j] = psum32(t, dh) * scale;
    if (s[j] > m) m = s[j];
  }
  for (int j = 0; j < n_keys; ++j) s[j] = expf(s[j] - m);
  const float l = psum32(s, n_keys);
  for (int c = 0; c < dh; ++c) {
    for (int j = 0; j < n_keys; ++j) t[j] = s[j] * V[(size_t)j * dh + c];
    o[c] = psum32(t, n_keys) / l;
  }
  free(s);
  free(t);
}

void orc_attend(const float* q, const float* K, const float* V, int n_keys, int dh, float* o) {
  if (g_sum32) {
    attend32(q, K, V, n_keys, dh, o);
    return;
  }
  double scale = 1.0 / sqrt((double)dh);
  double* s = (double*)malloc(sizeof(double) * (size_t)(n_keys > 0 ? n_keys : 1));
  double m = -INFINITY;
  for (int j = 0; j < n_keys; ++j) {
    double acc = 0;
    for (int t = 0; t < dh; ++t) acc += (double)q[t] * K[(size_t)j * dh + t];
    s[j] = (double)(float)((double)(float)acc * scale); /* float32 score */
    if (s[j] > m) m = s[j];
  }
  double l = 0;
  for (int j = 0; j < n_keys; ++j) {
    s[j] = exp(s[j] - m);
    l += s[j];
  }
  for (int t = 0; t < dh; ++t) {
    double acc = 0;
    for (int j = 0; j < n_keys; ++j) acc += s[j] * V[(size_t)j * dh + t];
    o[t] = (float)(acc / l);
  }
  free(s);
}

static inline double silu(double g) { return g / (1.0 + exp(-g)); }

/* ---------------------------------------------------------------- */
/* attention sub-layer over a KV slab [2][nh][cap][dh] (float values   */
/* already at storage precision).                                      */
/* ---------------------------------------------------------------- */

/* h[r] += W_o . attn(RMSNorm(h[r]; g)) for rows at positions pos[r];
 * K/V of every row are written at its position before any row attends. */
static void attn_sublayer(const orc_dims* d, const float* g, const void* wqkv, const void* wo,
                          float* kvslab, int cap, int nr, const int32_t* pos, float* h) {
  const int H = d->hidden, nh = d->n_heads, dh = d->head_dim, nhd = nh * dh;
  float* a = (float*)malloc(sizeof(float) * (size_t)nr * H);
  float* qkv = (float*)malloc(sizeof(float) * (size_t)nr * 3 * nhd);
  float* o = (float*)malloc(sizeof(float) * (size_t)nr * nhd);
  float* proj = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r) {
    orc_rmsnorm(h + (size_t)r * H, g, H, d->rms_eps, a + (size_t)r * H);
    for (int i = 0; i < H; ++i) a[(size_t)r * H + i] = st_in(d, a[(size_t)r * H + i]);
  }
  linear(d, wqkv, 3 * nhd, H, a, nr, qkv);
  for (int r = 0; r < nr; ++r) {
    float* q = qkv + (size_t)r * 3 * nhd;
    float* k = q + nhd;
    float* v = k + nhd;
    for (int hh = 0; hh < nh; ++hh) {
      orc_rope(q + hh * dh, dh, pos[r], d->rope_theta);
      orc_rope(k + hh * dh, dh, pos[r], d->rope_theta);
      float* kd = kvslab + ((size_t)(0 * nh + hh) * cap + pos[r]) * dh;
      float* vd = kvslab + ((size_t)(1 * nh + hh) * cap + pos[r]) * dh;
      for (int t = 0; t < dh; ++t) {
        kd[t] = st_in(d, k[hh * dh + t]);
        vd[t] = st_in(d, v[hh * dh + t]);
      }
    }
  }
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int r = 0; r < nr; ++r)
    for (int hh = 0; hh < nh; ++hh) {
      const float* q = qkv + (size_t)r * 3 * nhd + hh * dh;
      const float* K = kvslab + (size_t)(0 * nh + hh) * cap * dh;
      const float* V = kvslab + (size_t)(1 * nh + hh) * cap * dh;
      float* out = o + (size_t)r * nhd + hh * dh;
      orc_attend(q, K, V, pos[r] + 1, dh, out);
      for (int t = 0; t < dh; ++t) out[t] = st_in(d, out[t]);
    }
  linear(d, wo, H, nhd, o, nr, proj);
  for (size_t i = 0; i < (size_t)nr * H; ++i) h[i] = (float)((double)h[i] + proj[i]);
  free(a); free(qkv); free(o); free(proj);
}

/* ---------------------------------------------------------------- */
/* router and MoE FFN (DeepSeekMoE; softmax gate over all routed       */
/* experts, top-k selection, shared experts with weight one)           */
/* ---------------------------------------------------------------- */

/* Router of one layer for one product-input row y: float32 logits
 * (+ bias), float32 softmax probabilities over all E experts, top-k by
 * logit (higher first, equal logits -> lower expert id), and the gap
 * between the k-th and (k+1)-th largest logit (0 when k == E). */
void orc_router(const orc_dims* d, const orc_weights* w, int layer, const float* y,
                float* logits, float* probs, int32_t* topk, float* gap) {
  const int H = d->hidden, E = d->n_routed, k = d->top_k;
  const void* Wr = woff(d, w->router, (size_t)layer * E * H);
  double mx = -INFINITY;
  for (int e = 0; e < E; ++e) {
    float r = (float)wdot(d, woff(d, Wr, (size_t)e * H), y, H);
    if (w->router_bias) r = (float)((double)r + w->router_bias[(size_t)layer * E + e]);
    logits[e] = r;
    if (r > mx) mx = r;
  }
  if (g_sum32) {
    for (int e = 0; e < E; ++e) probs[e] = expf(logits[e] - (float)mx);
    const float sum = psum32(probs, E);
    for (int e = 0; e < E; ++e) probs[e] /= sum;
  } else {
    double sum = 0;
    for (int e = 0; e < E; ++e) sum += exp((double)logits[e] - mx);
    for (int e = 0; e < E; ++e) probs[e] = (float)(exp((double)logits[e] - mx) / sum);
  }
  unsigned char* taken = (unsigned char*)calloc((size_t)E, 1);
  for (int j = 0; j < k; ++j) {
    int best = -1;
    for (int e = 0; e < E; ++e)
      if (!taken[e] && (best < 0 || logits[e] > logits[best])) best = e;
    topk[j] = best;
    taken[best] = 1;
  }
  if (gap) {
    int nxt = -1;
    for (int e = 0; e < E; ++e)
      if (!taken[e] && (nxt < 0 || logits[e] > logits[nxt])) nxt = e;
    *gap = nxt < 0 ? 0.0f : logits[topk[k - 1]] - logits[nxt];
  }
  free(taken);
}

/* One SwiGLU expert with gate rows Wg[I][H], up rows Wu[I][H] and down
 * Wd[H][ldd] (columns col0..col0+I-1): out = Wd (silu(Wg y) * (Wu y)). */
static void swiglu_expert(const orc_dims* d, const void* Wg, const void* Wu, const void* Wd,
                          int ldd, int col0, int I, const float* y, int nr, float* out) {
  const int H = d->hidden;
  float* g = (float*)malloc(sizeof(float) * (size_t)nr * I);
  float* u = (float*)malloc(sizeof(float) * (size_t)nr * I);
  float* act = (float*)malloc(sizeof(float) * (size_t)nr * I);
  linear(d, Wg, I, H, y, nr, g);
  linear(d, Wu, I, H, y, nr, u);
  for (size_t i = 0; i < (size_t)nr * I; ++i) {
    float gu = g_sum32 ? g[i] / (1.0f + expf(-g[i])) * u[i] : (float)(silu(g[i]) * (double)u[i]);
    act[i] = st_in(d, gu);
  }
#pragma omp parallel for schedule(static)
  for (int o = 0; o < H; ++o) {
    const void* wr = woff(d, Wd, (size_t)o * ldd + col0);
    for (int r = 0; r < nr; ++r) out[(size_t)r * H + o] = (float)wdot(d, wr, act + (size_t)r * I, I);
  }
  free(g); free(u); free(act);
}

/* Route check/follow.  If follow != NULL it holds a top-k set per row
 * chosen elsewhere; the set is accepted when it is a top-k set of the
 * oracle's logits up to tol (min chosen logit >= max unchosen - tol).
 * Accepted sets replace the oracle's own; rejected ones are counted and
 * the oracle's own set is used.  Returns the number of rejected rows. */
static int follow_route(const orc_dims* d, const float* logits, int32_t* topk,
                        const int32_t* given, float tol, int* n_followed) {
  const int E = d->n_routed, k = d->top_k;
  for (int t = 0; t < k; ++t) {
    if (given[t] < 0 || given[t] >= E) return 1;
    for (int u = 0; u < t; ++u)
      if (given[u] == given[t]) return 1;
  }
  int same = 1;
  for (int t = 0; t < k; ++t) same &= (given[t] == topk[t]);
  if (same) return 0;
  double min_in = INFINITY, max_out = -INFINITY;
  for (int e = 0; e < E; ++e) {
    int in = 0;
    for (int t = 0; t < k; ++t) in |= (given[t] == e);
    if (in && logits[e] < min_in) min_in = logits[e];
    if (!in && logits[e] > max_out) max_out = logits[e];
  }
  if (min_in >= max_out - tol) {
    for (int t = 0; t < k; ++t) topk[t] = given[t];
    if (n_followed) ++*n_followed;
    return 0;
  }
  return 1;
}

/* h[r] += sum_s FFN_s(y_r) + sum_{e in topk(r), ascending e} p_e FFN_e(y_r)
 * with y_r = RMSNorm(h[r]; ffn_norm).  Routing outputs are optional. */
static int moe_sublayer(const orc_dims* d, const orc_weights* w, int layer, int nr, float* h,
                        const int32_t* follow, float tol, int* n_followed, int32_t* route_idx,
                        float* route_w, float* route_gap, float* router_logits) {
  const int H = d->hidden, E = d->n_routed, k = d->top_k, S = d->n_shared, I = d->moe_inter;
  int bad = 0;
  float* y = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r) {
    orc_rmsnorm(h + (size_t)r * H, w->ffn_norm + (size_t)layer * H, H, d->rms_eps,
                y + (size_t)r * H);
    for (int i = 0; i < H; ++i) y[(size_t)r * H + i] = st_in(d, y[(size_t)r * H + i]);
  }
  int32_t* sel = (int32_t*)malloc(sizeof(int32_t) * (size_t)nr * k);
  float* pr = (float*)malloc(sizeof(float) * (size_t)nr * E);
  float* lg = (float*)malloc(sizeof(float) * (size_t)E);
  for (int r = 0; r < nr; ++r) {
    float gap;
    orc_router(d, w, layer, y + (size_t)r * H, lg, pr + (size_t)r * E, sel + (size_t)r * k, &gap);
    if (follow) bad += follow_route(d, lg, sel + (size_t)r * k, follow + (size_t)r * k, tol, n_followed);
    if (route_gap) route_gap[r] = gap;
    if (router_logits) memcpy(router_logits + (size_t)r * E, lg, sizeof(float) * (size_t)E);
  }
  free(lg);
  /* delta[r] accumulates the FFN output of row r in float64 */
  double* delta = (double*)calloc((size_t)nr * H, sizeof(double));
  float* tmp = (float*)malloc(sizeof(float) * (size_t)nr * H);
  /* shared experts: each is a width-I SwiGLU with weight one */
  const void* shg = woff(d, w->sh_gu, (size_t)layer * 2 * S * I * H);
  const void* shd = woff(d, w->sh_down, (size_t)layer * H * S * I);
  for (int s = 0; s < S; ++s) {
    swiglu_expert(d, woff(d, shg, (size_t)s * I * H), woff(d, shg, (size_t)(S + s) * I * H), shd,
                  S * I, s * I, I, y, nr, tmp);
    for (size_t i = 0; i < (size_t)nr * H; ++i)
      delta[i] = g_sum32 ? (double)((float)delta[i] + tmp[i]) : delta[i] + tmp[i];
  }
  /* routed experts, in ascending expert id, over the rows that chose them */
  int32_t* rows = (int32_t*)malloc(sizeof(int32_t) * (size_t)nr);
  float* ys = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int e = 0; e < E; ++e) {
    int ne = 0;
    for (int r = 0; r < nr; ++r)
      for (int j = 0; j < k; ++j)
        if (sel[(size_t)r * k + j] == e) rows[ne++] = r;
    if (!ne) continue;
    for (int t = 0; t < ne; ++t) memcpy(ys + (size_t)t * H, y + (size_t)rows[t] * H, sizeof(float) * H);
    const void* gu = woff(d, w->exp_gu, ((size_t)layer * E + e) * 2 * I * H);
    const void* dn = woff(d, w->exp_down, ((size_t)layer * E + e) * H * I);
    swiglu_expert(d, gu, woff(d, gu, (size_t)I * H), dn, I, 0, I, ys, ne, tmp);
    for (int t = 0; t < ne; ++t) {
      int r = rows[t];
      float p = pr[(size_t)r * E + e];
      for (int i = 0; i < H; ++i) {
        const float c = (float)((double)p * tmp[(size_t)t * H + i]);
        double* dv = delta + (size_t)r * H + i;
        *dv = g_sum32 ? (double)((float)*dv + c) : *dv + c;
      }
    }
  }
  for (int r = 0; r < nr; ++r) {
    for (int i = 0; i < H; ++i) {
      float dv = (float)delta[(size_t)r * H + i];
      h[(size_t)r * H + i] = (float)((double)h[(size_t)r * H + i] + dv);
    }
    if (route_idx || route_w) {
      for (int j = 0; j < k; ++j) {
        int e = sel[(size_t)r * k + j];
        if (route_idx) route_idx[(size_t)r * k + j] = e;
        if (route_w) route_w[(size_t)r * k + j] = pr[(size_t)r * E + e];
      }
    }
  }
  free(y); free(sel); free(pr); free(delta); free(tmp); free(rows); free(ys);
  return bad;
}

/* ---------------------------------------------------------------- */
/* LM head with argmax                                               */
/* ---------------------------------------------------------------- */

/* logits of the rows with mask[r] != 0 (all rows when mask == NULL):
 * l_v = W_lm[v] . in(x); argmax with ties to the lowest id; margin =
 * top-1 minus the largest other logit. */
static void lm_head(const orc_dims* d, const orc_weights* w, const float* x, int nr,
                    const uint8_t* mask, float* logits, int32_t* amax, float* margin) {
  const int H = d->hidden, V = d->vocab;
  const void* W = d->tie_lm_head ? w->embed : w->lm_head;
  float* xin = (float*)malloc(sizeof(float) * H);
  float* lg = (float*)malloc(sizeof(float) * (size_t)V);
  for (int r = 0; r < nr; ++r) {
    if (mask && !mask[r]) continue;
    for (int i = 0; i < H; ++i) xin[i] = st_in(d, x[(size_t)r * H + i]);
    linear(d, W, V, H, xin, 1, lg);
    int best = 0;
    for (int v = 1; v < V; ++v)
      if (lg[v] > lg[best]) best = v;
    float second = -INFINITY;
    for (int v = 0; v < V; ++v)
      if (v != best && lg[v] > second) second = lg[v];
    if (amax) amax[r] = best;
    if (margin) margin[r] = lg[best] - second;
    if (logits) memcpy(logits + (size_t)r * V, lg, sizeof(float) * V);
  }
  free(xin);
  free(lg);
}

/* input row: token embedding E[tok] (tok >= 0) or the given row emb[r] */
static void input_row(const orc_dims* d, const orc_weights* w, int32_t tok, const void* emb,
                      int r, float* out) {
  const int H = d->hidden;
  if (tok >= 0) {
    for (int i = 0; i < H; ++i) out[i] = wload(d, w->embed, (size_t)tok * H + i);
  } else {
    for (int i = 0; i < H; ++i) out[i] = wload(d, emb, (size_t)r * H + i);
  }
}

/* ---------------------------------------------------------------- */
/* verifier rows                                                     */
/* ---------------------------------------------------------------- */

/* Runs nr rows of one sequence through the verifier.  Row r is token
 * tok[r] (or, when tok[r] < 0, the vision row emb[r]) at position pos[r];
 * its K/V are written to kv = [L][2][nh][cap][dh] at pos[r].  Positions
 * below pos[r] must already hold K/V (earlier rows of the call count).
 * Outputs (each optional): b = final-norm state [nr][H]; LM-head results
 * for rows with head_mask set; routing per layer [L][nr][k]; k-th vs
 * (k+1)-th router-logit gap [L][nr]; router logits [L][nr][E].  follow_route [L][nr][k] makes the
 * oracle adopt externally chosen near-tie routes (see follow_route), with
 * tolerance route_tol[l] in layer l.
 * Returns the number of rejected route sets (0 without follow_route), or
 * -1 on a position outside the cache. */
int orc_verify_rows(const orc_dims* d, const orc_weights* w, float* kv, int cap, int nr,
                    const int32_t* tok, const void* emb, const int32_t* pos,
                    const int32_t* follow_route, const float* route_tol, int* n_followed,
                    float* b_out, const uint8_t* head_mask, float* logits, int32_t* amax,
                    float* margin, int32_t* route_idx, float* route_w, float* route_gap,
                    float* router_logits) {
  const int H = d->hidden, L = d->n_layers, nh = d->n_heads, dh = d->head_dim, k = d->top_k;
  for (int r = 0; r < nr; ++r)
    if (pos[r] < 0 || pos[r] >= cap) return -1;
  float* h = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r) input_row(d, w, tok[r], emb, r, h + (size_t)r * H);
  int bad = 0;
  const size_t slab = (size_t)2 * nh * cap * dh;
  const int nhd = nh * dh;
  for (int l = 0; l < L; ++l) {
    attn_sublayer(d, w->attn_norm + (size_t)l * H, woff(d, w->wqkv, (size_t)l * 3 * nhd * H),
                  woff(d, w->wo, (size_t)l * H * nhd), kv + (size_t)l * slab, cap, nr, pos, h);
    bad += moe_sublayer(d, w, l, nr, h, follow_route ? follow_route + (size_t)l * nr * k : NULL,
                        follow_route ? route_tol[l] : 0.f, n_followed,
                        route_idx ? route_idx + (size_t)l * nr * k : NULL,
                        route_w ? route_w + (size_t)l * nr * k : NULL,
                        route_gap ? route_gap + (size_t)l * nr : NULL,
                        router_logits ? router_logits + (size_t)l * nr * d->n_routed : NULL);
  }
  float* b = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r)
    orc_rmsnorm(h + (size_t)r * H, w->final_norm, H, d->rms_eps, b + (size_t)r * H);
  if (b_out) memcpy(b_out, b, sizeof(float) * (size_t)nr * H);
  if (logits || amax || margin) lm_head(d, w, b, nr, head_mask, logits, amax, margin);
  free(h);
  free(b);
  return bad;
}

/* One verifier layer (attention sub-layer, then MoE sub-layer) for nr rows
 * of one sequence at positions pos[r], from the layer input h [nr][H]
 * (overwritten with the layer output) and the layer's KV slab kv_l =
 * [2][nh][cap][dh] (the rows' K/V are written at their positions before
 * any row attends; positions below must hold K/V).  follow [nr][k] (or
 * NULL): routes adopted at near-ties up to tol, as in orc_verify_rows.
 * Routing outputs for this layer only.  Returns the number of rejected
 * route sets, or -1 on a bad position. */
int orc_verify_layer(const orc_dims* d, const orc_weights* w, int layer, float* kv_l, int cap,
                     int nr, const int32_t* pos, float* h, const int32_t* follow, float tol,
                     int* n_followed, int32_t* route_idx, float* route_gap,
                     float* router_logits) {
  const int H = d->hidden, nhd = d->n_heads * d->head_dim;
  for (int r = 0; r < nr; ++r)
    if (pos[r] < 0 || pos[r] >= cap) return -1;
  attn_sublayer(d, w->attn_norm + (size_t)layer * H, woff(d, w->wqkv, (size_t)layer * 3 * nhd * H),
                woff(d, w->wo, (size_t)layer * H * nhd), kv_l, cap, nr, pos, h);
  return moe_sublayer(d, w, layer, nr, h, follow, tol, n_followed, route_idx, NULL, route_gap,
                      router_logits);
}

/* The verifier's head on nr residual rows h [nr][H]: b = final RMSNorm
 * (b_out, optional), then the LM head and greedy argmax of every row
 * (logits [nr][V] optional, amax, margin). */
void orc_head(const orc_dims* d, const orc_weights* w, int nr, const float* h, float* b_out,
              float* logits, int32_t* amax, float* margin) {
  const int H = d->hidden;
  float* b = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r)
    orc_rmsnorm(h + (size_t)r * H, w->final_norm, H, d->rms_eps, b + (size_t)r * H);
  if (b_out) memcpy(b_out, b, sizeof(float) * (size_t)nr * H);
  lm_head(d, w, b, nr, NULL, logits, amax, margin);
  free(b);
}

/* LM head on given post-norm rows x [nr][H] (no final norm): logits
 * [nr][V] = W_lm in(x).  The draft-head objective's verifier distribution
 * Q_p is the softmax of these logits of b_{p+1}. */
void orc_lm_logits(const orc_dims* d, const orc_weights* w, int nr, const float* x,
                   float* logits) {
  lm_head(d, w, x, nr, NULL, logits, NULL, NULL);
}

/* ---------------------------------------------------------------- */
/* FastMTP draft rows (state-shift equation)                          */
/* ---------------------------------------------------------------- */

/* Runs nr draft rows.  Row r has state a[r] (float32 [H]) and next input
 * tok[r] (or vision row emb[r] when tok[r] < 0) at position pos[r]:
 *   z = P [N_e(e); N_h(a)]                  (embedding first, state second)
 *   z += W_o attn(RMSNorm(z)) over the draft KV dkv = [2][nh][cap][dh]
 *   z += FFN(RMSNorm(z))                    (dense SwiGLU, width F)
 *   u = N_o(z)                              (verifier final norm, tied)
 *   logits = W_lm in(u)                     (rows with head_mask set)
 * K/V of every row is written at pos[r].  Returns -1 on a bad position. */
int orc_draft_rows(const orc_dims* d, const orc_weights* w, float* dkv, int cap, int nr,
                   const int32_t* tok, const void* emb, const float* a, const int32_t* pos,
                   float* u_out, const uint8_t* head_mask, float* logits, int32_t* amax,
                   float* margin) {
  const int H = d->hidden, F = d->draft_inter;
  for (int r = 0; r < nr; ++r)
    if (pos[r] < 0 || pos[r] >= cap) return -1;
  float* cat = (float*)malloc(sizeof(float) * (size_t)nr * 2 * H);
  float* e = (float*)malloc(sizeof(float) * H);
  for (int r = 0; r < nr; ++r) {
    float* c = cat + (size_t)r * 2 * H;
    input_row(d, w, tok[r], emb, r, e);
    orc_rmsnorm(e, w->d_enorm, H, d->rms_eps, c);
    orc_rmsnorm(a + (size_t)r * H, w->d_hnorm, H, d->rms_eps, c + H);
    for (int i = 0; i < 2 * H; ++i) c[i] = st_in(d, c[i]);
  }
  float* z = (float*)malloc(sizeof(float) * (size_t)nr * H);
  linear(d, w->d_eh_proj, H, 2 * H, cat, nr, z);
  attn_sublayer(d, w->d_attn_norm, w->d_wqkv, w->d_wo, dkv, cap, nr, pos, z);
  /* dense FFN: gate rows 0..F-1, up rows F..2F-1 of d_gu */
  float* y = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r) {
    orc_rmsnorm(z + (size_t)r * H, w->d_ffn_norm, H, d->rms_eps, y + (size_t)r * H);
    for (int i = 0; i < H; ++i) y[(size_t)r * H + i] = st_in(d, y[(size_t)r * H + i]);
  }
  float* f = (float*)malloc(sizeof(float) * (size_t)nr * H);
  swiglu_expert(d, w->d_gu, woff(d, w->d_gu, (size_t)F * H), w->d_down, F, 0, F, y, nr, f);
  for (size_t i = 0; i < (size_t)nr * H; ++i) z[i] = (float)((double)z[i] + f[i]);
  float* u = (float*)malloc(sizeof(float) * (size_t)nr * H);
  for (int r = 0; r < nr; ++r)
    orc_rmsnorm(z + (size_t)r * H, w->final_norm, H, d->rms_eps, u + (size_t)r * H);
  if (u_out) memcpy(u_out, u, sizeof(float) * (size_t)nr * H);
  if (logits || amax || margin) lm_head(d, w, u, nr, head_mask, logits, amax, margin);
  free(cat); free(e); free(z); free(y); free(f); free(u);
  return 0;
}

/* MoE sub-layer of one layer alone (for the brute-force pin):
 * h_out = h_in + shared + routed FFN of RMSNorm(h_in; ffn_norm). */
void orc_moe_sublayer(const orc_dims* d, const orc_weights* w, int layer, int nr,
                      const float* h_in, float* h_out, int32_t* route_idx, float* route_w,
                      float* route_gap) {
  memcpy(h_out, h_in, sizeof(float) * (size_t)nr * d->hidden);
  moe_sublayer(d, w, layer, nr, h_out, NULL, 0.0f, NULL, route_idx, route_w, route_gap, NULL);
}
