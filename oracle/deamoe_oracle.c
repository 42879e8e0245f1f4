/* DeaMoE decode-layer oracle: TEST INFRASTRUCTURE ONLY (see deamoe_oracle.h).
 *
 * Written from the paper:
 *   Eq. 1     a standard SwiGLU expert  d(SiLU(W_g x) * W_u x)
 *   Eq. 2     S(x) = TopK(W_r x, k)
 *   Eq. 3     y = sum_{i in S(x)} p_i(x) E_i(x), p after softmax normalisation
 *             and scaling (Sec. 2.1)
 *   Sec. 3.1  departments share W_g^j, W_u^j, W_d^j; FACTORED expert (Eq. 4)
 *             d_i(g_i(x) * u_i(x)) with g_i = SiLU(A_g sigma(W_g x)),
 *             u_i = A_u sigma(W_u x), d_i(v) = W_d^T sigma(A_d^T v)
 *   Sec. 3.2  two-stage routing: department work once per collected token,
 *             then the private work per (expert, token), then W_d^T of the
 *             collected Z (oref_layer_two_stage)
 *   Sec. 3.3  group-limited top-k: at most k_dept departments per token
 *
 * SLICE form: each expert = department-shared SwiGLU slice (intermediate d_s)
 * plus a private SwiGLU slice (intermediate d_p), outputs summed.
 *
 * Readings where the paper is silent: ties in top-k go to the lower expert id;
 * expert e belongs to department floor(e / E_d); the group score of a
 * department is the maximum logit among its experts; softmax without
 * renormalisation divides by the sum over all n experts; the optional router
 * bias is added to the logits before both selection and weighting.
 */
#include "deamoe_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

int oref_num_threads(void) { return omp_get_max_threads(); }
void oref_set_num_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/* ---------------------------------------------------------------- decoding */

static double bf16_value(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* OCP e4m3fn: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; exponent
 * field 0 is subnormal; S.1111.111 is NaN; there is no infinity. */
double oref_fp8_value(uint8_t code) {
  int s = code >> 7, e = (code >> 3) & 15, m = code & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexp((double)m / 8.0, -6);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return s ? -v : v;
}

void oref_fp8_decode(const uint8_t *codes, size_t count, double *out) {
  for (size_t i = 0; i < count; ++i) out[i] = oref_fp8_value(codes[i]);
}

/* A stack of [R, C] matrices in one storage format. */
typedef struct {
  const void *p;
  const float *scale;   /* fp8 only: [stack, ceil(R/128), ceil(C/128)] */
  int dtype, R, C;
} mat_t;

static double mat_at(const mat_t *M, int idx, int r, int c) {
  size_t off = ((size_t)idx * M->R + r) * M->C + c;
  switch (M->dtype) {
    case OREF_F32: return (double)((const float *)M->p)[off];
    case OREF_BF16: return bf16_value(((const uint16_t *)M->p)[off]);
    default: {
      int rb = (M->R + 127) / 128, cb = (M->C + 127) / 128;
      double s = M->scale[((size_t)idx * rb + r / 128) * cb + c / 128];
      return oref_fp8_value(((const uint8_t *)M->p)[off]) * s;
    }
  }
}

/* out[r] = sum_c M[idx][r][c] * v[c], c ascending, fp64. */
static void matvec(const mat_t *M, int idx, const double *v, double *out) {
  for (int r = 0; r < M->R; ++r) {
    double acc = 0.0;
    for (int c = 0; c < M->C; ++c) acc += mat_at(M, idx, r, c) * v[c];
    out[r] = acc;
  }
}

static double silu(double v) { return v / (1.0 + exp(-v)); }

/* GeLU in its exact form v * Phi(v), Phi the standard normal CDF. */
static double gelu(double v) { return 0.5 * v * (1.0 + erf(v / sqrt(2.0))); }

/* The interface nonlinearity sigma of the FACTORED form (Sec. 3.1; the
 * variants compared in Sec. 3.4) applied in place to one d-vector.  SiLU,
 * GeLU and the identity act per element; RMSNorm divides the whole vector by
 * its root mean square (plus OREF_RMS_EPS), with unit gain. */
static void sigma_vec(const oref_config *cfg, double *v, int d) {
  if (cfg->sigma == OREF_SIGMA_NONE) return;
  if (cfg->sigma == OREF_SIGMA_RMSNORM) {
    double ss = 0.0;
    for (int r = 0; r < d; ++r) ss += v[r] * v[r];
    const double inv = 1.0 / sqrt(ss / d + OREF_RMS_EPS);
    for (int r = 0; r < d; ++r) v[r] *= inv;
    return;
  }
  for (int r = 0; r < d; ++r) v[r] = cfg->sigma == OREF_SIGMA_GELU ? gelu(v[r]) : silu(v[r]);
}

static void load_token(const oref_config *cfg, const void *x, int t, double *out) {
  int h = cfg->hidden;
  for (int c = 0; c < h; ++c) {
    size_t off = (size_t)t * h + c;
    out[c] = cfg->act_dtype == OREF_F32 ? (double)((const float *)x)[off]
                                        : bf16_value(((const uint16_t *)x)[off]);
  }
}

static int check_config(const oref_config *c) {
  if (c->hidden <= 0 || c->n_experts <= 0 || c->n_depts <= 0) return -1;
  if (c->n_experts % c->n_depts) return -1;
  if (c->top_k <= 0 || c->top_k > c->n_experts) return -1;
  if (c->top_k_dept < 0 || c->top_k_dept > c->n_depts) return -1;
  if (c->top_k_dept > 0 && c->top_k > c->top_k_dept * (c->n_experts / c->n_depts)) return -1;
  if (c->d_shared <= 0 || c->d_private < 0 || c->d_shared_expert < 0) return -1;
  if (c->sigma < OREF_SIGMA_SILU || c->sigma > OREF_SIGMA_RMSNORM) return -1;
  if (c->dept_cover != 0 && c->dept_cover != 1) return -1;
  if (c->dept_cover && (c->top_k_dept == 0 || c->top_k < c->top_k_dept)) return -1;
  return 0;
}

/* ------------------------------------------------------------------ routing */

/* a ranks before b: larger logit, then smaller index. */
static int better(float la, int a, float lb, int b) { return la > lb || (la == lb && a < b); }

/* Eq. 2 for one token: l[n] are the fp32 (biased) logits.  Writes the k
 * selected ids in rank order and their weights (Sec. 2.1: softmax
 * normalisation and scaling). */
static void route_one(const oref_config *cfg, const float *l, int32_t *ids, double *w) {
  int n = cfg->n_experts, m = cfg->n_depts, k = cfg->top_k, E = n / m;
  char *allowed = malloc(n), *taken = calloc(n, 1);
  memset(allowed, 1, n);
  if (cfg->top_k_dept > 0) {
    /* group-limited top-k: keep the k_dept departments with the largest group
       score (max logit of the department), ties to the lower department id. */
    float *gs = malloc(sizeof(float) * m);
    char *keep = calloc(m, 1);
    for (int j = 0; j < m; ++j) {
      gs[j] = l[j * E];
      for (int e = j * E + 1; e < (j + 1) * E; ++e) if (l[e] > gs[j]) gs[j] = l[e];
    }
    for (int r = 0; r < cfg->top_k_dept; ++r) {
      int best = -1;
      for (int j = 0; j < m; ++j)
        if (!keep[j] && (best < 0 || better(gs[j], j, gs[best], best))) best = j;
      keep[best] = 1;
    }
    for (int e = 0; e < n; ++e) allowed[e] = keep[e / E];
    free(gs);
    free(keep);
  }
  for (int r = 0; r < k; ++r) {
    int best = -1;
    for (int e = 0; e < n; ++e)
      if (allowed[e] && !taken[e] && (best < 0 || better(l[e], e, l[best], best))) best = e;
    taken[best] = 1;
    ids[r] = best;
  }
  if (cfg->dept_cover) {
    /* strict coverage (Sec. 3.4): while the selection spans fewer than k_dept
       departments, the lowest-ranked selected expert whose department keeps
       another selected expert gives way to the best allowed expert of a
       department not yet covered; the selection is then put back in rank
       order.  Each round covers one more department. */
    int *cnt = malloc(sizeof(int) * m);
    for (;;) {
      int D = 0;
      memset(cnt, 0, sizeof(int) * m);
      for (int r = 0; r < k; ++r) cnt[ids[r] / E] += 1;
      for (int j = 0; j < m; ++j) D += cnt[j] > 0;
      if (D >= cfg->top_k_dept) break;
      int add = -1, victim = -1;
      for (int e = 0; e < n; ++e)
        if (allowed[e] && cnt[e / E] == 0 && (add < 0 || better(l[e], e, l[add], add))) add = e;
      for (int r = k - 1; r >= 0 && victim < 0; --r)
        if (cnt[ids[r] / E] >= 2) victim = r;
      ids[victim] = add;
      for (int r = 1; r < k; ++r)
        for (int q = r; q > 0 && better(l[ids[q]], ids[q], l[ids[q - 1]], ids[q - 1]); --q) {
          const int tmp = ids[q];
          ids[q] = ids[q - 1];
          ids[q - 1] = tmp;
        }
    }
    free(cnt);
  }
  if (cfg->score == OREF_SOFTMAX) {
    double mx = -INFINITY, den = 0.0;
    if (cfg->renorm) {
      for (int r = 0; r < k; ++r) mx = fmax(mx, (double)l[ids[r]]);
      for (int r = 0; r < k; ++r) den += exp((double)l[ids[r]] - mx);
    } else {
      for (int e = 0; e < n; ++e) mx = fmax(mx, (double)l[e]);
      for (int e = 0; e < n; ++e) den += exp((double)l[e] - mx);
    }
    for (int r = 0; r < k; ++r) w[r] = exp((double)l[ids[r]] - mx) / den;
  } else {
    double den = 0.0;
    for (int r = 0; r < k; ++r) {
      w[r] = 1.0 / (1.0 + exp(-(double)l[ids[r]]));
      den += w[r];
    }
    if (cfg->renorm)
      for (int r = 0; r < k; ++r) w[r] /= den;
  }
  for (int r = 0; r < k; ++r) w[r] *= cfg->route_scale;
  free(allowed);
  free(taken);
}

/* fp32 logits of one token: the dot product in fp64 rounded once to fp32,
 * then the bias with one fp32 add. */
static void token_logits(const oref_config *cfg, const void *x, const void *router,
                         const float *logits_in, const float *bias, int t, float *l) {
  int n = cfg->n_experts, h = cfg->hidden;
  if (logits_in) {
    for (int e = 0; e < n; ++e) l[e] = logits_in[(size_t)t * n + e];
  } else {
    double *xv = malloc(sizeof(double) * h);
    mat_t R = {router, NULL, cfg->act_dtype, n, h};
    load_token(cfg, x, t, xv);
    for (int e = 0; e < n; ++e) {
      double acc = 0.0;
      for (int c = 0; c < h; ++c) acc += mat_at(&R, 0, e, c) * xv[c];
      l[e] = (float)acc;
    }
    free(xv);
  }
  if (bias)
    for (int e = 0; e < n; ++e) {
      float b = bias[e];
      l[e] = l[e] + b;
    }
}

int oref_route(const oref_config *cfg, int T, const void *x, const void *router,
               const float *logits_in, const float *bias, oref_routing *out) {
  if (check_config(cfg) || T < 0) return -1;
  int n = cfg->n_experts, m = cfg->n_depts, k = cfg->top_k, E = n / m;
  for (int t = 0; t < T; ++t) {
    float *l = out->logits + (size_t)t * n;
    int32_t *ids = out->topk_ids + (size_t)t * k;
    double *w = out->topk_w + (size_t)t * k;
    token_logits(cfg, x, router, logits_in, bias, t, l);
    route_one(cfg, l, ids, w);
    /* Sec. 3.2 stage one: the distinct departments of the selected experts,
       ascending, each with the summed weight of its selected experts. */
    int nd = 0;
    for (int j = 0; j < m; ++j) {
      double pj = 0.0;
      int hit = 0;
      for (int r = 0; r < k; ++r)
        if (ids[r] / E == j) { hit = 1; pj += w[r]; }
      if (hit) {
        out->tok_depts[(size_t)t * k + nd] = j;
        out->tok_dept_w[(size_t)t * k + nd] = pj;
        ++nd;
      }
    }
    for (int r = nd; r < k; ++r) {
      out->tok_depts[(size_t)t * k + r] = -1;
      out->tok_dept_w[(size_t)t * k + r] = 0.0;
    }
    out->tok_ndept[t] = nd;
  }
  /* X^j: the tokens of each department, ascending; likewise per expert. */
  int pos = 0;
  for (int j = 0; j < m; ++j) {
    out->dept_offset[j] = pos;
    for (int t = 0; t < T; ++t)
      for (int r = 0; r < out->tok_ndept[t]; ++r)
        if (out->tok_depts[(size_t)t * k + r] == j) out->dept_tokens[pos++] = t;
    out->dept_count[j] = pos - out->dept_offset[j];
  }
  out->dept_offset[m] = pos;
  pos = 0;
  for (int e = 0; e < n; ++e) {
    out->exp_offset[e] = pos;
    for (int t = 0; t < T; ++t)
      for (int r = 0; r < k; ++r)
        if (out->topk_ids[(size_t)t * k + r] == e) out->exp_tokens[pos++] = t;
    out->exp_count[e] = pos - out->exp_offset[e];
  }
  out->exp_offset[n] = pos;
  return 0;
}

/* ---------------------------------------------------------------- experts */

typedef struct {
  mat_t M[9];
} wset_t;

static void make_wset(const oref_config *cfg, const oref_weights *w, wset_t *s) {
  int h = cfg->hidden, d = cfg->d_shared, p = cfg->d_private, e = cfg->d_shared_expert;
  int wt = cfg->w_dtype;
  mat_t z = {NULL, NULL, wt, 0, 0};
  for (int i = 0; i < 9; ++i) s->M[i] = z;
  s->M[0] = (mat_t){w->mat[0], w->scale[0], wt, d, h};
  s->M[1] = (mat_t){w->mat[1], w->scale[1], wt, d, h};
  s->M[2] = (mat_t){w->mat[2], w->scale[2], wt, h, d};
  if (cfg->form == OREF_FACTORED) {
    s->M[3] = (mat_t){w->mat[3], w->scale[3], wt, d, d};
    s->M[4] = (mat_t){w->mat[4], w->scale[4], wt, d, d};
    s->M[5] = (mat_t){w->mat[5], w->scale[5], wt, d, d};
  } else if (p > 0) {
    s->M[3] = (mat_t){w->mat[3], w->scale[3], wt, p, h};
    s->M[4] = (mat_t){w->mat[4], w->scale[4], wt, p, h};
    s->M[5] = (mat_t){w->mat[5], w->scale[5], wt, h, p};
  }
  if (e > 0) {
    s->M[6] = (mat_t){w->mat[6], w->scale[6], wt, e, h};
    s->M[7] = (mat_t){w->mat[7], w->scale[7], wt, e, h};
    s->M[8] = (mat_t){w->mat[8], w->scale[8], wt, h, e};
  }
}

/* Eq. 1: out = Wd (SiLU(Wg x) * (Wu x)), Wd stored [h, f]. */
static void swiglu(const mat_t *G, const mat_t *U, const mat_t *D, int idx,
                   const double *x, double *out) {
  int f = G->R;
  double *g = malloc(sizeof(double) * f), *u = malloc(sizeof(double) * f);
  matvec(G, idx, x, g);
  matvec(U, idx, x, u);
  for (int r = 0; r < f; ++r) g[r] = silu(g[r]) * u[r];
  matvec(D, idx, g, out);
  free(g);
  free(u);
}

/* One expert i (department j = i / E_d) on one token, naive. */
static void expert_out(const oref_config *cfg, const wset_t *s, int i, const double *x,
                       double *out) {
  int h = cfg->hidden, d = cfg->d_shared, j = i / (cfg->n_experts / cfg->n_depts);
  if (cfg->form == OREF_FACTORED) {
    /* Eq. 4 with the projections of Sec. 3.1. */
    double *G = malloc(sizeof(double) * d), *U = malloc(sizeof(double) * d);
    double *a = malloc(sizeof(double) * d), *b = malloc(sizeof(double) * d);
    matvec(&s->M[0], j, x, G);
    matvec(&s->M[1], j, x, U);
    sigma_vec(cfg, G, d);
    sigma_vec(cfg, U, d);
    matvec(&s->M[3], i, G, a);                     /* A_g sigma(W_g x)            */
    matvec(&s->M[4], i, U, b);                     /* A_u sigma(W_u x)            */
    for (int r = 0; r < d; ++r) a[r] = silu(a[r]) * b[r];   /* g_i(x) * u_i(x)   */
    matvec(&s->M[5], i, a, b);                     /* (A_d)^T v                   */
    sigma_vec(cfg, b, d);                          /* sigma((A_d)^T v)            */
    matvec(&s->M[2], j, b, out);                   /* (W_d)^T sigma(...)          */
    free(G); free(U); free(a); free(b);
  } else {
    swiglu(&s->M[0], &s->M[1], &s->M[2], j, x, out);
    if (cfg->d_private > 0) {
      double *q = malloc(sizeof(double) * h);
      swiglu(&s->M[3], &s->M[4], &s->M[5], i, x, q);
      for (int c = 0; c < h; ++c) out[c] += q[c];
      free(q);
    }
  }
}

int oref_layer_naive(const oref_config *cfg, int T, const void *x, const oref_weights *w,
                     const float *logits_in, const float *bias,
                     int n_sel, const int32_t *sel, double *y) {
  if (check_config(cfg) || T < 0) return -1;
  if (!sel) n_sel = T;
  for (int q = 0; q < n_sel; ++q)
    if (sel && (sel[q] < 0 || sel[q] >= T)) return -1;
  int h = cfg->hidden, n = cfg->n_experts, k = cfg->top_k;
  wset_t s;
  make_wset(cfg, w, &s);
#pragma omp parallel for schedule(dynamic, 1)
  for (int q = 0; q < n_sel; ++q) {
    int t = sel ? sel[q] : q;
    double *xv = malloc(sizeof(double) * h), *o = malloc(sizeof(double) * h);
    float *l = malloc(sizeof(float) * n);
    int32_t *ids = malloc(sizeof(int32_t) * k);
    double *p = malloc(sizeof(double) * k), *yt = y + (size_t)q * h;
    load_token(cfg, x, t, xv);
    token_logits(cfg, x, w->router, logits_in, bias, t, l);
    route_one(cfg, l, ids, p);
    for (int c = 0; c < h; ++c) yt[c] = 0.0;
    for (int r = 0; r < k; ++r) {                  /* Eq. 3 */
      expert_out(cfg, &s, ids[r], xv, o);
      for (int c = 0; c < h; ++c) yt[c] += p[r] * o[c];
    }
    if (cfg->d_shared_expert > 0) {                /* always-on shared expert, weight 1 */
      swiglu(&s.M[6], &s.M[7], &s.M[8], 0, xv, o);
      for (int c = 0; c < h; ++c) yt[c] += o[c];
    }
    free(xv); free(o); free(l); free(ids); free(p);
  }
  return 0;
}

/* ------------------------------------------------------ two-stage (Sec. 3.2) */

/* p_{t,e}: the routing weight of expert e for token t (0 when not selected). */
static double expert_weight(const oref_routing *R, int k, int t, int e) {
  for (int r = 0; r < k; ++r)
    if (R->topk_ids[(size_t)t * k + r] == e) return R->topk_w[(size_t)t * k + r];
  return 0.0;
}

int oref_layer_two_stage(const oref_config *cfg, int T, const void *x, const oref_weights *w,
                         const float *logits_in, const float *bias, double *y) {
  if (check_config(cfg) || T < 0) return -1;
  int h = cfg->hidden, n = cfg->n_experts, m = cfg->n_depts, k = cfg->top_k, E = n / m;
  int d = cfg->d_shared;
  size_t Tk = (size_t)(T > 0 ? T : 1) * k;
  oref_routing R;
  R.logits = malloc(sizeof(float) * (size_t)(T > 0 ? T : 1) * n);
  R.topk_ids = malloc(sizeof(int32_t) * Tk);
  R.topk_w = malloc(sizeof(double) * Tk);
  R.tok_depts = malloc(sizeof(int32_t) * Tk);
  R.tok_dept_w = malloc(sizeof(double) * Tk);
  R.tok_ndept = malloc(sizeof(int32_t) * (T > 0 ? T : 1));
  R.dept_count = malloc(sizeof(int32_t) * m);
  R.dept_offset = malloc(sizeof(int32_t) * (m + 1));
  R.dept_tokens = malloc(sizeof(int32_t) * Tk);
  R.exp_count = malloc(sizeof(int32_t) * n);
  R.exp_offset = malloc(sizeof(int32_t) * (n + 1));
  R.exp_tokens = malloc(sizeof(int32_t) * Tk);
  oref_route(cfg, T, x, w->router, logits_in, bias, &R);
  wset_t s;
  make_wset(cfg, w, &s);
  double *X = malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * h);
  for (int t = 0; t < T; ++t) load_token(cfg, x, t, X + (size_t)t * h);
  memset(y, 0, sizeof(double) * (size_t)T * h);
  double *o = malloc(sizeof(double) * h);
  if (cfg->form == OREF_SLICE) {
    for (int j = 0; j < m; ++j) {                    /* department work, once per token of X^j */
      for (int q = R.dept_offset[j]; q < R.dept_offset[j + 1]; ++q) {
        int t = R.dept_tokens[q];
        double Pj = 0.0;
        for (int r = 0; r < R.tok_ndept[t]; ++r)
          if (R.tok_depts[(size_t)t * k + r] == j) Pj = R.tok_dept_w[(size_t)t * k + r];
        swiglu(&s.M[0], &s.M[1], &s.M[2], j, X + (size_t)t * h, o);
        for (int c = 0; c < h; ++c) y[(size_t)t * h + c] += Pj * o[c];
      }
    }
    if (cfg->d_private > 0)
      for (int e = 0; e < n; ++e)                    /* private work per (expert, token) */
        for (int q = R.exp_offset[e]; q < R.exp_offset[e + 1]; ++q) {
          int t = R.exp_tokens[q];
          double pe = expert_weight(&R, k, t, e);
          swiglu(&s.M[3], &s.M[4], &s.M[5], e, X + (size_t)t * h, o);
          for (int c = 0; c < h; ++c) y[(size_t)t * h + c] += pe * o[c];
        }
  } else {
    double *Xg = malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * d);
    double *Xu = malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * d);
    double *Zj = malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * d);
    double *a = malloc(sizeof(double) * d), *b = malloc(sizeof(double) * d);
    for (int j = 0; j < m; ++j) {
      /* X_g^j = sigma(W_g^j X^j), X_u^j = sigma(W_u^j X^j): once per collected token */
      for (int q = R.dept_offset[j]; q < R.dept_offset[j + 1]; ++q) {
        int t = R.dept_tokens[q];
        matvec(&s.M[0], j, X + (size_t)t * h, Xg + (size_t)t * d);
        matvec(&s.M[1], j, X + (size_t)t * h, Xu + (size_t)t * d);
        sigma_vec(cfg, Xg + (size_t)t * d, d);
        sigma_vec(cfg, Xu + (size_t)t * d, d);
        memset(Zj + (size_t)t * d, 0, sizeof(double) * d);
      }
      /* each expert of the department on its share of the tokens:
         Y = SiLU(A_g X_g) * (A_u X_u), Z = sigma(A_d^T Y), collected with p */
      for (int e = j * E; e < (j + 1) * E; ++e)
        for (int q = R.exp_offset[e]; q < R.exp_offset[e + 1]; ++q) {
          int t = R.exp_tokens[q];
          double pe = expert_weight(&R, k, t, e);
          matvec(&s.M[3], e, Xg + (size_t)t * d, a);
          matvec(&s.M[4], e, Xu + (size_t)t * d, b);
          for (int r = 0; r < d; ++r) a[r] = silu(a[r]) * b[r];
          matvec(&s.M[5], e, a, b);
          sigma_vec(cfg, b, d);
          for (int r = 0; r < d; ++r) Zj[(size_t)t * d + r] += pe * b[r];
        }
      /* O^j = (W_d^j)^T Z^j */
      for (int q = R.dept_offset[j]; q < R.dept_offset[j + 1]; ++q) {
        int t = R.dept_tokens[q];
        matvec(&s.M[2], j, Zj + (size_t)t * d, o);
        for (int c = 0; c < h; ++c) y[(size_t)t * h + c] += o[c];
      }
    }
    free(Xg); free(Xu); free(Zj); free(a); free(b);
  }
  if (cfg->d_shared_expert > 0)
    for (int t = 0; t < T; ++t) {
      swiglu(&s.M[6], &s.M[7], &s.M[8], 0, X + (size_t)t * h, o);
      for (int c = 0; c < h; ++c) y[(size_t)t * h + c] += o[c];
    }
  free(o); free(X);
  free(R.logits); free(R.topk_ids); free(R.topk_w); free(R.tok_depts); free(R.tok_dept_w);
  free(R.tok_ndept); free(R.dept_count); free(R.dept_offset); free(R.dept_tokens);
  free(R.exp_count); free(R.exp_offset); free(R.exp_tokens);
  return 0;
}

/* ------------------------------------------------------------- accounting */

static int64_t matrix_bytes(int w_dtype, int64_t R, int64_t C) {
  int64_t wb = w_dtype == OREF_F32 ? 4 : w_dtype == OREF_BF16 ? 2 : 1;
  int64_t b = R * C * wb;
  if (w_dtype == OREF_FP8) b += ((R + 127) / 128) * ((C + 127) / 128) * 4;
  return b;
}

int64_t oref_step_weight_bytes(const oref_config *cfg, const int32_t *dept_count,
                               const int32_t *exp_count) {
  int64_t h = cfg->hidden, d = cfg->d_shared, p = cfg->d_private, e = cfg->d_shared_expert;
  int wt = cfg->w_dtype;
  int64_t act_b = cfg->act_dtype == OREF_F32 ? 4 : 2;
  int64_t b = (int64_t)cfg->n_experts * h * act_b;      /* router */
  int64_t dept = 3 * matrix_bytes(wt, d, h);
  int64_t priv = 0;
  if (cfg->form == OREF_FACTORED) priv = 3 * matrix_bytes(wt, d, d);
  else if (p > 0) priv = 3 * matrix_bytes(wt, p, h);
  for (int j = 0; j < cfg->n_depts; ++j) if (dept_count[j] > 0) b += dept;
  for (int i = 0; i < cfg->n_experts; ++i) if (exp_count[i] > 0) b += priv;
  if (e > 0) b += 3 * matrix_bytes(wt, e, h);
  return b;
}
