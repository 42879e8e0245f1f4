/* deamoe.h -- C ABI of the MI355X (gfx950) DeaMoE decode-layer library.
 *
 * What is computed (the paper's notation; no code of the paper is used):
 *   Router (Sec. 2.1, Eq. 2): logits l = W_r x (+ optional bias), the top-k
 *     experts S(x) by (logit desc, expert id asc), optionally limited to the
 *     top_k_dept departments by group score (Sec. 3.3, group-limited top-k);
 *     routing weights p after softmax or sigmoid normalisation and scaling
 *     (Sec. 2.1, the sentence after Eq. 3).
 *   Departments (Sec. 3.1): n experts in m departments of E_d = n / m
 *     consecutive experts; expert e belongs to department e / E_d.
 *   Expert output, SLICE form: department-shared SwiGLU slice (intermediate
 *     d_shared) plus a private SwiGLU slice (intermediate d_private), summed.
 *   Expert output, FACTORED form (Sec. 3.1, Eq. 4):
 *     d_i(g_i(x) * u_i(x)), g_i = SiLU(A_g sigma(W_g x)), u_i = A_u sigma(W_u x),
 *     d_i(v) = W_d^T sigma(A_d^T v), sigma = SiLU, identity, GeLU or RMSNorm.
 *   Layer output (Eq. 3): y = sum_{i in S(x)} p_i expert_i(x), plus an optional
 *     always-on shared SwiGLU expert with weight 1.
 *   Two-stage evaluation (Sec. 3.2): each touched department's shared
 *     matrices are streamed once per step for all of its tokens (X^j), each
 *     touched expert's private matrices once for its tokens, then the weighted
 *     combine.  The result equals the per-expert definition up to rounding.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers owned by the caller, except where a
 *     parameter says "host".  `stream` is a hipStream_t (NULL = null stream).
 *   - All device work is enqueued on `stream`; no call allocates device or
 *     host memory, frees, or synchronises; every call is hipGraph-capturable.
 *   - Arguments are validated on the host before anything is enqueued; an
 *     invalid call returns a negative DEAMOE_ERR_* code and enqueues nothing.
 *     A launch failure returns DEAMOE_ERR_HIP.
 *   - T == 0 returns DEAMOE_OK and enqueues nothing once the configuration
 *     is valid (tensor pointers may then be NULL).
 *   - Identical inputs give bit-identical outputs (no atomics in any sum).
 *   - The library holds no state: calls on different streams are independent
 *     as long as each uses its own workspace and outputs.
 *
 * Layouts: every matrix is row-major [out, in] and stacked over departments
 * or experts.  Activations x and y are row-major [T, hidden].
 */
#ifndef DEAMOE_H
#define DEAMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define DEAMOE_OK 0
#define DEAMOE_ERR_INVALID (-1)      /* bad argument or inconsistent config        */
#define DEAMOE_ERR_UNSUPPORTED (-2)  /* valid but outside this build's limits      */
#define DEAMOE_ERR_WORKSPACE (-3)    /* workspace missing or too small             */
#define DEAMOE_ERR_HIP (-4)          /* a HIP launch failed                        */

/* element types */
#define DEAMOE_F32 0
#define DEAMOE_BF16 1
#define DEAMOE_FP8_E4M3_B128 2  /* OCP e4m3fn codes + one fp32 scale per 128x128 block */

/* expert form */
#define DEAMOE_FORM_SLICE 0
#define DEAMOE_FORM_FACTORED 1

/* routing score */
#define DEAMOE_SCORE_SOFTMAX 0
#define DEAMOE_SCORE_SIGMOID 1

/* interface nonlinearity sigma of the FACTORED form (Sec. 3.1; the
 * alternatives are the ones compared in Sec. 3.4) */
#define DEAMOE_SIGMA_SILU 0
#define DEAMOE_SIGMA_NONE 1      /* identity                                            */
#define DEAMOE_SIGMA_GELU 2      /* v * Phi(v), the exact (erf) form                     */
#define DEAMOE_SIGMA_RMSNORM 3   /* v / sqrt(mean(v^2) + 1e-6) over the d-vector, unit gain */

/* Limits of this build (DEAMOE_ERR_UNSUPPORTED beyond them). */
#define DEAMOE_MAX_TOKENS 128
#define DEAMOE_MAX_EXPERTS 2048
#define DEAMOE_MAX_TOPK 32
/* every width (hidden, d_shared, d_private, d_shared_expert) is at most this
 * many columns, so that the token rows one stage reads lie within 4 GiB of
 * their buffer (32-bit row offsets in the expert stages) */
#define DEAMOE_MAX_WIDTH 65536
/* fp8 weights: every contraction length (hidden, d_shared, d_private,
 * d_shared_expert) is at most this many columns (64 scale blocks) */
#define DEAMOE_MAX_FP8_K 8192

typedef struct {
  int32_t hidden;           /* h                                                        */
  int32_t n_experts;        /* n                                                        */
  int32_t n_depts;          /* m, divides n                                             */
  int32_t top_k;            /* k experts per token (Eq. 2)                              */
  int32_t top_k_dept;       /* at most this many departments per token; 0 = no limit    */
  int32_t d_shared;         /* SLICE: department slice intermediate; FACTORED: d        */
  int32_t d_private;        /* SLICE: private slice intermediate (0 = none);
                               FACTORED: ignored (private matrices are d x d)           */
  int32_t d_shared_expert;  /* always-on shared expert intermediate; 0 = none           */
  int32_t form;             /* DEAMOE_FORM_*                                            */
  int32_t score;            /* DEAMOE_SCORE_*                                           */
  int32_t renorm;           /* 1: weights renormalised over the selected k experts      */
  int32_t sigma;            /* DEAMOE_SIGMA_* (FACTORED only)                           */
  float route_scale;        /* routing weights are multiplied by this                   */
  int32_t w_dtype;          /* expert weight type: DEAMOE_F32 | BF16 | FP8_E4M3_B128    */
  int32_t act_dtype;        /* x, y and router weight type: DEAMOE_F32 | DEAMOE_BF16    */
  int32_t max_tokens;       /* largest T the workspace is sized for (<= 128)            */
  int32_t dept_cover;       /* 0: top_k_dept is an upper bound (group-limited top-k).
                               1: strict coverage (Sec. 3.4): while a token's k experts
                               span fewer than top_k_dept departments, its lowest-ranked
                               expert whose department holds another selected expert is
                               replaced by the best expert of a kept department not yet
                               covered.  Needs top_k_dept > 0 and top_k >= top_k_dept. */
} deamoe_config;

/* Expert weights.  Shapes ([out, in], stacked):
 *   router      [n, h]           act_dtype
 *   dept_gate   [m, d_s, h]      W_g^j
 *   dept_up     [m, d_s, h]      W_u^j
 *   dept_down   [m, h, d_s]      (W_d^j)^T
 *   SLICE:    priv_gate [n, d_p, h], priv_up [n, d_p, h], priv_down [n, h, d_p]
 *             (NULL when d_private == 0)
 *   FACTORED: priv_gate = A_g [n, d, d], priv_up = A_u [n, d, d],
 *             priv_down = (A_d)^T [n, d, d]
 *   se_gate [d_se, h], se_up [d_se, h], se_down [h, d_se] (NULL when d_se == 0)
 *   scale[0..8]: fp8 only, one fp32 per 128 x 128 block of each matrix, in the
 *     order dept_gate, dept_up, dept_down, priv_gate, priv_up, priv_down,
 *     se_gate, se_up, se_down; each [stack, ceil(out/128), in/128].
 * All pointers 16-byte aligned. */
typedef struct {
  const void *router;
  const void *dept_gate, *dept_up, *dept_down;
  const void *priv_gate, *priv_up, *priv_down;
  const void *se_gate, *se_up, *se_down;
  const float *scale[9];
} deamoe_weights;

/* Routing results (device arrays, caller-allocated).
 *   topk_ids   [T, k]  selected experts in rank order
 *   topk_w     [T, k]  routing weights p (fp32)
 *   tok_depts  [T, k]  distinct departments of the token, ascending, -1 padded
 *   tok_dept_w [T, k]  P_{t,j}: summed weight of the token's experts in each
 *   tok_ndept  [T]     number of distinct departments
 *   dept_count [m], dept_offset [m+1], dept_tokens [T*k]: the token list X^j of
 *     every department (ascending token index), CSR
 *   exp_count [n], exp_offset [n+1], exp_tokens [T*k]: the same per expert
 *   logits     [T, n]  fp32 logits after the bias (may be NULL) */
typedef struct {
  int32_t *topk_ids;
  float *topk_w;
  int32_t *tok_depts;
  float *tok_dept_w;
  int32_t *tok_ndept;
  int32_t *dept_count, *dept_offset, *dept_tokens;
  int32_t *exp_count, *exp_offset, *exp_tokens;
  float *logits;
} deamoe_routing;

/* Human-readable text of a status code (static storage). */
const char *deamoe_status_string(int status);

/* Host.  Bytes of device workspace that deamoe_route / deamoe_layer_forward /
 * deamoe_baseline_forward need for up to cfg->max_tokens tokens. */
int deamoe_workspace_bytes(const deamoe_config *cfg, size_t *bytes);

/* Router only (Eq. 2 and the department bookkeeping of Sec. 3.2).
 * x [T, h] act_dtype; router_w [n, h] act_dtype.  logits_in: optional fp32
 * [T, n] logits used instead of W_r x.  router_bias: optional fp32 [n] added
 * to the logits (one fp32 add after the complete dot product) before both
 * selection and weighting.  `out` receives every array of deamoe_routing
 * (out->logits may be NULL). */
int deamoe_route(const deamoe_config *cfg, int32_t T, const void *x, const void *router_w,
                 const float *logits_in, const float *router_bias, deamoe_routing *out,
                 void *ws, size_t ws_bytes, void *stream);

/* The DeaMoE layer (Eq. 3 over SLICE or FACTORED experts, two-stage order).
 * y [T, h] act_dtype.  routing_out: optional, receives the routing (NULL: the
 * routing lives in the workspace). */
int deamoe_layer_forward(const deamoe_config *cfg, int32_t T, const void *x,
                         const deamoe_weights *w, const float *logits_in,
                         const float *router_bias, deamoe_routing *routing_out, void *y,
                         void *ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call as deamoe_layer_forward, same kernels and results, with the workspace
 * taken from a library-owned device array of DEAMOE_SCRATCH_BYTES per GPU
 * (the current device's), held until the process ends.  Nothing is allocated
 * or freed.  A configuration whose workspace (deamoe_workspace_bytes, sized
 * for cfg->max_tokens) exceeds DEAMOE_SCRATCH_BYTES returns
 * DEAMOE_ERR_WORKSPACE before any HIP call.  The first call on a device
 * resolves that device's array address (DEAMOE_ERR_HIP if that fails).
 * Every call on one GPU shares its array: calls that overlap in time on one
 * GPU (other streams, other host threads) race and must be serialised by the
 * caller.  No part of the array needs clearing between calls; each call
 * writes everything it reads.  `stream` must belong to the current device. */
#define DEAMOE_SCRATCH_BYTES (64u << 20)
int deamoe_layer_forward_noalloc(const deamoe_config *cfg, int32_t T, const void *x,
                                 const deamoe_weights *w, const float *logits_in,
                                 const float *router_bias, deamoe_routing *routing_out, void *y,
                                 void *stream);

/* The same with caller-created hipEvent_t handles recorded on `stream` at the
 * stage boundaries, for timing: events[0] before the router, then one after
 * each launched kernel in order (SLICE: router GEMV, route, gate/up, down,
 * combine; FACTORED: router GEMV, route, department gate/up, private gate/up,
 * private down, Z collect, department down, combine).  Small batches may
 * run the last down stage and the combine as one kernel
 * (deamoe_trace_points gives the count).  n_events may be
 * smaller than that count; NULL / 0 records nothing.  With injected logits
 * the router GEMV is not launched and has no boundary. */
int deamoe_layer_forward_traced(const deamoe_config *cfg, int32_t T, const void *x,
                                const deamoe_weights *w, const float *logits_in,
                                const float *router_bias, deamoe_routing *routing_out, void *y,
                                void *ws, size_t ws_bytes, void *stream, void *const *events,
                                int32_t n_events);

/* Host: the number of events deamoe_layer_forward_traced records for a batch
 * of T tokens with computed logits (1 + one per stage listed above).  Returns
 * DEAMOE_ERR_INVALID for a NULL pointer, T < 1 or T > max_tokens. */
int deamoe_trace_points(const deamoe_config *cfg, int32_t T, int32_t *n_events);

/* Vanilla MoE of Eq. 1-3 at the same shape, the comparator for speedups:
 * cfg must describe one expert per department (n_depts == n_experts), no
 * private part (d_private == 0), SLICE form; d_shared is the expert
 * intermediate size f and dept_* hold the n experts' matrices. */
int deamoe_baseline_forward(const deamoe_config *cfg, int32_t T, const void *x,
                            const deamoe_weights *w, const float *logits_in,
                            const float *router_bias, deamoe_routing *routing_out, void *y,
                            void *ws, size_t ws_bytes, void *stream);

/* Host.  Algorithmic HBM bytes of one step: the per-step weight loading that
 * Sec. 3.3 compares between DeaMoE and vanilla MoE (Fig. 2), with the router
 * counted as that comparison's budget accounting counts it.  Given the
 * realised routing counts (host arrays dept_count [m], exp_count [n]):
 * every touched department's and expert's matrices once (fp8: plus block
 * scales), the router, the shared expert -> *weight_bytes; *total_bytes adds
 * x read and y written (T x h activations each).  Either output may be NULL.
 * DEAMOE_ERR_INVALID for a NULL count array or T < 0. */
int deamoe_loaded_bytes(const deamoe_config *cfg, int32_t T, const int32_t *dept_count,
                        const int32_t *exp_count, int64_t *weight_bytes, int64_t *total_bytes);

#ifdef __cplusplus
}
#endif
#endif /* DEAMOE_H */
