/* DeaMoE decode-layer oracle: TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU evaluation of what the DeaMoE layer
 * computes, written from the paper (Sec. 2.1 Eq. 1-3; Sec. 3.1 Eq. 4; Sec. 3.2).
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * use it.  It shares no code with the HIP library: separate header, separate
 * types, separate source.
 *
 * Arithmetic: every dot product is accumulated in fp64, one term at a time in
 * ascending index order.  The router logit that decides top-k is rounded to
 * fp32 (the precision the GPU decides in) and the optional bias is added with
 * one fp32 add; everything after that is fp64.
 *
 * All pointers are HOST pointers.  Weights are read in their storage format
 * (fp32, bf16 bit patterns, or e4m3 codes with fp32 128x128 block scales) and
 * upcast exactly on every access.
 */
#ifndef DEAMOE_ORACLE_H
#define DEAMOE_ORACLE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OREF_F32 = 0, OREF_BF16 = 1, OREF_FP8 = 2 };
enum { OREF_SLICE = 0, OREF_FACTORED = 1 };
enum { OREF_SOFTMAX = 0, OREF_SIGMOID = 1 };
enum { OREF_SIGMA_SILU = 0, OREF_SIGMA_NONE = 1, OREF_SIGMA_GELU = 2, OREF_SIGMA_RMSNORM = 3 };

/* RMSNorm variant of sigma: v / sqrt(mean(v^2) + eps) over the d-vector, unit gain. */
#define OREF_RMS_EPS 1e-6

typedef struct {
  int hidden, n_experts, n_depts, top_k, top_k_dept;
  int d_shared, d_private, d_shared_expert;
  int form, score, renorm, sigma;
  double route_scale;
  int w_dtype, act_dtype;
  int dept_cover;           /* 1: strict department coverage (Sec. 3.4), needs
                               top_k_dept > 0 and top_k >= top_k_dept */
} oref_config;

/* Weight storage, row-major [out, in], stacked over departments / experts.
 *   router     [n, h]                 act dtype
 *   dept_gate  [m, d, h]   W_g^j      dept_up [m, d, h]  W_u^j
 *   dept_down  [m, h, d]   (W_d^j)^T
 *   SLICE:     priv_gate/priv_up [n, d_p, h], priv_down [n, h, d_p]
 *   FACTORED:  priv_gate = A_g^i [n, d, d], priv_up = A_u^i [n, d, d],
 *              priv_down = (A_d^i)^T [n, d, d]
 *   se_gate/se_up [d_se, h], se_down [h, d_se]   (NULL when d_se == 0)
 *   scale[9]:  fp8 only, same order as the nine expert tensors, each
 *              [stack, ceil(out/128), ceil(in/128)] fp32. */
typedef struct {
  const void *router;
  const void *mat[9];       /* dept_gate, dept_up, dept_down, priv_gate, priv_up,
                               priv_down, se_gate, se_up, se_down */
  const float *scale[9];
} oref_weights;

/* Routing result of Eq. 2 plus the department bookkeeping of Sec. 3.2. */
typedef struct {
  float   *logits;       /* [T, n] fp32 logits after the optional bias        */
  int32_t *topk_ids;     /* [T, k] in selection order (logit desc, id asc)    */
  double  *topk_w;       /* [T, k] routing weights p_i                        */
  int32_t *tok_depts;    /* [T, k] ascending distinct departments, -1 padded  */
  double  *tok_dept_w;   /* [T, k] P_{t,j} = sum of p_i over the department   */
  int32_t *tok_ndept;    /* [T]                                               */
  int32_t *dept_count, *dept_offset, *dept_tokens;   /* [m], [m+1], [T*k]      */
  int32_t *exp_count, *exp_offset, *exp_tokens;      /* [n], [n+1], [T*k]      */
} oref_routing;

/* Threads the token loops of oref_layer_naive may use (OpenMP); the setter
 * changes it for later calls from the calling thread. */
int oref_num_threads(void);
void oref_set_num_threads(int n);

/* e4m3fn (OCP) code -> value. */
double oref_fp8_value(uint8_t code);
void oref_fp8_decode(const uint8_t *codes, size_t count, double *out);

/* Eq. 2 routing over all T tokens.  logits_in (fp32 [T, n]) replaces the
 * computed logits when non-NULL; bias (fp32 [n]) is added to either.
 * Returns 0, or -1 on an invalid configuration. */
int oref_route(const oref_config *cfg, int T, const void *x, const void *router,
               const float *logits_in, const float *bias, oref_routing *out);

/* Naive layer output (Eq. 3 over Eq. 1 / Eq. 4 per selected expert) for the
 * tokens listed in sel[0..n_sel) (all T tokens when sel == NULL, n_sel = T).
 * Routing is recomputed per token.  y: [n_sel, h] fp64. */
int oref_layer_naive(const oref_config *cfg, int T, const void *x, const oref_weights *w,
                     const float *logits_in, const float *bias,
                     int n_sel, const int32_t *sel, double *y);

/* The same layer evaluated in the paper's two-stage order (Sec. 3.2): the
 * department part once per (department, token), the private part once per
 * (expert, token), then combined.  y: [T, h] fp64. */
int oref_layer_two_stage(const oref_config *cfg, int T, const void *x, const oref_weights *w,
                         const float *logits_in, const float *bias, double *y);

/* Weight bytes one step must read given the realised per-department and
 * per-expert token counts: every touched department / expert matrix once,
 * the router, the shared expert, fp8 block scales. */
int64_t oref_step_weight_bytes(const oref_config *cfg, const int32_t *dept_count,
                               const int32_t *exp_count);

#ifdef __cplusplus
}
#endif
#endif
