// Host side of the C ABI: validation, workspace layout and the launch
// sequence of one decode step.  Nothing here allocates, frees or waits.
#include <string.h>

#include <algorithm>
#include <mutex>

#include "gemm_tile.h"
#include "launch.h"

using namespace deamoe;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int kstep_of(int w_dtype) { return w_dtype == DEAMOE_F32 ? 64 : 128; }
int wbytes_of(int w_dtype) { return w_dtype == DEAMOE_F32 ? 4 : w_dtype == DEAMOE_BF16 ? 2 : 1; }
int abytes_of(int act_dtype) { return act_dtype == DEAMOE_F32 ? 4 : 2; }

// Number of hidden-dimension chunks the router product is split into: the
// largest divisor of the K steps that keeps >= 4 steps per chunk (one per
// wave), at most 16 chunks, and about 256 workgroups in total.
int router_chunks(const deamoe_config &c) {
  const int ks = c.act_dtype == DEAMOE_F32 ? 64 : 128;
  const int steps = c.hidden / ks;
  const int tiles = (c.n_experts + kTile - 1) / kTile;
  const int want = (256 + tiles - 1) / tiles;
  int best = 1;
  for (int d = 1; d <= steps; ++d)
    if (steps % d == 0 && d <= want && d <= 16 && steps / d >= 4) best = d;
  return best;
}

int max_slots_of(const deamoe_config &c) { return 2 * c.top_k + 1; }

bool has_private(const deamoe_config &c) {
  return c.form == DEAMOE_FORM_FACTORED || c.d_private > 0;
}

struct Layout {
  size_t part, topk_ids, topk_w, tok_depts, tok_dept_w, tok_ndept, dept_count,
      dept_offset, dept_tokens, exp_count, exp_offset, exp_tokens;
  size_t counts, units[kMaxStages], slot_pair, slot_w, nslot, tok_exp_pair, exp_src, pair_dept;
  size_t abuf_dept, abuf_exp, abuf_se, gbuf, ubuf, ybuf, zbuf, zsbuf, partial;
  size_t wdense, cunits;   // fused SLICE down stage
  size_t total;
  int kc, max_units, max_dept_pairs, max_exp_pairs;
};

Layout make_layout(const deamoe_config &c) {
  Layout L;
  const size_t T = (size_t)c.max_tokens, n = c.n_experts, m = c.n_depts, k = c.top_k;
  const size_t h = c.hidden, ab = abytes_of(c.act_dtype);
  const size_t dk = std::min<size_t>(c.top_k_dept > 0 ? c.top_k_dept : k, std::min(k, m));
  L.kc = router_chunks(c);
  L.max_units = (int)(m + n + 1);
  L.max_dept_pairs = (int)(T * dk);
  L.max_exp_pairs = (int)(T * k);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + (bytes ? bytes : 1));
    return o;
  };
  L.part = take((size_t)L.kc * T * 64 * route_ns(c.n_experts) * 4);
  L.topk_ids = take(T * k * 4);
  L.topk_w = take(T * k * 4);
  L.tok_depts = take(T * k * 4);
  L.tok_dept_w = take(T * k * 4);
  L.tok_ndept = take(T * 4);
  L.dept_count = take(m * 4);
  L.dept_offset = take((m + 1) * 4);
  L.dept_tokens = take(T * k * 4);
  L.exp_count = take(n * 4);
  L.exp_offset = take((n + 1) * 4);
  L.exp_tokens = take(T * k * 4);
  L.counts = take(sizeof(PlanCounts));
  for (int s = 0; s < kMaxStages; ++s) L.units[s] = take((size_t)L.max_units * sizeof(GemmUnit));
  const size_t S = max_slots_of(c);
  L.slot_pair = take(T * S * 4);
  L.slot_w = take(T * S * 4);
  L.nslot = take(T * 4);
  L.tok_exp_pair = take(T * k * 4);
  L.exp_src = take(T * k * 4);
  L.pair_dept = take((size_t)L.max_dept_pairs * 4);
  const size_t dpairs = L.max_dept_pairs, epairs = L.max_exp_pairs;
  const size_t ds = c.d_shared, dp = c.d_private, dse = c.d_shared_expert;
  L.abuf_se = take(T * dse * ab);
  if (c.form == DEAMOE_FORM_SLICE) {
    L.abuf_dept = take(dpairs * ds * ab);
    L.abuf_exp = take(epairs * dp * ab);
    L.gbuf = L.ubuf = L.ybuf = L.zbuf = L.zsbuf = 0;
    L.partial = take((dpairs + (dp ? epairs : 0) + (dse ? T : 0)) * h * 4);
  } else {
    L.abuf_dept = L.abuf_exp = 0;
    L.gbuf = take(dpairs * ds * ab);
    L.ubuf = take(dpairs * ds * ab);
    L.ybuf = take(epairs * ds * ab);
    L.zbuf = take(epairs * ds * 4);
    L.zsbuf = take(dpairs * ds * ab);
    L.partial = take((dpairs + (dse ? T : 0)) * h * 4);
  }
  // fused down stage, batches of at most 32 tokens: routing weights per unit
  // and token (and a row of ones), the unit table
  L.wdense = take((m + n + 1) * kChainT * 4);
  L.cunits = take((size_t)kMaxChainUnits * sizeof(ChainUnit));
  L.total = off;
  return L;
}

int validate_config(const deamoe_config *c) {
  if (!c) return DEAMOE_ERR_INVALID;
  if (c->hidden <= 0 || c->n_experts <= 0 || c->n_depts <= 0) return DEAMOE_ERR_INVALID;
  if (c->n_experts % c->n_depts) return DEAMOE_ERR_INVALID;
  if (c->top_k <= 0 || c->top_k > c->n_experts) return DEAMOE_ERR_INVALID;
  if (c->top_k_dept < 0 || c->top_k_dept > c->n_depts) return DEAMOE_ERR_INVALID;
  const int E = c->n_experts / c->n_depts;
  if (c->top_k_dept > 0 && c->top_k > c->top_k_dept * E) return DEAMOE_ERR_INVALID;
  if (c->d_shared <= 0 || c->d_private < 0 || c->d_shared_expert < 0) return DEAMOE_ERR_INVALID;
  if (c->form != DEAMOE_FORM_SLICE && c->form != DEAMOE_FORM_FACTORED) return DEAMOE_ERR_INVALID;
  if (c->score != DEAMOE_SCORE_SOFTMAX && c->score != DEAMOE_SCORE_SIGMOID) return DEAMOE_ERR_INVALID;
  if (c->renorm != 0 && c->renorm != 1) return DEAMOE_ERR_INVALID;
  if (c->sigma < DEAMOE_SIGMA_SILU || c->sigma > DEAMOE_SIGMA_RMSNORM) return DEAMOE_ERR_INVALID;
  if (c->dept_cover != 0 && c->dept_cover != 1) return DEAMOE_ERR_INVALID;
  if (c->dept_cover && (c->top_k_dept == 0 || c->top_k < c->top_k_dept)) return DEAMOE_ERR_INVALID;
  if (!(c->route_scale == c->route_scale)) return DEAMOE_ERR_INVALID;
  if (c->w_dtype < DEAMOE_F32 || c->w_dtype > DEAMOE_FP8_E4M3_B128) return DEAMOE_ERR_INVALID;
  if (c->act_dtype != DEAMOE_F32 && c->act_dtype != DEAMOE_BF16) return DEAMOE_ERR_INVALID;
  if (c->max_tokens <= 0) return DEAMOE_ERR_INVALID;
  // limits of this build
  if (c->max_tokens > DEAMOE_MAX_TOKENS || c->n_experts > DEAMOE_MAX_EXPERTS ||
      c->top_k > DEAMOE_MAX_TOPK || c->n_depts > kMaxM)
    return DEAMOE_ERR_UNSUPPORTED;
  if (c->top_k_dept > 0 && c->n_depts > kMaxMGrouped) return DEAMOE_ERR_UNSUPPORTED;
  if (c->hidden > DEAMOE_MAX_WIDTH || c->d_shared > DEAMOE_MAX_WIDTH ||
      c->d_private > DEAMOE_MAX_WIDTH || c->d_shared_expert > DEAMOE_MAX_WIDTH)
    return DEAMOE_ERR_UNSUPPORTED;
  // fp32 weights pair with fp32 activations, bf16 / fp8 weights with bf16
  if ((c->w_dtype == DEAMOE_F32) != (c->act_dtype == DEAMOE_F32)) return DEAMOE_ERR_UNSUPPORTED;
  // every contraction length is a whole number of matrix-core K steps
  const int ks = kstep_of(c->w_dtype);
  if (c->hidden % ks || c->d_shared % ks) return DEAMOE_ERR_UNSUPPORTED;
  if (c->form == DEAMOE_FORM_SLICE && c->d_private % ks) return DEAMOE_ERR_UNSUPPORTED;
  if (c->d_shared_expert % ks) return DEAMOE_ERR_UNSUPPORTED;
  // a work item holds its fp8 block scales as one 64-entry window
  if (c->w_dtype == DEAMOE_FP8_E4M3_B128 &&
      (c->hidden > DEAMOE_MAX_FP8_K || c->d_shared > DEAMOE_MAX_FP8_K ||
       c->d_private > DEAMOE_MAX_FP8_K || c->d_shared_expert > DEAMOE_MAX_FP8_K))
    return DEAMOE_ERR_UNSUPPORTED;
  return DEAMOE_OK;
}

int validate_weights(const deamoe_config &c, const deamoe_weights *w, bool need_router) {
  if (!w) return DEAMOE_ERR_INVALID;
  if (need_router && !w->router) return DEAMOE_ERR_INVALID;
  const void *mats[9] = {w->dept_gate, w->dept_up, w->dept_down, w->priv_gate, w->priv_up,
                         w->priv_down, w->se_gate, w->se_up, w->se_down};
  bool used[9] = {true, true, true, has_private(c), has_private(c), has_private(c),
                  c.d_shared_expert > 0, c.d_shared_expert > 0, c.d_shared_expert > 0};
  for (int i = 0; i < 9; ++i) {
    if (!used[i]) continue;
    if (!mats[i] || ((uintptr_t)mats[i] & 15)) return DEAMOE_ERR_INVALID;
    if (c.w_dtype == DEAMOE_FP8_E4M3_B128 && (!w->scale[i] || ((uintptr_t)w->scale[i] & 3)))
      return DEAMOE_ERR_INVALID;
  }
  if (w->router && ((uintptr_t)w->router & 15)) return DEAMOE_ERR_INVALID;
  return DEAMOE_OK;
}

int ntt_of(int T) { return T <= 16 ? 1 : T <= 32 ? 2 : T <= 64 ? 4 : 8; }

// Token tiles per wave in the gate/up stage.  A unit with more tokens than
// one wave holds gets one work item per token group, and every group
// streams the unit's rows.  SLICE: one tile up to 16 tokens, two above, and
// on layers at least 4096 wide four above 64 tokens (fp8: above 96).
// Same-process A/B, us per step, two tiles -> four, outputs bit-identical,
// with the token rows loaded as whole segments: the DeepSeek-V3 shape 950.2
// -> 917.3 at 128 tokens, 868.4 -> 864.8 at 96, 818.8 -> 818.1 at 72;
// skewed routing 463.2 -> 447.2 at 128, 412.7 -> 402.7 at 96, 369.1 ->
// 363.3 at 72; fp8 645.3 -> 631.1 at 128 but 515.8 -> 531.2 at 96 and 477.2
// -> 489.3 at 72.  The 2048-wide 7B-class layer was slower with four
// (145.8 -> 153.1 at 128, before the whole-segment rows): they halve its
// work items and leave the three-wave two-tile kernel for a two-wave one.  The FACTORED stages keep one tile at
// every batch: its private gate/up then runs at three waves per SIMD, which
// outweighs streaming the rows of a unit with more than 16 tokens once per
// group.
int wave_ntt_of(const deamoe_config &c, int T) {
  if (c.form == DEAMOE_FORM_FACTORED) return 1;
  const int four_from = c.w_dtype == DEAMOE_FP8_E4M3_B128 ? 97 : 65;
  return T <= kTile ? 1 : T < four_from || c.hidden < 4096 ? 2 : 4;
}
int token_groups_max(const deamoe_config &c, int T) {
  const int gt = kTile * wave_ntt_of(c, T);
  return (T + gt - 1) / gt;
}
// Token tiles per wave in the separate down stages (above 32 tokens for
// SLICE).  Layers narrower than 4096 keep one tile up to 56 tokens: there
// the one-tile row pairs at three waves per SIMD outweigh streaming the rows
// of a unit with more than 16 tokens once per group (same-process A/B with
// the token rows loaded as whole segments, us per step, one tile -> two: the
// 7B-class layer 84.0 -> 91.3 at 40 tokens, 85.3 -> 92.2 at 52, 87.9 ->
// 92.9 at 56, but 96.3 -> 94.2 at 60 and 98.9 -> 96.9 at 64; before those
// rows two tiles lost at 64 too, 106.2 -> 110.5).  Wider layers take two
// (the DeepSeek-V3 shape 776.5 -> 775.3 at 56, 819.6 -> 806.3 at 64; fp8
// 482.7 -> 480.4 and skewed routing 368.5 -> 361.5 at 64; even at 48).
// Where the gate/up stage takes four token tiles, the bf16 down stage takes
// four too (row pairs of 64 tokens, two waves per SIMD): same-process A/B,
// us per step, outputs bit-identical: skewed routing 363.2 -> 353.6 at 72
// tokens, 402.5 -> 393.4 at 96, 447.6 -> 437.8 at 128; the DeepSeek-V3
// shape 817.5 -> 815.3 at 72, 919.3 -> 907.7 at 128.  fp8 keeps two (569.9
// -> 581.2 at 128 with four).  The FACTORED down stages (the
// private B_e and the department W_d^T) take two from 17 tokens on layers at
// least 4096 wide, where a department's W_d^T then streams once per 32
// tokens instead of once per 16 (same-process A/B, us per step, outputs
// bit-identical: DeepSeek-V3 FACTORED 1215.6 -> 1203.9 at 32 tokens and
// 1960.9 -> 1944.5 at 64, the W_d^T stage 85.2 -> 66.0; Qwen3 494.0 ->
// 485.7 at 32 and 706.0 -> 695.9 at 64; Kimi-K2 2265.0 -> 2244.4 at 64);
// the 1024-wide Baseline-7B layer was slower (120.6 -> 124.3 at 64).
int down_ntt_of(const deamoe_config &c, int T) {
  if (c.form == DEAMOE_FORM_FACTORED) return T > kTile && c.hidden >= 4096 ? 2 : 1;
  if (c.form == DEAMOE_FORM_SLICE && T <= 56 && c.hidden < 4096) return 1;
  const int n = wave_ntt_of(c, T);
  return c.w_dtype == DEAMOE_FP8_E4M3_B128 ? std::min(2, n) : n;
}
int down_groups_max(const deamoe_config &c, int T) {
  const int gt = kTile * down_ntt_of(c, T);
  return (T + gt - 1) / gt;
}

// Waves sharing one SLICE gate/up tile: four, and two above 32 tokens, where
// two token tiles leave two waves per SIMD and twice the tiles in flight per
// workgroup stream faster.
int slice_gate_up_ks_of(int T) { return T > kChainT ? 2 : 4; }

// K split of the FACTORED stages: the department gate/up over 4 waves, the
// private gate/up (split token operands) over 2 (4 was slower at every
// batch), or over none where its contraction (d) is shorter than 1024 and
// more than 16 tokens give enough tiles (Baseline-7B, d = 384: 143.3 ->
// 134.0 us per step at 64 tokens; even at 16; the wider Table 1 layers
// were 1-2 % slower without the split).
constexpr int kFactoredGateUpKs = 4;
int factored_priv_ks_of(const deamoe_config &c, int T) {
  return c.d_shared < 1024 && T > 16 ? 1 : 2;
}

// Down-projection tiles are row pairs: two adjacent 16-row tiles of a matrix
// streamed by one wave with one token operand for both.
constexpr int kDownRows = 2 * kTile;

// Waves sharing one down-projection tile.  The SLICE form packs several
// short private tiles per work item and keeps whole tiles per wave (K split
// over two waves up to two tokens, where the batch leaves few work items);
// the FACTORED form (every contraction d long) splits K four ways up to 8
// tokens and two ways up to 32 (64 where h >= 4096), while the batch leaves
// too few tiles to occupy the waves.  From 9 to 16 tokens the split follows
// the contraction: four ways for d >= 2048, none for d < 1024 (same-process
// A/B at 16 tokens, us per step: the DeepSeek-V3 FACTORED layer 711.2 ->
// 698.6, Kimi-K2 852.2 -> 846.2, Baseline-7B 71.5 -> 70.2; Qwen3 and
// DeepSeek-V2, d = 1536, were even either way).
int down_ks_of(const deamoe_config &c, int T) {
  if (c.form == DEAMOE_FORM_SLICE) return T <= 2 ? 2 : 1;
  if (T <= 8) return 4;
  if (T <= 16 && c.d_shared >= 2048) return 4;
  if (T <= 16 && c.d_shared < 1024) return 1;
  const bool wide = c.hidden >= 4096;
  return T <= 32 || (wide && T <= 64) ? 2 : 1;
}


// Down projections and combine fused into one kernel (the SLICE down stage,
// the FACTORED department down stage): batches whose active units fit the
// kernel's unit table.  Its grid is one workgroup per 32 rows of y.  SLICE:
// up to 32 tokens (two token tiles from 17 on); below kChainMinTiles row
// pairs (a hidden size under 4096, where the kernel takes 16-row blocks) up
// to kChainNarrowMaxT tokens from kChainNarrowMinTiles row pairs on
// (same-process A/B on the 2048-wide 7B-class layer against the separate
// down stage and combine, us per step: 66.5 -> 61.5 at 5 tokens, 81.0 ->
// 76.1 at 16, 89.6 -> 85.6 at 24, but 89.9 -> 91.1 at 32), and up to 4
// tokens on narrower layers, where the kernel's workgroups leave most CUs
// idle (the 1024-wide Baseline-7B vanilla layer, separate stage against the
// fused kernel: 58.9 -> 46.5 at 8 tokens, 88.6 -> 64.5 at 16).  FACTORED: up to 16 tokens at every Table 1 width (at
// least kChainMinTilesFactored row pairs, h >= 1024): the fused kernel saves
// the combine launch.  Same-process A/B against the separate department down
// stage and combine, us per step: Baseline-7B (h = 1024) 38.3 -> 36.3 at one
// token, 77.7 -> 75.6 at 16; Qwen3 (h = 4096, with 16-row blocks) 79.8 ->
// 76.9 at one token, 220.7 -> 214.4 at 8, 308.2 -> 305.1 at 16; DeepSeek-V2
// (h = 5120) 90.3 -> 86.6 at one token, 389.7 -> 389.0 at 16.
constexpr int kChainMinTiles = 128, kChainMinTilesFactored = 32;
constexpr int kChainNarrowMinTiles = 64, kChainNarrowMaxT = 24;
bool use_chain(const deamoe_config &c, int T) {
  if (T > kChainT) return false;
  // the plan builds the fused kernel's units for one token group only
  if (token_groups_max(c, T) > 1) return false;
  const int tiles = c.hidden / (2 * kTile);
  if (c.form == DEAMOE_FORM_FACTORED && (T > kTile || tiles < kChainMinTilesFactored)) return false;
  if (c.form == DEAMOE_FORM_SLICE && tiles < kChainMinTiles &&
      T > (tiles >= kChainNarrowMinTiles ? kChainNarrowMaxT : 4))
    return false;
  const int dk = std::min(c.top_k_dept > 0 ? c.top_k_dept : c.top_k, std::min(c.top_k, c.n_depts));
  const bool slice_priv = c.form == DEAMOE_FORM_SLICE && c.d_private > 0;
  const int units = std::min(c.n_depts, T * dk) +
                    (slice_priv ? std::min(c.n_experts, T * c.top_k) : 0) +
                    (c.d_shared_expert ? 1 : 0);
  return units <= kMaxChainUnits;
}

// Upper bound of the row tiles of a stage, for the grid size.
int tiles_bound(int units_max, int R, int rows = kTile) {
  return units_max * ((R + rows - 1) / rows);
}

// Tiles of the first expert stage a step of T tokens can have at most.
int first_stage_items(const deamoe_config &c, int T) {
  const int dk = std::min(c.top_k_dept > 0 ? c.top_k_dept : c.top_k, std::min(c.top_k, c.n_depts));
  const bool slice = c.form == DEAMOE_FORM_SLICE;
  return tiles_bound(std::min(c.n_depts, T * dk), c.d_shared) +
         (slice && c.d_private ? tiles_bound(std::min(c.n_experts, T * c.top_k), c.d_private)
                               : 0) +
         (c.d_shared_expert ? tiles_bound(1, c.d_shared_expert) : 0);
}

// Batches of at most kSmallMaxT tokens route inside the launch of the first
// expert stage (every workgroup routes the tokens itself; workgroup 0
// publishes the routing and runs the plan): one dependent launch fewer, and
// no unit-table round trip before the weights stream, where that pays off
// (small_route_pays).
bool use_small(const deamoe_config &c, int T) {
  const int wt = c.w_dtype == DEAMOE_F32 ? WT_F32 : c.w_dtype == DEAMOE_BF16 ? WT_BF16 : WT_FP8;
  return T <= kSmallMaxT &&
         small_route_pays(wt, c.n_experts, c.hidden, wbytes_of(c.w_dtype),
                          c.top_k_dept > 0, first_stage_items(c, T));
}

template <class P>
P *at(void *ws, size_t off) {
  return reinterpret_cast<P *>(static_cast<char *>(ws) + off);
}

struct Events {
  void *const *ev;
  int n, next;
  hipStream_t s;
  hipError_t mark() {
    if (!ev || next >= n) return hipSuccess;
    return hipEventRecord(static_cast<hipEvent_t>(ev[next++]), s);
  }
};

int check(hipError_t e) { return e == hipSuccess ? DEAMOE_OK : DEAMOE_ERR_HIP; }

#define DEAMOE_TRY(expr)                    \
  do {                                      \
    const int _rc = check(expr);            \
    if (_rc != DEAMOE_OK) return _rc;       \
  } while (0)

// Router product: partial logits over the hidden-dimension chunks.
int enqueue_router(const deamoe_config &c, int T, const void *x, const void *router_w, void *ws,
                   const Layout &L, Events &ev, hipStream_t s) {
  RouterArgs ra;
  ra.w = router_w;
  ra.x = x;
  ra.part = at<float>(ws, L.part);
  ra.n = c.n_experts;
  ra.h = c.hidden;
  ra.T = T;
  ra.kchunk = c.hidden / L.kc;
  ra.tiles = (c.n_experts + kTile - 1) / kTile;
  ra.ldp = 64 * route_ns(c.n_experts);
  DEAMOE_TRY(launch_router(ra, c.act_dtype == DEAMOE_F32 ? WT_F32 : WT_BF16, ntt_of(T), L.kc, s));
  DEAMOE_TRY(ev.mark());
  return DEAMOE_OK;
}

// Argument block of the routing kernels (and of the plan they write).
void fill_route_args(RouteArgs &a, const deamoe_config &c, int T, const void *x,
                     const float *logits_in, const float *bias, const deamoe_routing &r,
                     void *ws, const Layout &L, int plan, const deamoe_weights *w) {
  memset(&a, 0, sizeof a);
  a.T = T;
  a.n = c.n_experts;
  a.m = c.n_depts;
  a.k = c.top_k;
  a.kdept = c.top_k_dept;
  a.dept_cover = c.dept_cover;
  a.E = c.n_experts / c.n_depts;
  a.score = c.score;
  a.renorm = c.renorm;
  a.route_scale = c.route_scale;
  a.h = c.hidden;
  a.d_s = c.d_shared;
  a.d_p = c.form == DEAMOE_FORM_SLICE ? c.d_private : 0;
  a.d_se = c.d_shared_expert;
  a.act_f32 = c.act_dtype == DEAMOE_F32;
  a.w_bytes = wbytes_of(c.w_dtype);
  a.fp8 = c.w_dtype == DEAMOE_FP8_E4M3_B128;
  a.plan = plan;
  a.down_rows = kDownRows;
  a.down_ks = down_ks_of(c, T);
  a.wave_tokens = kTile * wave_ntt_of(c, T);
  a.wave_tokens_b = kTile * down_ntt_of(c, T);
  a.sigma = c.sigma;
  a.part = at<float>(ws, L.part);
  a.kc = L.kc;
  a.ldp = 64 * route_ns(c.n_experts);
  a.logits_in = logits_in;
  a.bias = bias;
  a.r = r;
  a.counts = at<PlanCounts>(ws, L.counts);
  for (int i = 0; i < kMaxStages; ++i) a.units[i] = at<GemmUnit>(ws, L.units[i]);
  a.slot_pair = at<int32_t>(ws, L.slot_pair);
  a.nslot = at<int32_t>(ws, L.nslot);
  a.slot_w = at<float>(ws, L.slot_w);
  a.tok_exp_pair = at<int32_t>(ws, L.tok_exp_pair);
  a.exp_src = at<int32_t>(ws, L.exp_src);
  a.pair_dept = at<int32_t>(ws, L.pair_dept);
  a.max_slots = max_slots_of(c);
  if (w) a.w = *w;
  a.x = x;
  a.abuf_dept = at<void>(ws, L.abuf_dept);
  a.abuf_exp = at<void>(ws, L.abuf_exp);
  a.abuf_se = at<void>(ws, L.abuf_se);
  a.gbuf = at<void>(ws, L.gbuf);
  a.ubuf = at<void>(ws, L.ubuf);
  a.ybuf = at<void>(ws, L.ybuf);
  a.zsbuf = at<void>(ws, L.zsbuf);
  a.zbuf = at<float>(ws, L.zbuf);
  a.partial = at<float>(ws, L.partial);
  if (plan != PLAN_NONE && use_chain(c, T)) {
    a.chain = 1;
    a.cunits = at<ChainUnit>(ws, L.cunits);
    a.wdense = at<float>(ws, L.wdense);
  }
}

// Router product and route/plan kernels.
int enqueue_route(const deamoe_config &c, int T, const void *x, const void *router_w,
                  const float *logits_in, const float *bias, const deamoe_routing &r, void *ws,
                  const Layout &L, int plan, const deamoe_weights *w, Events &ev,
                  hipStream_t s) {
  DEAMOE_TRY(ev.mark());
  if (!logits_in) {
    const int rc = enqueue_router(c, T, x, router_w, ws, L, ev, s);
    if (rc) return rc;
  }
  RouteArgs a;
  fill_route_args(a, c, T, x, logits_in, bias, r, ws, L, plan, w);
  DEAMOE_TRY(launch_route(a, s));
  DEAMOE_TRY(ev.mark());
  return DEAMOE_OK;
}

deamoe_routing routing_in_ws(void *ws, const Layout &L, const deamoe_routing *user) {
  deamoe_routing r;
  if (user) {
    r = *user;
  } else {
    r.topk_ids = at<int32_t>(ws, L.topk_ids);
    r.topk_w = at<float>(ws, L.topk_w);
    r.tok_depts = at<int32_t>(ws, L.tok_depts);
    r.tok_dept_w = at<float>(ws, L.tok_dept_w);
    r.tok_ndept = at<int32_t>(ws, L.tok_ndept);
    r.dept_count = at<int32_t>(ws, L.dept_count);
    r.dept_offset = at<int32_t>(ws, L.dept_offset);
    r.dept_tokens = at<int32_t>(ws, L.dept_tokens);
    r.exp_count = at<int32_t>(ws, L.exp_count);
    r.exp_offset = at<int32_t>(ws, L.exp_offset);
    r.exp_tokens = at<int32_t>(ws, L.exp_tokens);
    r.logits = nullptr;   // no kernel reads them back
  }
  return r;
}

bool routing_complete(const deamoe_routing &r) {
  return r.topk_ids && r.topk_w && r.tok_depts && r.tok_dept_w && r.tok_ndept && r.dept_count &&
         r.dept_offset && r.dept_tokens && r.exp_count && r.exp_offset && r.exp_tokens;
}


// Launch of a down-projection stage (row-pair tiles).
hipError_t launch_down(const GemmStage &st, int wt, int ntt, int groups, int ks, int units_max,
                       int R, int cap, hipStream_t s) {
  return launch_grouped_gemm(st, wt, 2, GEMM_PAIR, ntt, ks,
                             tiles_bound(units_max, R, kDownRows) * groups, cap, s);
}

constexpr int kGridCap = 8192;   // 256 CUs x 32 workgroups

int layer_impl(const deamoe_config *cfg, int32_t T, const void *x, const deamoe_weights *w,
               const float *logits_in, const float *bias, deamoe_routing *routing_out, void *y,
               void *ws, size_t ws_bytes, void *stream, void *const *events, int32_t n_events) {
  int rc = validate_config(cfg);
  if (rc) return rc;
  const deamoe_config &c = *cfg;
  if (T < 0 || T > c.max_tokens) return T < 0 ? DEAMOE_ERR_INVALID : DEAMOE_ERR_UNSUPPORTED;
  if (T == 0) return DEAMOE_OK;   // empty batch: nothing to read or write
  if ((rc = validate_weights(c, w, !logits_in))) return rc;
  if (!x || !y) return DEAMOE_ERR_INVALID;
  if (routing_out && !routing_complete(*routing_out)) return DEAMOE_ERR_INVALID;
  if (n_events < 0 || (n_events > 0 && !events)) return DEAMOE_ERR_INVALID;
  const Layout L = make_layout(c);
  if (!ws || ws_bytes < L.total) return DEAMOE_ERR_WORKSPACE;
  if ((uintptr_t)ws % kAlign) return DEAMOE_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Events ev{events, n_events, 0, s};
  const deamoe_routing r = routing_in_ws(ws, L, routing_out);
  const bool slice = c.form == DEAMOE_FORM_SLICE;
  const int wt = c.w_dtype == DEAMOE_F32 ? WT_F32 : c.w_dtype == DEAMOE_BF16 ? WT_BF16 : WT_FP8;
  const bool small = use_small(c, T);
  if (small) {   // router, then routing + plan + the first expert stage in one launch
    DEAMOE_TRY(ev.mark());
    if (!logits_in && (rc = enqueue_router(c, T, x, w->router, ws, L, ev, s))) return rc;
    RouteArgs a;
    fill_route_args(a, c, T, x, logits_in, bias, r, ws, L, slice ? PLAN_SLICE : PLAN_FACTORED,
                    w);
    DEAMOE_TRY(launch_small_route_gate_up(a, wt, first_stage_items(c, T), s));
  } else {
    rc = enqueue_route(c, T, x, w->router, logits_in, bias, r, ws, L,
                       slice ? PLAN_SLICE : PLAN_FACTORED, w, ev, s);
    if (rc) return rc;
  }
  const int ntt = wave_ntt_of(c, T), groups = token_groups_max(c, T);
  const PlanCounts *pc = at<PlanCounts>(ws, L.counts);
  auto stage = [&](int i) {
    GemmStage st;
    st.units = at<GemmUnit>(ws, L.units[i]);
    st.counts = pc->stage[i];
    st.sigma = c.sigma;
    return st;
  };
  const int m = c.n_depts, dk = L.max_dept_pairs / c.max_tokens;
  const int act_depts = std::min(m, T * dk);
  const int act_exps = std::min(c.n_experts, T * c.top_k);
  const int se = c.d_shared_expert > 0 ? 1 : 0;
  if (slice) {
    const int ta = tiles_bound(act_depts, c.d_shared) +
                   (c.d_private ? tiles_bound(act_exps, c.d_private) : 0) +
                   se * tiles_bound(1, c.d_shared_expert);
    if (!small)
      DEAMOE_TRY(launch_grouped_gemm(stage(0), wt, 2, GEMM_PLAIN, ntt, slice_gate_up_ks_of(T),
                                     ta * groups, kGridCap, s, c.hidden < 4096));
    DEAMOE_TRY(ev.mark());
    if (use_chain(c, T)) {   // down projections and combine in one kernel
      ChainArgs ch;
      ch.units = at<ChainUnit>(ws, L.cunits);
      ch.counts = pc->stage[1];
      ch.y = y;
      ch.T = T;
      ch.h = c.hidden;
      ch.act_f32 = c.act_dtype == DEAMOE_F32;
      DEAMOE_TRY(launch_chain(ch, wt, s));
      DEAMOE_TRY(ev.mark());
      return DEAMOE_OK;
    }
    const int units = act_depts + (c.d_private ? act_exps : 0) + se;
    DEAMOE_TRY(launch_down(stage(1), wt, down_ntt_of(c, T), down_groups_max(c, T),
                           down_ks_of(c, T), units, c.hidden, kGridCap, s));
    DEAMOE_TRY(ev.mark());
  } else {
    const int d = c.d_shared;
    const int t0 = tiles_bound(act_depts, d) + se * tiles_bound(1, c.d_shared_expert);
    if (!small)
      DEAMOE_TRY(launch_grouped_gemm(stage(0), wt, 2, GEMM_PLAIN, ntt, kFactoredGateUpKs, t0 * groups,
                                     kGridCap, s));
    if (c.sigma == DEAMOE_SIGMA_RMSNORM) {   // timed with stage 0
      RowNormArgs na;
      na.counts = pc;
      na.g = at<void>(ws, L.gbuf);
      na.u = at<void>(ws, L.ubuf);
      na.d = d;
      na.act_f32 = c.act_dtype == DEAMOE_F32;
      DEAMOE_TRY(launch_rownorm(na, T * dk, s));
    }
    DEAMOE_TRY(ev.mark());
    DEAMOE_TRY(launch_grouped_gemm(stage(1), wt, 2, GEMM_SPLIT, ntt,
                                   factored_priv_ks_of(c, T), tiles_bound(act_exps, d) * groups,
                                   kGridCap, s));
    DEAMOE_TRY(ev.mark());
    DEAMOE_TRY(launch_down(stage(2), wt, down_ntt_of(c, T), down_groups_max(c, T),
                           down_ks_of(c, T), act_exps, d, kGridCap, s));
    DEAMOE_TRY(ev.mark());
    ZsumArgs za;
    za.counts = pc;
    za.dept_tokens = r.dept_tokens;
    za.pair_dept = at<int32_t>(ws, L.pair_dept);
    za.topk_ids = r.topk_ids;
    za.tok_exp_pair = at<int32_t>(ws, L.tok_exp_pair);
    za.topk_w = r.topk_w;
    za.z = at<float>(ws, L.zbuf);
    za.zs = at<void>(ws, L.zsbuf);
    za.m = m;
    za.k = c.top_k;
    za.E = c.n_experts / m;
    za.d = d;
    za.act_f32 = c.act_dtype == DEAMOE_F32;
    za.rms = c.sigma == DEAMOE_SIGMA_RMSNORM;
    DEAMOE_TRY(launch_zsum(za, T * dk, s));
    DEAMOE_TRY(ev.mark());
    if (use_chain(c, T)) {   // department down projections and combine in one kernel
      ChainArgs ch;
      ch.units = at<ChainUnit>(ws, L.cunits);
      ch.counts = pc->stage[3];
      ch.y = y;
      ch.T = T;
      ch.h = c.hidden;
      ch.act_f32 = c.act_dtype == DEAMOE_F32;
      DEAMOE_TRY(launch_chain(ch, wt, s));
      DEAMOE_TRY(ev.mark());
      return DEAMOE_OK;
    }
    DEAMOE_TRY(launch_down(stage(3), wt, down_ntt_of(c, T), down_groups_max(c, T),
                           down_ks_of(c, T), act_depts + se, c.hidden, kGridCap, s));
    DEAMOE_TRY(ev.mark());
  }
  CombineArgs ca;
  ca.partial = at<float>(ws, L.partial);
  ca.slot_pair = at<int32_t>(ws, L.slot_pair);
  ca.nslot = at<int32_t>(ws, L.nslot);
  ca.slot_w = at<float>(ws, L.slot_w);
  ca.y = y;
  ca.T = T;
  ca.h = c.hidden;
  ca.max_slots = max_slots_of(c);
  ca.act_f32 = c.act_dtype == DEAMOE_F32;
  DEAMOE_TRY(launch_combine(ca, s));
  DEAMOE_TRY(ev.mark());
  return DEAMOE_OK;
}

int64_t matrix_bytes(int w_dtype, int64_t R, int64_t C) {
  int64_t b = R * C * wbytes_of(w_dtype);
  if (w_dtype == DEAMOE_FP8_E4M3_B128) b += ((R + 127) / 128) * ((C + 127) / 128) * 4;
  return b;
}

// Workspace of deamoe_layer_forward_noalloc: one library-owned device array
// per GPU, held until the process ends.  Host code never passes the array's
// name to a kernel or a copy: each device's address comes from
// hipGetSymbolAddress, resolved once per device with that device current.
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchDevices] = {};

}  // namespace

static __device__ __align__(256) unsigned char scratch[DEAMOE_SCRATCH_BYTES];

namespace {

int scratch_of_current_device(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DEAMOE_ERR_HIP;
  if (dev < 0 || dev >= kScratchDevices) return DEAMOE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DEAMOE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DEAMOE_OK;
}

}  // namespace

extern "C" {

const char *deamoe_status_string(int status) {
  switch (status) {
    case DEAMOE_OK: return "ok";
    case DEAMOE_ERR_INVALID: return "invalid argument";
    case DEAMOE_ERR_UNSUPPORTED: return "unsupported by this build";
    case DEAMOE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case DEAMOE_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int deamoe_workspace_bytes(const deamoe_config *cfg, size_t *bytes) {
  const int rc = validate_config(cfg);
  if (rc) return rc;
  if (!bytes) return DEAMOE_ERR_INVALID;
  *bytes = make_layout(*cfg).total;
  return DEAMOE_OK;
}

int deamoe_route(const deamoe_config *cfg, int32_t T, const void *x, const void *router_w,
                 const float *logits_in, const float *router_bias, deamoe_routing *out, void *ws,
                 size_t ws_bytes, void *stream) {
  int rc = validate_config(cfg);
  if (rc) return rc;
  const deamoe_config &c = *cfg;
  if (T < 0) return DEAMOE_ERR_INVALID;
  if (T > c.max_tokens) return DEAMOE_ERR_UNSUPPORTED;
  if (T == 0) return DEAMOE_OK;   // empty batch: nothing to read or write
  if (!out || !routing_complete(*out)) return DEAMOE_ERR_INVALID;
  if (!logits_in && (!x || !router_w)) return DEAMOE_ERR_INVALID;
  if (router_w && ((uintptr_t)router_w & 15)) return DEAMOE_ERR_INVALID;
  const Layout L = make_layout(c);
  if (!ws || ws_bytes < L.total || (uintptr_t)ws % kAlign) return DEAMOE_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Events ev{nullptr, 0, 0, s};
  const deamoe_routing r = routing_in_ws(ws, L, out);
  return enqueue_route(c, T, x, router_w, logits_in, router_bias, r, ws, L, PLAN_NONE, nullptr,
                       ev, s);
}

int deamoe_layer_forward(const deamoe_config *cfg, int32_t T, const void *x,
                         const deamoe_weights *w, const float *logits_in,
                         const float *router_bias, deamoe_routing *routing_out, void *y, void *ws,
                         size_t ws_bytes, void *stream) {
  return layer_impl(cfg, T, x, w, logits_in, router_bias, routing_out, y, ws, ws_bytes, stream,
                    nullptr, 0);
}

int deamoe_layer_forward_noalloc(const deamoe_config *cfg, int32_t T, const void *x,
                                 const deamoe_weights *w, const float *logits_in,
                                 const float *router_bias, deamoe_routing *routing_out, void *y,
                                 void *stream) {
  // the same validation as the workspace call, and the size limit, before any
  // HIP call
  int rc = validate_config(cfg);
  if (rc) return rc;
  if (make_layout(*cfg).total > (size_t)DEAMOE_SCRATCH_BYTES) return DEAMOE_ERR_WORKSPACE;
  if (T < 0) return DEAMOE_ERR_INVALID;
  if (T > cfg->max_tokens) return DEAMOE_ERR_UNSUPPORTED;
  if (T == 0) return DEAMOE_OK;   // empty batch: no HIP call
  void *ws = nullptr;
  if ((rc = scratch_of_current_device(&ws))) return rc;
  return layer_impl(cfg, T, x, w, logits_in, router_bias, routing_out, y, ws,
                    DEAMOE_SCRATCH_BYTES, stream, nullptr, 0);
}

int deamoe_layer_forward_traced(const deamoe_config *cfg, int32_t T, const void *x,
                                const deamoe_weights *w, const float *logits_in,
                                const float *router_bias, deamoe_routing *routing_out, void *y,
                                void *ws, size_t ws_bytes, void *stream, void *const *events,
                                int32_t n_events) {
  return layer_impl(cfg, T, x, w, logits_in, router_bias, routing_out, y, ws, ws_bytes, stream,
                    events, n_events);
}

int deamoe_trace_points(const deamoe_config *cfg, int32_t T, int32_t *n_events) {
  const int rc = validate_config(cfg);
  if (rc) return rc;
  if (!n_events || T < 1 || T > cfg->max_tokens) return DEAMOE_ERR_INVALID;
  *n_events = (cfg->form == DEAMOE_FORM_SLICE ? 6 : 9) - (use_chain(*cfg, T) ? 1 : 0) -
              (use_small(*cfg, T) ? 1 : 0);
  return DEAMOE_OK;
}

int deamoe_baseline_forward(const deamoe_config *cfg, int32_t T, const void *x,
                            const deamoe_weights *w, const float *logits_in,
                            const float *router_bias, deamoe_routing *routing_out, void *y,
                            void *ws, size_t ws_bytes, void *stream) {
  if (!cfg) return DEAMOE_ERR_INVALID;
  if (cfg->n_depts != cfg->n_experts || cfg->d_private != 0 || cfg->form != DEAMOE_FORM_SLICE ||
      cfg->top_k_dept != 0 || cfg->dept_cover != 0)
    return DEAMOE_ERR_INVALID;
  return layer_impl(cfg, T, x, w, logits_in, router_bias, routing_out, y, ws, ws_bytes, stream,
                    nullptr, 0);
}

int deamoe_loaded_bytes(const deamoe_config *cfg, int32_t T, const int32_t *dept_count,
                        const int32_t *exp_count, int64_t *weight_bytes, int64_t *total_bytes) {
  const int rc = validate_config(cfg);
  if (rc) return rc;
  if (T < 0 || !dept_count || !exp_count) return DEAMOE_ERR_INVALID;
  const deamoe_config &c = *cfg;
  const int64_t h = c.hidden, d = c.d_shared, p = c.d_private, e = c.d_shared_expert;
  const int wt = c.w_dtype;
  const int64_t ab = abytes_of(c.act_dtype);
  int64_t dept = 3 * matrix_bytes(wt, d, h);
  int64_t priv = 0;
  if (c.form == DEAMOE_FORM_FACTORED) priv = 3 * matrix_bytes(wt, d, d);
  else if (p > 0) priv = 3 * matrix_bytes(wt, p, h);
  int64_t b = (int64_t)c.n_experts * h * ab;
  for (int j = 0; j < c.n_depts; ++j) b += dept_count[j] > 0 ? dept : 0;
  for (int i = 0; i < c.n_experts; ++i) b += exp_count[i] > 0 ? priv : 0;
  if (e > 0) b += 3 * matrix_bytes(wt, e, h);
  if (weight_bytes) *weight_bytes = b;
  if (total_bytes) *total_bytes = b + 2 * (int64_t)T * h * ab;
  return DEAMOE_OK;
}

}  // extern "C"
