// Kernel argument blocks and host-side launchers shared by the library's
// translation units.
#pragma once

#include "internal.h"

namespace deamoe {

constexpr int kRouteThreads = 1024;
constexpr int kMaxT = DEAMOE_MAX_TOKENS;
constexpr int kMaxK = DEAMOE_MAX_TOPK;
constexpr int kMaxTK = kMaxT * kMaxK;
constexpr int kMaxN = DEAMOE_MAX_EXPERTS;
constexpr int kMaxM = 1024;
constexpr int kMaxMGrouped = 64;   // departments when top_k_dept > 0

// Router product: logits partial sums over KC chunks of the hidden dimension.
struct RouterArgs {
  const void *w;        // [n, h] act dtype
  const void *x;        // [T, h] act dtype
  float *part;          // [kc, T, ldp]
  int32_t n, h, T, kchunk, tiles, ldp;
};

// Logits per lane of the per-token routing kernel (expert e = lane * NS + s);
// the router's partial rows are padded to 64 * NS values.
inline int route_ns(int n) {
  int ns = 1;
  while (64 * ns < n) ns *= 2;
  return ns;
}

enum PlanMode : int32_t { PLAN_NONE = 0, PLAN_SLICE = 1, PLAN_FACTORED = 2 };

struct RouteArgs {
  // configuration
  int32_t T, n, m, k, kdept, E, score, renorm;
  int32_t dept_cover;    // strict coverage of exactly kdept departments
  float route_scale;
  int32_t h, d_s, d_p, d_se, act_f32, w_bytes, fp8, plan;
  int32_t down_rows;     // weight rows of a down-projection tile (16, or 32 for row pairs)
  int32_t down_ks;       // waves sharing one down-projection tile (K split)
  int32_t wave_tokens;   // tokens of one token group of the gate/up stages (16 * NTT)
  int32_t wave_tokens_b; // the same for the down stages
  int32_t sigma;         // DEAMOE_SIGMA_* of the FACTORED gate/up stage
  // logits: sum of kc partial products, or injected; optional bias
  const float *part;
  int32_t kc, ldp;
  const float *logits_in, *bias;
  // routing outputs
  deamoe_routing r;
  // plan outputs
  PlanCounts *counts;
  GemmUnit *units[kMaxStages];
  int32_t *slot_pair, *nslot, *tok_exp_pair, *exp_src;
  int32_t *pair_dept;    // FACTORED: department of every department pair
  float *slot_w;
  int32_t max_slots;
  // inputs of the planned stages
  deamoe_weights w;
  const void *x;
  void *abuf_dept, *abuf_exp, *abuf_se;      // SLICE gate/up outputs
  void *gbuf, *ubuf, *ybuf, *zsbuf;           // FACTORED intermediates (act dtype)
  float *zbuf;                                // FACTORED sigma(A_d^T Y), fp32
  float *partial;                             // [pairs, h] fp32
  // at most kChainT tokens: down projections fused with the combine
  int32_t chain;
  ChainUnit *cunits;                          // units of the fused down stage
  float *wdense;                              // [m + n + 1][kChainT] routing weight per unit
                                              // and token (last row: ones)
};

struct CombineArgs {
  const float *partial;
  const int32_t *slot_pair, *nslot;
  const float *slot_w;
  void *y;
  int32_t T, h, max_slots, act_f32;
};

// Fused down projection and combine (T <= kChainT): one workgroup per 32
// rows of y.
constexpr int kMaxChainUnits = 512;
constexpr int kChainT = 32;   // tokens; also the row length of the token-weight table
struct ChainArgs {
  const ChainUnit *units;
  const int32_t *counts;    // [0] = number of units, [1] = K steps of the concatenation
  void *y;                  // [T, h] act dtype
  int32_t T, h, act_f32;
};

struct ZsumArgs {
  const PlanCounts *counts;
  const int32_t *dept_tokens, *pair_dept, *topk_ids, *tok_exp_pair;
  const float *topk_w, *z;
  void *zs;
  int32_t m, k, E, d, act_f32;
  int32_t rms;           // sigma = RMSNorm: each Z row is divided by its root mean square
};

// sigma = RMSNorm at the gate / up interface of the FACTORED form: rows
// [0, n_dept_pairs) of g and u, each of length d, divided in place by their
// root mean square.
struct RowNormArgs {
  const PlanCounts *counts;
  void *g, *u;
  int32_t d, act_f32;
};

hipError_t launch_router(const RouterArgs &a, int wtype, int ntt, int kc, hipStream_t s);
hipError_t launch_rownorm(const RowNormArgs &a, int max_dept_pairs, hipStream_t s);
// The per-token kernel (grid T) followed by the plan kernel (one workgroup).
hipError_t launch_route(const RouteArgs &a, hipStream_t s);
// Token-operand modes of two-matrix stages (nw == 2).
enum GemmMode : int {
  GEMM_PLAIN = 0,   // both matrices read the same token operand
  GEMM_SPLIT = 1,   // the two matrices read different token operands (in0 / in1)
  GEMM_PAIR = 2,    // the "two matrices" are adjacent 16-row tiles of one matrix
};
// max_tiles bounds the stage's work items (row tiles of kTile rows, or of
// 2 * kTile rows in GEMM_PAIR mode) for the grid size.  narrow: a gate/up
// stage of a layer narrower than 4096 (two token tiles then run at three
// waves per SIMD).
hipError_t launch_grouped_gemm(const GemmStage &st, int wtype, int nw, int mode, int ntt,
                               int ks, int max_tiles, int grid_cap, hipStream_t s,
                               bool narrow = false);
hipError_t launch_combine(const CombineArgs &a, hipStream_t s);
// SLICE batches of 1..4 tokens with the fused down kernel (a.chain): routing,
// the gate/up stage and the down kernel's units in one launch (items: the
// most 16-row gate/up tiles a step can have).
hipError_t launch_small_route_gate_up(const RouteArgs &a, int wtype, int items, hipStream_t s);
// Whether that launch pays off: a short routing prologue (no group limit),
// short tiles (persistent workgroups route once), or every tile resident in
// one round.  Routers of at most 1024 experts.
bool small_route_pays(int wtype, int n, int h, int w_bytes, bool group_limited, int items);
constexpr int kSmallMaxT = 4;
hipError_t launch_chain(const ChainArgs &a, int wtype, hipStream_t s);
hipError_t launch_zsum(const ZsumArgs &a, int max_dept_pairs, hipStream_t s);

}  // namespace deamoe
