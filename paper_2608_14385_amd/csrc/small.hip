// Batches of at most four tokens: routing (Eq. 2 and the department
// bookkeeping of Sec. 3.2), the plan of the later stages and the first
// expert stage (SLICE: every active department's, expert's and the shared
// expert's gate/up pair with SwiGLU; FACTORED: every active department's
// W_g, W_u with sigma, and the shared expert) in one launch after the router
// product.
//
// Every workgroup routes the tokens itself from the router's partial logits
// (one wave per token, results in LDS only) and derives its own work item
// from the step's active units instead of reading a unit table written by an
// earlier launch.  With short tiles (PERSIST) a workgroup routes once and
// then streams every (gridDim.x - 1)-th tile, the grid being sized to the
// workgroups the chip holds at once, so the routing is paid once per
// workgroup rather than once per tile; with long tiles each workgroup
// streams one, and the hardware hands a finishing workgroup's place to the
// next tile.  The units are ordered as the plan orders them: active
// departments ascending, then (SLICE) active experts ascending, then the
// shared expert; a unit's member tokens are in ascending order and its
// output rows start at the unit's CSR offset, the sum of the member counts
// of the units of its kind before it.  Workgroup 0 publishes the routing and
// runs the plan (CSR lists, counts, the unit tables of the later stages,
// combine slots); workgroup 1 + w streams tile w (PERSIST: and
// w + gridDim.x - 1, ...).  No workgroup reads anything another one of this
// launch writes.
#include <algorithm>
#include <atomic>

#include "route_dev.h"

namespace deamoe {

constexpr int kSmallT = 4;             // tokens (one routing wave each)
constexpr int kSmallDW = kMaxM / 32;   // words of a department bitmap
constexpr int kSmallEW = kMaxN / 32;   // words of an expert bitmap (one wave)
static_assert(kSmallEW <= kWave && kSmallDW <= kWave, "bitmap words per wave");

struct SmallSmem {
  uint32_t db[kSmallT][kSmallDW];      // departments of token t
  uint32_t eb[kSmallT][kSmallEW];      // selected experts of token t
  uint32_t pd[kSmallT][kSmallDW];      // exclusive word prefix of popc(department bitmap of t)
  uint32_t pe[kSmallT][kSmallEW];      // the same for eb[t]
  uint32_t ud[kSmallDW], pud[kSmallDW];   // departments of any token, word prefix
  uint32_t ue[kSmallEW], pue[kSmallEW];   // experts of any token, word prefix
  int32_t nud, nue;                    // active departments, active experts
};

// Set bits below bit i of a bitmap with exclusive word prefix `pre`.
__device__ inline int rank_pre(const uint32_t *bits, const uint32_t *pre, int i) {
  return (int)pre[i >> 5] + __popc(bits[i >> 5] & ((1u << (i & 31)) - 1u));
}

// Index of set bit r (0-based) of a bitmap of nw <= 64 words with exclusive
// word prefix `pre`; every lane of the wave calls it with the same r.  The
// word is the last one whose prefix is <= r (lane 0 always qualifies).
__device__ inline int wave_select(const uint32_t *bits, const uint32_t *pre, int nw, int r) {
  const int l = lane_id();
  const uint64_t b = __ballot(l < nw && (int)pre[l] <= r);
  const int w = uniform(63 - __clzll(b));
  uint32_t v = bits[w];
  for (int q = r - (int)pre[w]; q > 0; --q) v &= v - 1u;
  return 32 * w + __ffs(v) - 1;
}

// The routing scratch (and workgroup 0's plan) lives in the weight staging
// space, which is free until the first tile streams; the bitmaps that locate
// the tiles stay beside it.
using SmallPlan = PlanSmemT<kSmallT>;
template <int WT>
union SmallLds {
  typename TileRunner<WT, 2, 1, 4>::Smem run;
  TokSmem tsm[kSmallT];
  struct {
    TokSmem tsm[kSmallT];
    SmallPlan plan;
    RouteArgs sa;
  } pl;
};

template <int WT, int NS, bool PERSIST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
void small_route_gate_up_kernel(RouteArgs a) {
  using Run = TileRunner<WT, 2, 1, 4>;   // four waves share a tile's K steps
  __shared__ SmallLds<WT> lds;
  __shared__ SmallSmem ps;
  __shared__ int32_t s_idx[kSmallT][kSmallT];   // per wave: member tokens of its unit
  TokSmem *tsm = lds.tsm;
  const int wave = uniform(threadIdx.x / kWave), lane = lane_id();
  const bool planner = blockIdx.x == 0;
  const int T = a.T, m = a.m, n = a.n;
  const int dwords = (m + 31) / 32, ewords = (n + 31) / 32;

  if (planner) {   // routing published, then the plan
    args_to_lds<256>(a, lds.pl.sa);
    if (wave < T)
      route_one<NS>(a, wave, lane, lds.pl.tsm[wave],
                    PlanIn{lds.pl.plan.ids, lds.pl.plan.dep, lds.pl.plan.nd, nullptr}, true);
    lds_barrier();
    plan_body<256, true>(lds.pl.sa, lds.pl.plan);
    return;
  }

  // 1. routing: wave t routes token t
  if (wave < T)
    route_one<NS>(a, wave, lane, tsm[wave], PlanIn{nullptr, nullptr, nullptr, ps.eb[wave]},
                  false);
  lds_barrier();

  // 2. unions of the tokens' department and expert bitmaps, word prefixes
  if (wave == 0) {
    uint32_t u = 0;
    for (int t = 0; t < T; ++t) {
      const uint32_t v = lane < dwords ? tsm[t].db[lane] : 0u;
      const int c = __popc(v), s = wave_incl_scan(c);   // every lane takes part
      if (lane < dwords) {
        ps.db[t][lane] = v;
        ps.pd[t][lane] = s - c;
      }
      u |= v;
    }
    const int c = __popc(u), s = wave_incl_scan(c);
    if (lane < dwords) {
      ps.ud[lane] = u;
      ps.pud[lane] = s - c;
    }
    if (lane == 63) ps.nud = s;
  } else if (wave == 1) {
    uint32_t u = 0;
    for (int t = 0; t < T; ++t) {
      const uint32_t v = lane < ewords ? ps.eb[t][lane] : 0u;
      const int c = __popc(v);
      const int s = wave_incl_scan(c);
      if (lane < ewords) ps.pe[t][lane] = s - c;
      u |= v;
    }
    const int c = __popc(u), s = wave_incl_scan(c);
    if (lane < ewords) {
      ps.ue[lane] = u;
      ps.pue[lane] = s - c;
    }
    if (lane == 63) ps.nue = s;
  }
  lds_barrier();

  const bool slice = a.plan == PLAN_SLICE;
  const bool has_priv = slice && a.d_p > 0, has_se = a.d_se > 0;
  const int ud = uniform(ps.nud), ue = has_priv ? uniform(ps.nue) : 0;
  const int wb = a.w_bytes, ab = a.act_f32 ? 4 : 2, h = a.h;
  const char *x = static_cast<const char *>(a.x);
  const deamoe_weights &W = a.w;
  auto wptr = [&](const void *base, int i, int R, int C) -> const void * {
    return static_cast<const char *>(base) + (size_t)i * R * C * wb;
  };
  auto sptr = [&](const float *base, int i, int R, int C) -> const float * {
    return a.fp8 ? base + (size_t)i * ((R + 127) / 128) * (C / 128) : nullptr;
  };
  // member tokens and CSR offset of department j / expert e
  auto dept_members = [&](int j) {
    uint32_t mt = 0;
    for (int t = 0; t < T; ++t) mt |= ((ps.db[t][j >> 5] >> (j & 31)) & 1u) << t;
    return mt;
  };
  auto dept_off = [&](int j) {
    int o = 0;
    for (int t = 0; t < T; ++t) o += rank_pre(ps.db[t], ps.pd[t], j);
    return o;
  };
  auto exp_members = [&](int e) {
    uint32_t mt = 0;
    for (int t = 0; t < T; ++t) mt |= ((ps.eb[t][e >> 5] >> (e & 31)) & 1u) << t;
    return mt;
  };
  auto exp_off = [&](int e) {
    int o = 0;
    for (int t = 0; t < T; ++t) o += rank_pre(ps.eb[t], ps.pe[t], e);
    return o;
  };

  // 3. this workgroup's 16-row tiles of the first stage
  const int ia_d = (a.d_s + kTile - 1) / kTile, ia_e = has_priv ? (a.d_p + kTile - 1) / kTile : 0;
  const int ia_se = has_se ? (a.d_se + kTile - 1) / kTile : 0;
  const int total = ud * ia_d + ue * ia_e + ia_se;
  int32_t *idx = s_idx[wave];
  auto stream_tile = [&](int item) {
    GemmUnit U = {};
    uint32_t mt;
    int sigma = DEAMOE_SIGMA_SILU;
    U.epi = EPI_SWIGLU;
    if (item < ud * ia_d) {
      const int u = item / ia_d;
      item -= u * ia_d;
      const int j = wave_select(ps.ud, ps.pud, dwords, u);
      mt = dept_members(j);
      const size_t off = dept_off(j);
      U.w0 = wptr(W.dept_gate, j, a.d_s, h);
      U.w1 = wptr(W.dept_up, j, a.d_s, h);
      U.s0 = sptr(W.scale[0], j, a.d_s, h);
      U.s1 = sptr(W.scale[1], j, a.d_s, h);
      if (slice) {
        U.out0 = static_cast<char *>(a.abuf_dept) + off * a.d_s * ab;
      } else {   // FACTORED: sigma(W_g x) and sigma(W_u x) kept apart
        U.out0 = static_cast<char *>(a.gbuf) + off * a.d_s * ab;
        U.out1 = static_cast<char *>(a.ubuf) + off * a.d_s * ab;
        U.epi = EPI_SIGMA2;
        sigma = a.sigma;
      }
      U.R = a.d_s;
      U.ldout = a.d_s;
    } else if ((item -= ud * ia_d) < ue * ia_e) {
      const int u = item / ia_e;
      item -= u * ia_e;
      const int e = wave_select(ps.ue, ps.pue, ewords, u);
      mt = exp_members(e);
      const size_t off = exp_off(e);
      U.w0 = wptr(W.priv_gate, e, a.d_p, h);
      U.w1 = wptr(W.priv_up, e, a.d_p, h);
      U.s0 = sptr(W.scale[3], e, a.d_p, h);
      U.s1 = sptr(W.scale[4], e, a.d_p, h);
      U.out0 = static_cast<char *>(a.abuf_exp) + off * a.d_p * ab;
      U.R = a.d_p;
      U.ldout = a.d_p;
    } else {
      item -= ue * ia_e;   // the shared expert
      mt = (1u << T) - 1u;
      U.w0 = W.se_gate;
      U.w1 = W.se_up;
      U.s0 = sptr(W.scale[6], 0, a.d_se, h);
      U.s1 = sptr(W.scale[7], 0, a.d_se, h);
      U.out0 = a.abuf_se;
      U.R = a.d_se;
      U.ldout = a.d_se;
    }
    // the unit's tokens in ascending order, in this wave's LDS slot (the
    // previous tile's loads have all been issued: TileRunner ends with a
    // workgroup barrier)
    if (lane == 0) {
      int i = 0;
      for (int t = 0; t < T; ++t)
        if ((mt >> t) & 1u) idx[i++] = t;
    }
    wave_lds_sync();
    U.in0 = U.in1 = x;
    U.idx = idx;
    U.K = h;
    U.ldw = h;
    U.ldin = h;
    U.ntok = __popc(mt);
    U.out_f32 = a.act_f32;
    U.tpg = 1;
    Run::run(lds.run, &U, item, true, sigma);
  };
  if constexpr (PERSIST) {
    for (int it = blockIdx.x - 1; it < total; it += gridDim.x - 1) stream_tile(it);
  } else if ((int)blockIdx.x - 1 < total) {
    stream_tile(blockIdx.x - 1);
  }
}

// Workgroups of kernel K the current device holds at once (0 if unknown),
// queried once per device and kernel.
template <auto K>
static int resident_workgroups() {
  constexpr int kDevices = 64;
  static std::atomic<int> cache[kDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, K, 256, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    v = per_cu * cus;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// Gate/up tiles (two 16-row matrices) shorter than this stream in
// persistent workgroups when they outnumber the one-tile workgroups the chip
// holds at once.
constexpr size_t kPersistTileBytes = 256 << 10;

template <int WT, int NS>
static hipError_t launch_small_ns(const RouteArgs &a, int items, hipStream_t s) {
  const size_t tile_bytes = (size_t)2 * kTile * a.h * a.w_bytes;
  if (tile_bytes < kPersistTileBytes &&
      items >= resident_workgroups<small_route_gate_up_kernel<WT, NS, false>>()) {
    // one workgroup per tile up to what the chip holds at once (then each
    // streams several), plus the publishing workgroup
    constexpr auto kernel = small_route_gate_up_kernel<WT, NS, true>;
    const int slots = resident_workgroups<kernel>() - 1;
    const int g = slots > 0 ? std::min(items, slots) : items;
    hipLaunchKernelGGL(kernel, dim3(1 + std::max(g, 1)), dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((small_route_gate_up_kernel<WT, NS, false>), dim3(1 + items), dim3(256), 0,
                       s, a);
  }
  return hipGetLastError();
}

template <int WT>
static hipError_t launch_small_wt(const RouteArgs &a, int items, hipStream_t s) {
  switch (route_ns(a.n)) {
    case 1: return launch_small_ns<WT, 1>(a, items, s);
    case 2: return launch_small_ns<WT, 2>(a, items, s);
    case 4: return launch_small_ns<WT, 4>(a, items, s);
    case 8: return launch_small_ns<WT, 8>(a, items, s);
    case 16: return launch_small_ns<WT, 16>(a, items, s);
    default: return hipErrorInvalidValue;
  }
}

// One-tile workgroups of this kernel an MI355X holds at once: 256 CUs, three
// per CU for bf16 and fp32 weights (registers), four for fp8 (LDS).
constexpr int kCUs = 256;
static int single_tile_slots(int wtype) { return kCUs * (wtype == WT_FP8 ? 4 : 3) - 1; }

bool small_route_pays(int wtype, int n, int h, int w_bytes, bool group_limited, int items) {
  if (route_ns(n) > 16) return false;
  if (!group_limited) return true;                     // set-only top-k: a short prologue
  if ((size_t)2 * kTile * h * w_bytes < kPersistTileBytes) return true;   // routes once
  const int slots = single_tile_slots(wtype);          // (nearly) every tile in one round
  return items <= slots + slots / 8;
}

hipError_t launch_small_route_gate_up(const RouteArgs &a, int wtype, int items, hipStream_t s) {
  if (a.T < 1 || a.T > kSmallT || a.plan == PLAN_NONE || route_ns(a.n) > 16)
    return hipErrorInvalidValue;
  switch (wtype) {
    case WT_F32: return launch_small_wt<WT_F32>(a, items, s);
    case WT_BF16: return launch_small_wt<WT_BF16>(a, items, s);
    default: return launch_small_wt<WT_FP8>(a, items, s);
  }
}

}  // namespace deamoe
