// Batches of at most four tokens, SLICE form: routing (Eq. 2 and the
// department bookkeeping of Sec. 3.2), the gate/up stage of every active
// department, expert and the shared expert, and the unit table of the fused
// down kernel, in one launch after the router product.
//
// Every workgroup routes the tokens itself from the router's partial logits
// (one wave per token, results in LDS only) and derives its own work item
// from the step's active units instead of reading a unit table written by an
// earlier launch.  With short tiles (PERSIST) a workgroup routes once and
// then streams every (gridDim.x - 1)-th tile, the grid being sized to the
// workgroups the chip holds at once, so the routing is paid once per
// workgroup rather than once per tile; with long tiles each workgroup
// streams one, and the hardware hands a finishing workgroup's place to the
// next tile.  The units are ordered as the plan kernel orders them:
// active departments ascending, then active experts ascending, then the
// shared expert; a unit's member tokens are in ascending order and its
// gate/up output rows start at the unit's CSR offset, the sum of the member
// counts of the units of its kind before it.  Workgroup 0 publishes the
// routing (ids, weights, department lists, CSR lists, counts) and the fused
// down kernel's units; workgroup 1 + w streams 16-row tile w (PERSIST: and
// w + gridDim.x - 1, ...) of the step's gate/up pairs.  No workgroup reads
// anything another one of this launch writes.
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
  int32_t ids[kSmallT * kMaxK];        // [t][rank] selected expert
  int32_t dep[kSmallT * kMaxK];        // [t][slot] departments, -1 padded
  int32_t nd[kSmallT];
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

// The per-token routing scratch lives in the weight staging space, which is
// free until the first tile streams; the bitmaps that locate the tiles stay
// beside it.
template <int WT>
union SmallLds {
  typename TileRunner<WT, 2, 1, 4>::Smem run;
  TokSmem tsm[kSmallT];
};

template <int WT, int NS, bool PERSIST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
void small_route_gate_up_kernel(RouteArgs a) {
  using Run = TileRunner<WT, 2, 1, 4>;
  __shared__ SmallLds<WT> lds;
  __shared__ SmallSmem ps;
  __shared__ int32_t s_idx[kSmallT][kSmallT];   // per wave: member tokens of its unit
  TokSmem *tsm = lds.tsm;
  const int wave = uniform(threadIdx.x / kWave), lane = lane_id(), tid = threadIdx.x;
  const bool planner = blockIdx.x == 0;
  const int T = a.T, m = a.m, n = a.n, k = a.k;
  const int dwords = (m + 31) / 32, ewords = (n + 31) / 32;

  // 1. routing: wave t routes token t
  if (wave < T)
    route_one<NS>(a, wave, lane, tsm[wave],
                  PlanIn{ps.ids, ps.dep, ps.nd, ps.eb[wave]}, planner);
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

  const bool has_priv = a.d_p > 0, has_se = a.d_se > 0;
  const int ud = uniform(ps.nud), ue = has_priv ? uniform(ps.nue) : 0;
  const int wb = a.w_bytes, ab = a.act_f32 ? 4 : 2, h = a.h;
  const int kstep = wb == 4 ? 64 : 128;
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

  if (!planner) {
    // 3. this workgroup's 16-row tiles of the gate/up pairs
    const int ia_d = (a.d_s + kTile - 1) / kTile, ia_e = (a.d_p + kTile - 1) / kTile;
    const int ia_se = has_se ? (a.d_se + kTile - 1) / kTile : 0;
    const int total = ud * ia_d + ue * ia_e + ia_se;
    int32_t *idx = s_idx[wave];
    auto stream_tile = [&](int item) {
      GemmUnit U = {};
      uint32_t mt;
      if (item < ud * ia_d) {
        const int u = item / ia_d;
        item -= u * ia_d;
        const int j = wave_select(ps.ud, ps.pud, dwords, u);
        mt = dept_members(j);
        const int off = dept_off(j);
        U.w0 = wptr(W.dept_gate, j, a.d_s, h);
        U.w1 = wptr(W.dept_up, j, a.d_s, h);
        U.s0 = sptr(W.scale[0], j, a.d_s, h);
        U.s1 = sptr(W.scale[1], j, a.d_s, h);
        U.out0 = static_cast<char *>(a.abuf_dept) + (size_t)off * a.d_s * ab;
        U.R = a.d_s;
        U.ldout = a.d_s;
      } else if ((item -= ud * ia_d) < ue * ia_e) {
        const int u = item / ia_e;
        item -= u * ia_e;
        const int e = wave_select(ps.ue, ps.pue, ewords, u);
        mt = exp_members(e);
        const int off = exp_off(e);
        U.w0 = wptr(W.priv_gate, e, a.d_p, h);
        U.w1 = wptr(W.priv_up, e, a.d_p, h);
        U.s0 = sptr(W.scale[3], e, a.d_p, h);
        U.s1 = sptr(W.scale[4], e, a.d_p, h);
        U.out0 = static_cast<char *>(a.abuf_exp) + (size_t)off * a.d_p * ab;
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
      U.epi = EPI_SWIGLU;
      U.out_f32 = a.act_f32;
      U.tpg = 1;
      Run::run(lds.run, &U, item, true, DEAMOE_SIGMA_SILU);
    };
    if constexpr (PERSIST) {
      for (int it = blockIdx.x - 1; it < total; it += gridDim.x - 1) stream_tile(it);
    } else if ((int)blockIdx.x - 1 < total) {
      stream_tile(blockIdx.x - 1);
    }
    return;
  }

  // 4. workgroup 0: CSR lists, counts and the fused down kernel's units
  gmem<int32_t> *dept_count = glob(a.r.dept_count), *exp_count = glob(a.r.exp_count);
  gmem<int32_t> *dept_offset = glob(a.r.dept_offset), *exp_offset = glob(a.r.exp_offset);
  gmem<int32_t> *dept_tokens = glob(a.r.dept_tokens), *exp_tokens = glob(a.r.exp_tokens);
  int ndp = 0;
  for (int t = 0; t < T; ++t) ndp += ps.nd[t];
  for (int j = tid; j < m; j += blockDim.x) {
    dept_count[j] = __popc(dept_members(j));
    dept_offset[j] = dept_off(j);
  }
  for (int e = tid; e < n; e += blockDim.x) {
    exp_count[e] = __popc(exp_members(e));
    exp_offset[e] = exp_off(e);
  }
  if (tid == 0) {
    dept_offset[m] = ndp;
    exp_offset[n] = T * k;
  }
  for (int i = tid; i < T * k; i += blockDim.x) {
    const int t = i / k, q = i - t * k;
    const uint32_t below = (1u << t) - 1u;
    const int e = ps.ids[i];
    exp_tokens[exp_off(e) + __popc(exp_members(e) & below)] = t;
    if (q < ps.nd[t]) {
      const int j = ps.dep[i];
      dept_tokens[dept_off(j) + __popc(dept_members(j) & below)] = t;
    }
  }
  const int sd = a.d_s / kstep, sp = a.d_p / kstep;
  for (int j = tid; j < m; j += blockDim.x) {
    if (!((ps.ud[j >> 5] >> (j & 31)) & 1u)) continue;
    const int u = rank_pre(ps.ud, ps.pud, j);
    char *ao = static_cast<char *>(a.abuf_dept) + (size_t)dept_off(j) * a.d_s * ab;
    put_chain(glob(a.cunits) + u, wptr(W.dept_down, j, h, a.d_s), sptr(W.scale[2], j, h, a.d_s),
              ao, a.wdense + (size_t)j * kChainT, a.d_s, dept_members(j), u * sd);
  }
  if (has_priv) {
    for (int e = tid; e < n; e += blockDim.x) {
      if (!((ps.ue[e >> 5] >> (e & 31)) & 1u)) continue;
      const int ui = rank_pre(ps.ue, ps.pue, e);
      char *ao = static_cast<char *>(a.abuf_exp) + (size_t)exp_off(e) * a.d_p * ab;
      put_chain(glob(a.cunits) + ud + ui, wptr(W.priv_down, e, h, a.d_p),
                sptr(W.scale[5], e, h, a.d_p), ao, a.wdense + (size_t)(m + e) * kChainT, a.d_p,
                exp_members(e), ud * sd + ui * sp);
    }
  }
  // weight 1 of the shared expert: the row after the experts'
  if (tid < kChainT) glob(a.wdense)[(size_t)(m + n) * kChainT + tid] = 1.0f;
  if (tid == 0) {
    int units = ud + ue, steps = ud * sd + ue * sp;
    int items = ud * ((a.d_s + kTile - 1) / kTile) + ue * ((a.d_p + kTile - 1) / kTile);
    if (has_se) {
      put_chain(glob(a.cunits) + units, W.se_down, sptr(W.scale[8], 0, h, a.d_se), a.abuf_se,
                a.wdense + (size_t)(m + n) * kChainT, a.d_se, (1u << T) - 1u, steps);
      steps += a.d_se / kstep;
      items += (a.d_se + kTile - 1) / kTile;
      ++units;
    }
    gmem<PlanCounts> *counts = glob(a.counts);
    counts->stage[0][0] = units;
    counts->stage[0][1] = items;
    counts->stage[1][0] = units;
    counts->stage[1][1] = steps;
    counts->n_dept_pairs = ndp;
    counts->n_exp_pairs = has_priv ? T * k : 0;
    counts->n_pairs = ndp + (has_priv ? T * k : 0) + (has_se ? T : 0);
  }
}

// Workgroups of a kernel the current device holds at once (0 if unknown),
// queried once per device and kernel.
template <class K>
static int resident_workgroups(K kernel) {
  constexpr int kDevices = 64;
  static std::atomic<int> cache[kDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, 0) != hipSuccess ||
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
      items >= resident_workgroups(small_route_gate_up_kernel<WT, NS, false>)) {
    // one workgroup per tile up to what the chip holds at once (then each
    // streams several), plus the publishing workgroup
    auto kernel = small_route_gate_up_kernel<WT, NS, true>;
    const int slots = resident_workgroups(kernel) - 1;
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
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_small_route_gate_up(const RouteArgs &a, int wtype, int items, hipStream_t s) {
  if (a.T < 1 || a.T > kSmallT || a.plan != PLAN_SLICE || !a.chain || route_ns(a.n) > 8)
    return hipErrorInvalidValue;
  switch (wtype) {
    case WT_F32: return launch_small_wt<WT_F32>(a, items, s);
    case WT_BF16: return launch_small_wt<WT_BF16>(a, items, s);
    default: return launch_small_wt<WT_FP8>(a, items, s);
  }
}

}  // namespace deamoe
