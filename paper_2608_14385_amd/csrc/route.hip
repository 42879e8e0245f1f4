// Router (Eq. 2), department bookkeeping (Sec. 3.2) and the device-side plan
// of the expert stages.
//
// router_kernel: the logits W_r x as a grouped skinny product, split over KC
//   chunks of the hidden dimension so that the n x h router matrix is read by
//   many workgroups; each chunk's partial logits go to part[c][t][e] (rows
//   padded to 64 * NS values).
// route_token_kernel: one wave per token: logits = sum of the KC partials in
//   chunk order (+ bias, one fp32 add), optional group-limited department
//   choice, top-k by (logit desc, id asc), the routing weights, and the
//   token's distinct departments with P_{t,j}.
// plan_kernel: one workgroup: per-department and per-expert token lists in
//   ascending token order (no atomics on any order-sensitive value), the
//   unit tables of every expert stage (pointers, row-tile prefix), the
//   combine slots of every token, and the counts.
// route_plan_kernel: both of the above in one workgroup for batches of up
//   to four tokens, the per-token results passed on through LDS.
#include "route_dev.h"

namespace deamoe {

// --------------------------------------------------------------- router GEMV

template <int WT, int NTT>
__global__ __launch_bounds__(256) void router_kernel(RouterArgs a) {
  using Run = TileRunner<WT, 1, NTT, 4>;
  __shared__ typename Run::Smem sm;
  using Tr = WTraits<WT>;
  const int rt = blockIdx.x % a.tiles, c = blockIdx.x / a.tiles;
  GemmUnit U = {};
  U.w0 = static_cast<const char *>(a.w) + (size_t)c * a.kchunk * Tr::W_BYTES;
  U.in0 = U.in1 = static_cast<const char *>(a.x) + (size_t)c * a.kchunk * Tr::A_BYTES;
  U.idx = nullptr;
  U.out0 = a.part + (size_t)c * a.T * a.ldp;
  U.R = a.n;
  U.K = a.kchunk;
  U.ldw = a.h;
  U.ldin = a.h;
  U.ldout = a.ldp;
  U.ntok = a.T;
  U.epi = EPI_STORE;
  U.out_f32 = 1;
  U.tpg = 1;
  Run::run(sm, &U, rt, true, DEAMOE_SIGMA_NONE);
}

template <int WT>
static hipError_t router_ntt(const RouterArgs &a, int ntt, int kc, hipStream_t s) {
  dim3 grid(a.tiles * kc);
  switch (ntt) {
    case 1: hipLaunchKernelGGL((router_kernel<WT, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((router_kernel<WT, 2>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((router_kernel<WT, 4>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((router_kernel<WT, 8>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_router(const RouterArgs &a, int wtype, int ntt, int kc, hipStream_t s) {
  return wtype == WT_F32 ? router_ntt<WT_F32>(a, ntt, kc, s) : router_ntt<WT_BF16>(a, ntt, kc, s);
}

template <int NS>
__global__ __launch_bounds__(64) void route_token_kernel(RouteArgs a) {
  __shared__ TokSmem sm;
  route_one<NS>(a, blockIdx.x, threadIdx.x, sm);
}

// One workgroup: the per-department and per-expert token lists (ascending
// token order) from the per-token results, then the unit tables of every
// expert stage and the combine slots.
//
// Membership is kept as token bitmaps in LDS for every expert and
// department.  A token's position in a CSR list is the offset of the list
// plus the number of member tokens below it, so every (token, rank) pair is
// placed independently.  Counts and the number of active units are summed
// in one scan over departments then experts, packed as count | active << 16
// (both sums stay below 2^16).
struct PlanSmem {
  int32_t ids[kMaxTK];               // [t][rank] selected expert
  int32_t dep[kMaxTK];               // [t][slot] departments, -1 padded
  uint32_t etok[kMaxN * kTW];        // [e] token bitmap
  uint32_t dtok[kMaxM * kTW];        // [j] token bitmap
  int32_t scan[kMaxM + kMaxN];       // [depts, experts] packed prefix
  int32_t nd[kMaxT];
  int32_t tmp[64];
};

// Every thread of the workgroup (BT threads) calls it.  LDS_IN: the
// per-token results are already in sm.ids, sm.dep and sm.nd.
template <int BT, bool LDS_IN = false>
__device__ __attribute__((always_inline)) void plan_body(const RouteArgs &a, PlanSmem &sm) {
  constexpr int EPT = kMaxN / BT;   // experts per thread in the per-expert loops
  int32_t *s_ids = sm.ids, *s_dep = sm.dep, *s_scan = sm.scan, *s_nd = sm.nd, *s_tmp = sm.tmp;
  uint32_t *s_etok = sm.etok, *s_dtok = sm.dtok;
  const int tid = threadIdx.x;
  const int T = a.T, n = a.n, m = a.m, k = a.k, E = a.E;
  const int tw = (T + 31) / 32;
  const bool slice = a.plan == PLAN_SLICE;
  const bool exp_slots = slice && a.d_p > 0;
  const bool has_priv = a.plan == PLAN_FACTORED || a.d_p > 0;
  const bool has_se = a.d_se > 0;
  const int S = a.max_slots;
  gmem<int32_t> *dept_count = glob(a.r.dept_count), *exp_count = glob(a.r.exp_count);
  gmem<int32_t> *dept_offset = glob(a.r.dept_offset), *exp_offset = glob(a.r.exp_offset);
  gmem<int32_t> *dept_tokens = glob(a.r.dept_tokens), *exp_tokens = glob(a.r.exp_tokens);
  gmem<int32_t> *slot_pair = glob(a.slot_pair), *tok_exp_pair = glob(a.tok_exp_pair);
  gmem<int32_t> *exp_src = glob(a.exp_src), *pair_dept = glob(a.pair_dept);
  gmem<PlanCounts> *counts = glob(a.counts);
  for (int i = tid; i < n * kTW; i += BT) s_etok[i] = 0;
  for (int i = tid; i < m * kTW; i += BT) s_dtok[i] = 0;
  lds_barrier();
  for (int idx = tid; idx < T * k; idx += BT) {
    const int t = idx / k;
    const uint32_t bit = 1u << (t & 31);
    const int e = LDS_IN ? s_ids[idx] : glob(a.r.topk_ids)[idx];
    const int j = LDS_IN ? s_dep[idx] : glob(a.r.tok_depts)[idx];
    if (!LDS_IN) {
      s_ids[idx] = e;
      s_dep[idx] = j;
    }
    atomicOr(&s_etok[e * kTW + (t >> 5)], bit);
    if (j >= 0) atomicOr(&s_dtok[j * kTW + (t >> 5)], bit);
  }
  if (!LDS_IN)
    for (int t = tid; t < T; t += BT) s_nd[t] = glob(a.r.tok_ndept)[t];
  lds_barrier();

  // counts
  int my_dc = 0, my_ec[EPT] = {};
  if (tid < m) {
    for (int w = 0; w < tw; ++w) my_dc += __popc(s_dtok[tid * kTW + w]);
    dept_count[tid] = my_dc;
    s_scan[tid] = my_dc | ((my_dc > 0) << 16);
  }
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = tid + q * BT;
    if (e < n) {
      int c = 0;
      for (int w = 0; w < tw; ++w) c += __popc(s_etok[e * kTW + w]);
      my_ec[q] = c;
      exp_count[e] = c;
      s_scan[m + e] = c | ((has_priv && c > 0) << 16);
    }
  }
  lds_barrier();
  const int tot = block_exscan(s_scan, m + n, s_tmp);
  const int ndp = s_scan[m] & 0xffff, ud = s_scan[m] >> 16;
  const int nep = (tot & 0xffff) - ndp, ue = (tot >> 16) - ud;
  const int nep_priv = has_priv ? nep : 0;
  auto doff = [&](int j) { return s_scan[j] & 0xffff; };
  auto eoff = [&](int e) { return (s_scan[m + e] & 0xffff) - ndp; };
  if (tid < m) dept_offset[tid] = doff(tid);
  for (int e = tid; e < n; e += BT) exp_offset[e] = eoff(e);
  if (tid == 0) {
    dept_offset[m] = ndp;
    exp_offset[n] = nep;
  }
  // every (token, rank) pair places itself: the expert of that rank and, for
  // ranks below the token's department count, the department of that slot
  for (int idx = tid; idx < T * k; idx += BT) {
    const int t = idx / k, q = idx - t * k;
    const int e = s_ids[idx];
    const int pe = eoff(e) + rank_below(s_etok + e * kTW, t);
    exp_tokens[pe] = t;
    if (a.plan) {
      tok_exp_pair[idx] = pe;
      if (exp_slots) slot_pair[(size_t)t * S + s_nd[t] + q] = ndp + pe;
      if (a.plan == PLAN_FACTORED) {
        const int j = e / E;
        exp_src[pe] = doff(j) + rank_below(s_dtok + j * kTW, t);
      }
    }
    const int j = s_dep[idx];
    if (j >= 0) {
      const int pd = doff(j) + rank_below(s_dtok + j * kTW, t);
      dept_tokens[pd] = t;
      if (a.plan) slot_pair[(size_t)t * S + q] = pd;
      if (a.plan == PLAN_FACTORED) pair_dept[pd] = j;
    }
  }
  if (!a.plan) return;
  if (has_se)
    for (int t = tid; t < T; t += BT)
      slot_pair[(size_t)t * S + s_nd[t] + (exp_slots ? k : 0)] = ndp + (slice ? nep_priv : 0) + t;

  // unit tables: unit index of an active department / expert = number of
  // active ones before it.  A unit's work items are its row-tile items times
  // its token groups (wave_tokens tokens each).  Item prefixes over the units
  // in table order are closed forms while no unit has more than one group;
  // otherwise they come from block scans over an array with every
  // department's items, then every expert's (the expert bitmaps' LDS, free
  // after the placement above).
  const int wb = a.w_bytes, ab = a.act_f32 ? 4 : 2;
  const char *x = static_cast<const char *>(a.x);
  auto wptr = [&](const void *base, int idx, int R, int C) -> const void * {
    return static_cast<const char *>(base) + (size_t)idx * R * C * wb;
  };
  auto sptr = [&](const float *base, int idx, int R, int C) -> const float * {
    if (!a.fp8) return nullptr;
    return base + (size_t)idx * ((R + 127) / 128) * (C / 128);
  };
  const deamoe_weights &W = a.w;
  const int wt = a.wave_tokens;
  const bool multi = T > wt;
  auto groups = [&](int cnt) { return multi ? (cnt + wt - 1) / wt : 1; };
  int32_t *s_ia = reinterpret_cast<int32_t *>(s_etok);           // [m + n] items, stage pair A
  int32_t *s_ib = s_ia + kMaxM + kMaxN;                           // [m + n] items, stage pair B
  const int dr = a.down_rows, dk = a.down_ks;
  // items per row-tile item: (A dept, A expert, B dept, B expert)
  int ia_d, ia_e, ib_d, ib_e;
  if (slice) {
    const int gd = tiles_per_item(a.d_s, dr, dk), gp = a.d_p ? tiles_per_item(a.d_p, dr, dk) : 1;
    ia_d = (a.d_s + kTile - 1) / kTile;
    ia_e = has_priv ? (a.d_p + kTile - 1) / kTile : 0;
    ib_d = items_of(a.h, gd, dr);
    ib_e = has_priv ? items_of(a.h, gp, dr) : 0;
  } else {
    const int d = a.d_s;
    const int gd = tiles_per_item(d, dr, dk), g2 = tiles_per_item(d, dr, dk);
    ia_d = (d + kTile - 1) / kTile;   // stage 0: W_g, W_u
    ia_e = ia_d;                      // stage 1: A_g, A_u
    ib_d = items_of(a.h, gd, dr);     // stage 3: W_d^T
    ib_e = items_of(d, g2, dr);       // stage 2: A_d^T
  }
  int tot_a = 0, tot_b = 0;
  if (multi) {
    lds_barrier();   // the expert bitmaps are no longer read
    if (tid < m) {
      s_ia[tid] = my_dc > 0 ? ia_d * groups(my_dc) : 0;
      s_ib[tid] = my_dc > 0 ? ib_d * groups(my_dc) : 0;
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      const int e = tid + q * BT;
      if (e < n) {
        const bool act = has_priv && my_ec[q] > 0;
        s_ia[m + e] = act ? ia_e * groups(my_ec[q]) : 0;
        s_ib[m + e] = act ? ib_e * groups(my_ec[q]) : 0;
      }
    }
    lds_barrier();
    const int2 tot = block_exscan2(s_ia, s_ib, m + n, s_tmp);
    tot_a = tot.x;
    tot_b = tot.y;
  } else {
    tot_a = ud * ia_d + ue * ia_e;
    tot_b = ud * ib_d + ue * ib_e;
  }
  // first item of department j / expert e (unit index uj / ue_e) in each pair
  auto dbeg_a = [&](int j, int uj) { return multi ? s_ia[j] : uj * ia_d; };
  auto dbeg_b = [&](int j, int uj) { return multi ? s_ib[j] : uj * ib_d; };
  auto ebeg_a = [&](int e, int ui) { return multi ? s_ia[m + e] : ud * ia_d + ui * ia_e; };
  auto ebeg_b = [&](int e, int ui) { return multi ? s_ib[m + e] : ud * ib_d + ui * ib_e; };
  const int dept_a = multi ? s_ia[m] : ud * ia_d;   // items of all departments
  const int dept_b = multi ? s_ib[m] : ud * ib_d;
  const int kstep = a.w_bytes == 4 ? 64 : 128;   // K step of the weight type
  if (slice) {
    const int gd = tiles_per_item(a.d_s, dr, dk), gp = a.d_p ? tiles_per_item(a.d_p, dr, dk) : 1;
    const int gse = a.d_se ? tiles_per_item(a.d_se, dr, dk) : 1;
    const int bse = items_of(a.h, gse, dr);
    // fused down stage (T <= 32): the units' K steps are concatenated in
    // table order (departments, experts, the shared expert)
    const int sd = a.d_s / kstep, sp = a.d_p / kstep;
    if (tid < m && my_dc > 0) {
      const int j = tid, u = s_scan[j] >> 16, off = doff(j);
      const int32_t *idx = a.r.dept_tokens + off;
      char *ao = static_cast<char *>(a.abuf_dept) + (size_t)off * a.d_s * ab;
      put_unit(glob(a.units[0]) + u, wptr(W.dept_gate, j, a.d_s, a.h), wptr(W.dept_up, j, a.d_s, a.h),
               sptr(W.scale[0], j, a.d_s, a.h), sptr(W.scale[1], j, a.d_s, a.h), x, x, idx, ao,
               nullptr, a.d_s, a.h, a.h, a.d_s, my_dc, dbeg_a(j, u), EPI_SWIGLU, a.act_f32);
      if (a.chain)
        put_chain(glob(a.cunits) + u, wptr(W.dept_down, j, a.h, a.d_s),
                  sptr(W.scale[2], j, a.h, a.d_s), ao, a.wdense + (size_t)j * kChainT, a.d_s,
                  s_dtok[j * kTW], u * sd);
      else
        put_unit(glob(a.units[1]) + u, wptr(W.dept_down, j, a.h, a.d_s), nullptr,
                 sptr(W.scale[2], j, a.h, a.d_s), nullptr, ao, ao, nullptr,
                 a.partial + (size_t)off * a.h, nullptr, a.h, a.d_s, a.d_s, a.h, my_dc,
                 dbeg_b(j, u), EPI_STORE, 1, gd);
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      const int e = tid + q * BT;
      if (!has_priv || e >= n || my_ec[q] == 0) continue;
      const int ui = (s_scan[m + e] >> 16) - ud, u = ud + ui, off = eoff(e);
      const int32_t *idx = a.r.exp_tokens + off;
      char *ao = static_cast<char *>(a.abuf_exp) + (size_t)off * a.d_p * ab;
      put_unit(glob(a.units[0]) + u, wptr(W.priv_gate, e, a.d_p, a.h), wptr(W.priv_up, e, a.d_p, a.h),
               sptr(W.scale[3], e, a.d_p, a.h), sptr(W.scale[4], e, a.d_p, a.h), x, x, idx, ao,
               nullptr, a.d_p, a.h, a.h, a.d_p, my_ec[q], ebeg_a(e, ui), EPI_SWIGLU,
               a.act_f32);
      if (a.chain)
        put_chain(glob(a.cunits) + u, wptr(W.priv_down, e, a.h, a.d_p),
                  sptr(W.scale[5], e, a.h, a.d_p), ao, a.wdense + (size_t)(m + e) * kChainT, a.d_p,
                  s_etok[e * kTW], ud * sd + ui * sp);
      else
        put_unit(glob(a.units[1]) + u, wptr(W.priv_down, e, a.h, a.d_p), nullptr,
                 sptr(W.scale[5], e, a.h, a.d_p), nullptr, ao, ao, nullptr,
                 a.partial + (size_t)(ndp + off) * a.h, nullptr, a.h, a.d_p, a.d_p, a.h,
                 my_ec[q], ebeg_b(e, ui), EPI_STORE, 1, gp);
    }
    // weight 1 of the shared expert: the row after the experts'
    if (a.chain && tid < kChainT) glob(a.wdense)[(size_t)(m + n) * kChainT + tid] = 1.0f;
    if (tid == 0) {
      int units = ud + ue, items_a = tot_a, items_b = tot_b;
      int steps = ud * sd + ue * sp;
      if (has_se) {
        put_unit(glob(a.units[0]) + units, W.se_gate, W.se_up, sptr(W.scale[6], 0, a.d_se, a.h),
                 sptr(W.scale[7], 0, a.d_se, a.h), x, x, nullptr, a.abuf_se, nullptr, a.d_se, a.h,
                 a.h, a.d_se, T, items_a, EPI_SWIGLU, a.act_f32);
        if (a.chain) {
          put_chain(glob(a.cunits) + units, W.se_down, sptr(W.scale[8], 0, a.h, a.d_se), a.abuf_se,
                    a.wdense + (size_t)(m + n) * kChainT, a.d_se,
                    T >= 32 ? 0xffffffffu : (1u << T) - 1u, steps);
          steps += a.d_se / kstep;
        } else {
          put_unit(glob(a.units[1]) + units, W.se_down, nullptr, sptr(W.scale[8], 0, a.h, a.d_se),
                   nullptr, a.abuf_se, a.abuf_se, nullptr,
                   a.partial + (size_t)(ndp + nep_priv) * a.h, nullptr, a.h, a.d_se, a.d_se, a.h,
                   T, items_b, EPI_STORE, 1, gse);
        }
        items_a += (a.d_se + kTile - 1) / kTile * groups(T);
        items_b += bse * groups(T);
        ++units;
      }
      counts->stage[0][0] = units;
      counts->stage[0][1] = items_a;
      counts->stage[1][0] = units;
      counts->stage[1][1] = a.chain ? steps : items_b;
    }
  } else {  // PLAN_FACTORED
    const int d = a.d_s;
    const int gd = tiles_per_item(d, dr, dk), gse = a.d_se ? tiles_per_item(a.d_se, dr, dk) : 1;
    const int bse = items_of(a.h, gse, dr);
    const int g2 = tiles_per_item(d, dr, dk);   // A_d^T: d x d, streamed like the down projections
    if (tid < m && my_dc > 0) {
      const int j = tid, u = s_scan[j] >> 16, off = doff(j);
      const int32_t *idx = a.r.dept_tokens + off;
      char *go = static_cast<char *>(a.gbuf) + (size_t)off * d * ab;
      char *uo = static_cast<char *>(a.ubuf) + (size_t)off * d * ab;
      char *zs = static_cast<char *>(a.zsbuf) + (size_t)off * d * ab;
      put_unit(glob(a.units[0]) + u, wptr(W.dept_gate, j, d, a.h), wptr(W.dept_up, j, d, a.h),
               sptr(W.scale[0], j, d, a.h), sptr(W.scale[1], j, d, a.h), x, x, idx, go, uo, d,
               a.h, a.h, d, my_dc, dbeg_a(j, u), EPI_SIGMA2, a.act_f32);
      if (a.chain)   // Z already carries the routing weights: unit weight 1
        put_chain(glob(a.cunits) + u, wptr(W.dept_down, j, a.h, d), sptr(W.scale[2], j, a.h, d), zs,
                  a.wdense + (size_t)(m + n) * kChainT, d, s_dtok[j * kTW], u * (d / kstep));
      else
        put_unit(glob(a.units[3]) + u, wptr(W.dept_down, j, a.h, d), nullptr,
                 sptr(W.scale[2], j, a.h, d), nullptr, zs, zs, nullptr,
                 a.partial + (size_t)off * a.h, nullptr, a.h, d, d, a.h, my_dc, dbeg_b(j, u),
                 EPI_STORE, 1, gd);
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      const int e = tid + q * BT;
      if (e >= n || my_ec[q] == 0) continue;
      const int u = (s_scan[m + e] >> 16) - ud, off = eoff(e);
      char *yo = static_cast<char *>(a.ybuf) + (size_t)off * d * ab;
      put_unit(glob(a.units[1]) + u, wptr(W.priv_gate, e, d, d), wptr(W.priv_up, e, d, d),
               sptr(W.scale[3], e, d, d), sptr(W.scale[4], e, d, d), a.gbuf, a.ubuf,
               a.exp_src + off, yo, nullptr, d, d, d, d, my_ec[q], ebeg_a(e, u) - dept_a,
               EPI_SWIGLU, a.act_f32);
      put_unit(glob(a.units[2]) + u, wptr(W.priv_down, e, d, d), nullptr, sptr(W.scale[5], e, d, d),
               nullptr, yo, yo, nullptr, a.zbuf + (size_t)off * d, nullptr, d, d, d, d,
               my_ec[q], ebeg_b(e, u) - dept_b, EPI_SIGMA, 1, g2);
    }
    if (a.chain && tid < kChainT) glob(a.wdense)[(size_t)(m + n) * kChainT + tid] = 1.0f;
    if (tid == 0) {
      int units0 = ud, items0 = dept_a, units3 = ud, items3 = dept_b;
      int steps = ud * (d / kstep);
      if (has_se) {
        put_unit(glob(a.units[0]) + units0, W.se_gate, W.se_up, sptr(W.scale[6], 0, a.d_se, a.h),
                 sptr(W.scale[7], 0, a.d_se, a.h), x, x, nullptr, a.abuf_se, nullptr, a.d_se, a.h,
                 a.h, a.d_se, T, items0, EPI_SWIGLU, a.act_f32);
        if (a.chain) {
          put_chain(glob(a.cunits) + units3, W.se_down, sptr(W.scale[8], 0, a.h, a.d_se), a.abuf_se,
                    a.wdense + (size_t)(m + n) * kChainT, a.d_se,
                    T >= 32 ? 0xffffffffu : (1u << T) - 1u, steps);
          steps += a.d_se / kstep;
        } else {
          put_unit(glob(a.units[3]) + units3, W.se_down, nullptr, sptr(W.scale[8], 0, a.h, a.d_se),
                   nullptr, a.abuf_se, a.abuf_se, nullptr, a.partial + (size_t)ndp * a.h,
                   nullptr, a.h, a.d_se, a.d_se, a.h, T, items3, EPI_STORE, 1, gse);
        }
        ++units0;
        items0 += (a.d_se + kTile - 1) / kTile * groups(T);
        ++units3;
        items3 += bse * groups(T);
      }
      if (a.chain) items3 = steps;
      counts->stage[0][0] = units0;
      counts->stage[0][1] = items0;
      counts->stage[1][0] = ue;
      counts->stage[1][1] = tot_a - dept_a;
      counts->stage[2][0] = ue;
      counts->stage[2][1] = tot_b - dept_b;
      counts->stage[3][0] = units3;
      counts->stage[3][1] = items3;
    }
  }
  if (tid == 0) {
    counts->n_dept_pairs = ndp;
    counts->n_exp_pairs = nep_priv;
    counts->n_pairs = ndp + (slice ? nep_priv : 0) + (has_se ? T : 0);
  }
}

template <int BT>
__global__ __launch_bounds__(BT) void plan_kernel(RouteArgs a) {
  __shared__ PlanSmem sm;
  __shared__ RouteArgs sa;
  args_to_lds<BT>(a, sa);
  lds_barrier();
  plan_body<BT>(sa, sm);
}

// Batches of at most kFusedMaxT tokens route and plan in one workgroup: wave
// t routes token t (one routing wave per SIMD) and leaves its results in LDS
// as well, and the plan starts after a barrier that waits for LDS only (the
// results' global stores complete in the background).  Larger batches route
// in a workgroup per token, which spreads the routing over as many CUs.
// Wider routers (more experts per lane) take fewer waves for the plan, which
// leaves each wave more registers.
constexpr int kFusedMaxT = 4;
template <int NS>
constexpr int fused_waves() { return NS <= 4 ? 16 : NS <= 16 ? 8 : 4; }

template <int NS>
__global__ __launch_bounds__(fused_waves<NS>() * 64) void route_plan_kernel(RouteArgs a) {
  __shared__ TokSmem tsm[fused_waves<NS>()];
  __shared__ PlanSmem psm;
  __shared__ RouteArgs sa;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  args_to_lds<fused_waves<NS>() * 64>(a, sa);
  if (w < a.T) route_one<NS>(a, w, lane, tsm[w], PlanIn{psm.ids, psm.dep, psm.nd, nullptr});
  lds_barrier();
  plan_body<fused_waves<NS>() * 64, true>(sa, psm);
}

template <int NS>
static hipError_t launch_route_ns(const RouteArgs &a, hipStream_t s) {
  if (a.T <= kFusedMaxT) {
    hipLaunchKernelGGL((route_plan_kernel<NS>), dim3(1), dim3(fused_waves<NS>() * 64), 0, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((route_token_kernel<NS>), dim3(a.T), dim3(64), 0, s, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((plan_kernel<1024>), dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_route(const RouteArgs &a, hipStream_t s) {
  switch (route_ns(a.n)) {
    case 1: return launch_route_ns<1>(a, s);
    case 2: return launch_route_ns<2>(a, s);
    case 4: return launch_route_ns<4>(a, s);
    case 8: return launch_route_ns<8>(a, s);
    case 16: return launch_route_ns<16>(a, s);
    default: return launch_route_ns<32>(a, s);
  }
}

}  // namespace deamoe
