// Device helpers of the routing kernels: wave reductions and scans, order
// keys, LDS-only barriers, unit-table writers, and route_one (one wave routes
// one token: Eq. 2 top-k, routing weights, departments of Sec. 3.2).
#pragma once

#include "gemm_tile.h"
#include "launch.h"

namespace deamoe {
// ------------------------------------------------------------ route and plan

__device__ inline bool ranks_before(float va, int a, float vb, int b) {
  return va > vb || (va == vb && a < b);
}

// Order-preserving map of a float onto an unsigned int (larger float, larger
// key).  -0 takes the key of +0: the two are equal values, so a tie between
// them goes to the lower expert id like any other tie.
__device__ inline uint32_t ord_u32(float f) {
  uint32_t u = __float_as_uint(f);
  u = u == 0x80000000u ? 0u : u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Wave-wide maximum of a 64-bit key, returned to every lane: DPP exchanges
// within each row of 16 lanes (xor 1, xor 2, half-row mirror, row mirror),
// then the four row maxima through readlane.
__device__ inline uint64_t wave_max_u64(uint64_t v) {
#define DEAMOE_DPP_STEP(ctrl)                                                               \
  do {                                                                                      \
    const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);                              \
    const uint32_t olo = __builtin_amdgcn_update_dpp(lo, lo, ctrl, 0xf, 0xf, false);        \
    const uint32_t ohi = __builtin_amdgcn_update_dpp(hi, hi, ctrl, 0xf, 0xf, false);        \
    const uint64_t o = ((uint64_t)ohi << 32) | olo;                                         \
    v = o > v ? o : v;                                                                      \
  } while (0)
  DEAMOE_DPP_STEP(0xB1);    // quad_perm [1,0,3,2]
  DEAMOE_DPP_STEP(0x4E);    // quad_perm [2,3,0,1]
  DEAMOE_DPP_STEP(0x141);   // row_half_mirror
  DEAMOE_DPP_STEP(0x140);   // row_mirror
#undef DEAMOE_DPP_STEP
  uint64_t best = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, 16 * r);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), 16 * r);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    best = o > best ? o : best;
  }
  return best;
}

// DPP exchange of a 32-bit value within rows of 16 lanes.
template <int CTRL>
__device__ inline float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL,
                                                    0xf, 0xf, false));
}

// Wave-wide sum / maximum returned to every lane: butterflies within each row
// of 16 lanes (xor 1, xor 2, half-row mirror, row mirror), then the four row
// results through readlane, combined in row order.
__device__ inline float wave_sum(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x141>(v);
  v += dpp_f32<0x140>(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return ((r0 + r1) + r2) + r3;
}

__device__ inline float wave_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  v = fmaxf(v, dpp_f32<0x140>(v));
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

// Inclusive prefix sum over the wave: shifts by 1, 2, 4, 8 within each row
// of 16 lanes (lanes shifted in from outside the row add 0), then the row
// totals below each lane's row through readlane.
__device__ inline int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
  const int lane = __lane_id();
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47);
  return v + (lane >= 16 ? r0 : 0) + (lane >= 32 ? r1 : 0) + (lane >= 48 ? r2 : 0);
}

// Order-preserving float <-> int map for integer max.
__device__ inline int ord_key(float f) {
  const int i = __float_as_int(f);
  return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ inline float ord_val(int i) { return __int_as_float(i >= 0 ? i : i ^ 0x7fffffff); }

// Workgroup barrier that orders LDS accesses only: global stores issued
// before it may still be in flight.  The route and plan kernels never read
// back, within a launch, global data they wrote, so their barriers need no
// more (a full barrier would wait for every outstanding store).
__device__ inline void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Exclusive prefix sum of s[0..N) in place, N <= 4 * blockDim; returns the
// total.  Every thread of the block must call it.
__device__ inline int block_exscan(int32_t *s, int N, int32_t *s_tmp) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int nwaves = nt / 64;
  const int per = (N + nt - 1) / nt;
  const int b = min(tid * per, N), e = min(b + per, N);
  int local = 0;
  for (int i = b; i < e; ++i) local += s[i];
  const int v = wave_incl_scan(local);
  if (lane == 63) s_tmp[wave] = v;
  lds_barrier();
  if (wave == 0) {
    const int w = wave_incl_scan(lane < nwaves ? s_tmp[lane] : 0);
    if (lane < nwaves) s_tmp[lane] = w;
  }
  lds_barrier();
  int run = (wave > 0 ? s_tmp[wave - 1] : 0) + v - local;
  for (int i = b; i < e; ++i) {
    const int x = s[i];
    s[i] = run;
    run += x;
  }
  const int total = s_tmp[nwaves - 1];
  lds_barrier();
  return total;
}

// Exclusive prefix sums of two arrays a[0..N) and b[0..N) in place, in one
// pass (shared barriers); returns both totals.  Every thread of the block
// must call it; s_tmp holds 2 * (blockDim / 64) values.
__device__ inline int2 block_exscan2(int32_t *a, int32_t *b, int N, int32_t *s_tmp) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int nwaves = nt / 64;
  const int per = (N + nt - 1) / nt;
  const int lo = min(tid * per, N), hi = min(lo + per, N);
  int la = 0, lb = 0;
  for (int i = lo; i < hi; ++i) {
    la += a[i];
    lb += b[i];
  }
  const int va = wave_incl_scan(la), vb = wave_incl_scan(lb);
  if (lane == 63) {
    s_tmp[wave] = va;
    s_tmp[32 + wave] = vb;
  }
  lds_barrier();
  if (wave == 0) {
    const int wa = wave_incl_scan(lane < nwaves ? s_tmp[lane] : 0);
    const int wb = wave_incl_scan(lane < nwaves ? s_tmp[32 + lane] : 0);
    if (lane < nwaves) {
      s_tmp[lane] = wa;
      s_tmp[32 + lane] = wb;
    }
  }
  lds_barrier();
  int ra = (wave > 0 ? s_tmp[wave - 1] : 0) + va - la;
  int rb = (wave > 0 ? s_tmp[32 + wave - 1] : 0) + vb - lb;
  for (int i = lo; i < hi; ++i) {
    const int xa = a[i], xb = b[i];
    a[i] = ra;
    b[i] = rb;
    ra += xa;
    rb += xb;
  }
  const int2 total = make_int2(s_tmp[nwaves - 1], s_tmp[32 + nwaves - 1]);
  lds_barrier();
  return total;
}

__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

constexpr int kMaxKC = 16;   // router chunks (host caps the split)

// Fill one unit of a stage table field by field (no temporary struct).
__device__ inline void put_unit(gmem<GemmUnit> *U, const void *w0, const void *w1, const float *s0,
                                const float *s1, const void *in0, const void *in1,
                                const int32_t *idx, void *out0, void *out1, int R, int K, int ldin,
                                int ldout, int ntok, int tile_begin, int epi, int out_f32,
                                int tpg = 1) {
  U->w0 = w0; U->w1 = w1; U->s0 = s0; U->s1 = s1; U->in0 = in0; U->in1 = in1; U->idx = idx;
  U->out0 = out0; U->out1 = out1; U->R = R; U->K = K; U->ldw = K; U->ldin = ldin;
  U->ldout = ldout; U->ntok = ntok; U->tile_begin = tile_begin; U->epi = epi;
  U->out_f32 = out_f32; U->tpg = tpg;
}

__device__ inline void put_chain(gmem<ChainUnit> *U, const void *w, const float *s, const void *in,
                                 const float *pw, int K, uint32_t mask, int step0) {
  U->w = w; U->s = s; U->in = in; U->pw = pw; U->K = K; U->mask = mask; U->step0 = step0;
  U->pad_ = 0;
}

// Row tiles per work item of a stage whose K is not split across waves: short
// contractions take several tiles so that a work item streams enough bytes.
__device__ inline int tiles_per_item(int K, int rows, int ks) {
  if (ks > 1) return 1;
  int t = max(1, min(8, 2048 * kTile / (rows * K)));
  // fp8: the item's block scales, (t * rows / 128 + 1) scale rows of K / 128,
  // fit the 64-entry window of a work item
  while (t > 1 && (t * rows / 128 + 1) * (K / 128) > 64) --t;
  return t;
}
__device__ inline int items_of(int R, int tpg, int rows) {
  return ((R + rows - 1) / rows + tpg - 1) / tpg;
}

__device__ inline bool bit_at(const uint32_t *row, int i) { return (row[i >> 5] >> (i & 31)) & 1; }

// Number of set bits below bit i of a bitmap row.
__device__ inline int rank_below(const uint32_t *row, int i) {
  int r = 0;
  for (int w = 0; w < (i >> 5); ++w) r += __popc(row[w]);
  return r + __popc(row[i >> 5] & ((1u << (i & 31)) - 1u));
}

constexpr int kTW = kMaxT / 32;   // words of a token bitmap
constexpr int kDW = kMaxM / 32;   // words of a department bitmap

// NS consecutive fp32 values at p (aligned to 4 * NS bytes up to 16).
template <int NS>
__device__ inline void load_run(const float *p, float (&v)[NS]) {
  if constexpr (NS == 1) {
    v[0] = *p;
  } else if constexpr (NS == 2) {
    const float2 q = *reinterpret_cast<const float2 *>(p);
    v[0] = q.x;
    v[1] = q.y;
  } else {
#pragma unroll
    for (int i = 0; i < NS / 4; ++i) {
      const f32x4 q = *reinterpret_cast<const f32x4 *>(p + 4 * i);
      v[4 * i] = q[0];
      v[4 * i + 1] = q[1];
      v[4 * i + 2] = q[2];
      v[4 * i + 3] = q[3];
    }
  }
}

__device__ inline int popc64(uint64_t v) { return __popcll(v); }

// One wave routes one token: logits, optional group limit, top-k, routing
// weights and the token's distinct departments with P_{t,j}; the token's
// combine slots when a plan follows.
//
// Top-k works on order keys (a monotone map of the logit to an unsigned
// int).  A threshold is found by radix selection (built bit by bit from the
// top; a bit stays if at least k keys reach the value), first over the
// per-lane maxima; the few candidates at or above it rank themselves by
// (logit desc, id asc) through LDS.
struct TokSmem {
  uint64_t sel[64];                  // candidates in expert order
  uint64_t ord[kMaxK];               // winners in rank order
  int32_t gs[kMaxMGrouped];          // department scores (group limit)
  uint32_t db[kDW];                  // the token's department bitmap
};

// Per-token results handed to a plan in the same workgroup through LDS
// (all null when the plan runs as its own kernel).
// eb: optional bitmap of the token's selected experts (ceil(n / 32) words).
struct PlanIn {
  int32_t *ids, *dep, *nd;
  uint32_t *eb;
};

// gw: write the routing results to global memory (false: LDS outputs only,
// for workgroups that need the routing but do not publish it).
template <int NS>
__device__ __attribute__((always_inline)) void route_one(const RouteArgs &a, const int t,
                                                        const int lane, TokSmem &sm,
                                                        PlanIn lds = {nullptr, nullptr, nullptr,
                                                                      nullptr},
                                                        const bool gw = true) {
  uint64_t *s_sel = sm.sel, *s_ord = sm.ord;
  int32_t *s_gs = sm.gs;
  uint32_t *s_db = sm.db;
  const int n = a.n, k = a.k, E = a.E, m = a.m;
  const int dwords = (m + 31) / 32;
  const int e0 = lane * NS;
  if (lane < dwords) s_db[lane] = 0;
  if (lds.eb && lane < (n + 31) / 32) lds.eb[lane] = 0;

  float lv[NS];
  uint32_t nanbits = 0;   // bit s: expert e0 + s has a NaN logit
  {
    float l[NS];
    if (a.logits_in) {
#pragma unroll
      for (int s = 0; s < NS; ++s) l[s] = a.logits_in[(size_t)t * n + min(e0 + s, n - 1)];
    } else {
      // partial sums of the router chunks, added in chunk order; loads of a
      // batch are issued together (chunks past kc re-read the last one)
      constexpr int CB = NS >= 4 ? 64 / NS : 16;
      const float *p = a.part + (size_t)t * a.ldp + e0;
      const size_t cs = (size_t)a.T * a.ldp;
      for (int c0 = 0; c0 < a.kc; c0 += CB) {
        float pc[CB][NS];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) load_run<NS>(p + (size_t)min(c0 + cb, a.kc - 1) * cs, pc[cb]);
        // selects, not branches: a branch here would serialize the loads
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          const int c = c0 + cb;
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            const float sum = l[s] + pc[cb][s];
            l[s] = c == 0 ? pc[cb][s] : (c < a.kc ? sum : l[s]);
          }
        }
      }
    }
    if (a.bias) {
#pragma unroll
      for (int s = 0; s < NS; ++s) l[s] = l[s] + a.bias[min(e0 + s, n - 1)];
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      lv[s] = (e0 + s < n && l[s] == l[s]) ? l[s] : -INFINITY;   // NaN ranks last
      nanbits |= (uint32_t)(l[s] != l[s]) << s;
    }
  }

  // departments of the lane's experts: one division, then stepped along the
  // run (a division by the runtime E is a long instruction sequence)
  int dep[NS];
  {
    int d = e0 / E, r = e0 - d * E;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      dep[s] = d;
      const bool wrap = ++r == E;
      r = wrap ? 0 : r;
      d = wrap ? d + 1 : d;
    }
  }

  // group-limited top-k: keep the kdept departments with the largest maximum
  // logit (ties to the lower department id)
  uint64_t keep = ~0ull;
  if (a.kdept > 0) {
    if (lane < m) s_gs[lane] = ord_key(-INFINITY);
    wave_lds_sync();
    if (E >= NS) {
      // the lane's run of experts spans at most two departments, dep[0] and
      // dep[0] + 1: both maxima in straight-line code, one atomic each
      int b0 = ord_key(-INFINITY), b1 = b0;
      bool two = false;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int kv = ord_key(lv[s]);   // -inf past the last expert
        const bool first = dep[s] == dep[0];
        b0 = first ? max(b0, kv) : b0;
        b1 = first ? b1 : max(b1, kv);
        two |= !first && e0 + s < n;
      }
      if (e0 < n) atomicMax(&s_gs[dep[0]], b0);
      if (two) atomicMax(&s_gs[dep[0] + 1], b1);
    } else {
      // one atomic per department of the run, with the run's maximum in it
      // (predicated, not an early exit, so that the loop unrolls and dep
      // stays in registers)
      int cur = dep[0], best = ord_key(-INFINITY);
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bool in = e0 + s < n;
        if (in && dep[s] != cur) {
          atomicMax(&s_gs[cur], best);
          cur = dep[s];
          best = ord_key(-INFINITY);
        }
        best = in ? max(best, ord_key(lv[s])) : best;
      }
      if (e0 < n) atomicMax(&s_gs[cur], best);
    }
    wave_lds_sync();
    // department j is kept if fewer than kdept departments rank before it
    // by (score desc, id asc); lane j counts them with one pass over the m
    // scores (the order keys of -0 and +0 agree, as in the expert keys)
    const uint32_t gu = lane < m ? ord_u32(ord_val(s_gs[lane])) : 0u;
    int before = 0;
    for (int i = 0; i < m; ++i) {
      const uint32_t gi = __builtin_amdgcn_readlane(gu, i);
      before += gi > gu || (gi == gu && i < lane);
    }
    keep = __ballot(lane < m && before < a.kdept);
  }

  // order keys; experts that may not be chosen get 0, below every eligible
  // key (the key of -inf is 0x007fffff)
  // (keep is all ones without a group limit; bitwise operators, not && and
  // ||, so that no branch splits the wave per expert)
  uint32_t key[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const uint32_t ok = (uint32_t)(e0 + s < n) & (uint32_t)(keep >> (dep[s] & 63));
    key[s] = (ok & 1u) ? ord_u32(lv[s]) : 0u;
  }
  // Candidates.  theta, the k-th largest of the per-lane maxima, bounds the
  // k-th largest key from below (k lanes hold a key >= theta), so every
  // winner has a key >= theta; usually only a few keys reach it.  When more
  // than 64 do, the exact k-th largest key tau is found by radix selection
  // and the candidates are exactly the k winners.
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  // Exact k-th largest key tau by radix selection (a bit stays if at least k
  // keys reach the value), then the selection: every key above tau, and the
  // keys equal to tau in ascending expert order (lanes first, then s) up to k.
  auto exact_select = [&]() {
    uint32_t tau = 0;
    for (int b = 31; b >= 0; --b) {
      const uint32_t cand = tau | (1u << b);
      int cnt = 0;
#pragma unroll
      for (int s = 0; s < NS; ++s) cnt += popc64(__ballot(key[s] >= cand));
      if (cnt >= k) tau = cand;
    }
    int cnt_gt = 0, ties = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      cnt_gt += popc64(__ballot(key[s] > tau));
      ties += popc64(__ballot(key[s] == tau) & below);
    }
    const int need = k - cnt_gt;
    uint32_t bits = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bool eq = key[s] == tau;
      if (key[s] > tau || (eq && ties < need)) bits |= 1u << s;
      ties += eq;
    }
    return bits;
  };
  // Set only (no published routing, no group limit or coverage rule): the
  // token's expert and department bitmaps, without rank order or weights.
  if (!gw && a.kdept == 0 && !a.dept_cover) {
    const uint32_t bits = exact_select();
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if ((bits >> s) & 1u) {
        const int e = e0 + s, d = dep[s];
        if (lds.eb) atomicOr(&lds.eb[e >> 5], 1u << (e & 31));
        atomicOr(&s_db[d >> 5], 1u << (d & 31));
      }
    }
    wave_lds_sync();
    return;
  }
  uint32_t lmax = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s) lmax = max(lmax, key[s]);
  uint32_t theta = 0;
  for (int b = 31; b >= 0; --b) {
    const uint32_t cand = theta | (1u << b);
    if (popc64(__ballot(lmax >= cand)) >= k) theta = cand;
  }
  int ncand = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s) ncand += popc64(__ballot(key[s] >= theta));
  uint32_t selbits = 0;
  if (ncand <= 64) {
#pragma unroll
    for (int s = 0; s < NS; ++s) selbits |= (uint32_t)(key[s] >= theta) << s;
  } else {
    selbits = exact_select();
    ncand = k;
  }
  // candidates to LDS in expert order, then each ranks itself by (key desc,
  // expert asc); the k best land in rank order
  int pos = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s) pos += popc64(__ballot((selbits >> s) & 1) & below);
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if ((selbits >> s) & 1) {
      s_sel[pos] = ((uint64_t)key[s] << 32) | (uint32_t)~(uint32_t)(e0 + s);
      ++pos;
    }
  }
  wave_lds_sync();
  if (lane < ncand) {
    // a batch of 8 LDS reads is issued before any is compared (entries past
    // ncand are read but not counted)
    const uint64_t mine = s_sel[lane];
    int rank = 0;
    for (int j0 = 0; j0 < ncand; j0 += 8) {
      uint64_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = s_sel[(j0 + u) & 63];
#pragma unroll
      for (int u = 0; u < 8; ++u) rank += (j0 + u < ncand) & (v[u] > mine);
    }
    if (rank < k) s_ord[rank] = mine;
  }
  wave_lds_sync();
  const bool sel = lane < k;
  uint64_t kk = sel ? s_ord[lane] : 0ull;
  // Strict coverage (Sec. 3.4).  While the k winners span fewer than kdept
  // departments, the lowest-ranked winner whose department holds another
  // winner gives way to the best eligible expert (key != 0: a kept
  // department) of a department not yet covered, and the winners are ranked
  // again.  Each round covers one more department.
  if (a.dept_cover) {
    for (int it = 0; it < a.kdept; ++it) {
      const int dl = sel ? (int)(~(uint32_t)kk) / E : 0;
      uint64_t cov = 0;
      int mult = 0;
      for (int q = 0; q < k; ++q) {
        const int dq = __builtin_amdgcn_readlane(dl, q);
        cov |= 1ull << (dq & 63);
        mult += dq == dl;
      }
      if (popc64(cov) >= a.kdept) break;
      uint64_t best = 0;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int e = e0 + s;
        const uint64_t c = ((uint64_t)key[s] << 32) | (uint32_t)~(uint32_t)e;
        if (key[s] != 0u && !((cov >> (dep[s] & 63)) & 1) && c > best) best = c;
      }
      best = wave_max_u64(best);
      const uint64_t vm = __ballot(sel && mult >= 2);
      if (vm == 0 || best == 0) break;   // not reached when k >= kdept
      if (lane == 63 - __clzll(vm)) kk = best;
      if (sel) s_ord[lane] = kk;
      wave_lds_sync();
      int rank = 0;
      for (int j = 0; j < k; ++j) rank += s_ord[j] > kk;
      wave_lds_sync();
      if (sel) s_ord[rank] = kk;
      wave_lds_sync();
      kk = sel ? s_ord[lane] : 0ull;
      wave_lds_sync();
    }
  }
  const int my_id = sel ? (int)~(uint32_t)kk : 0;
  const uint32_t ob = (uint32_t)(kk >> 32);
  const float my_l = __uint_as_float((ob & 0x80000000u) ? (ob & 0x7fffffffu) : ~ob);

  // routing weights
  float p;
  if (a.score == DEAMOE_SCORE_SOFTMAX) {
    float mx, den;
    if (a.renorm) {
      mx = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_l), 0));
      den = wave_sum(sel ? expf(my_l - mx) : 0.f);
    } else {
      float lm = -INFINITY;
#pragma unroll
      for (int s = 0; s < NS; ++s) lm = fmaxf(lm, lv[s]);
      mx = wave_max(lm);
      float ls = 0.f;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        if (e0 + s < n) ls += expf(lv[s] - mx);
      den = wave_sum(ls);
    }
    p = expf(my_l - mx) / den;
  } else {
    const float sg = 1.0f / (1.0f + expf(-my_l));
    p = a.renorm ? sg / wave_sum(sel ? sg : 0.f) : sg;
  }
  p *= a.route_scale;
  const int d = sel ? my_id / E : 0;
  if (sel) {
    if (gw) {
      a.r.topk_ids[t * k + lane] = my_id;
      a.r.topk_w[t * k + lane] = p;
      if (a.wdense) glob(a.wdense)[(size_t)(a.m + my_id) * kChainT + t] = p;
    }
    if (lds.ids) lds.ids[t * k + lane] = my_id;
    if (lds.eb) atomicOr(&lds.eb[my_id >> 5], 1u << (my_id & 31));
    atomicOr(&s_db[d >> 5], 1u << (d & 31));
  }
  wave_lds_sync();
  // distinct departments, ascending, each with the weights of its selected
  // experts summed in rank order
  int nd = 0;
  for (int w = 0; w < dwords; ++w) nd += __popc(s_db[w]);
  nd = __builtin_amdgcn_readfirstlane(nd);
  float P = 0.f;
  uint32_t eqm = 0;
  for (int q = 0; q < k; ++q) {
    const int dq = __builtin_amdgcn_readlane(d, q);
    const float pq = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), q));
    if (dq == d) { P += pq; eqm |= 1u << q; }
  }
  const bool first = sel && (eqm & ((1u << lane) - 1u)) == 0;
  const bool slice = a.plan == PLAN_SLICE;
  const bool exp_slots = slice && a.d_p > 0;
  const int S = a.max_slots;
  if (first) {
    const int dpos = rank_below(s_db, d);
    if (lds.dep) lds.dep[t * k + dpos] = d;
    if (gw) {
      a.r.tok_depts[t * k + dpos] = d;
      a.r.tok_dept_w[t * k + dpos] = P;
      if (a.wdense) glob(a.wdense)[(size_t)d * kChainT + t] = P;
      if (a.plan) a.slot_w[(size_t)t * S + dpos] = slice ? P : 1.0f;
    }
  }
  if (lane >= nd && lane < k) {
    if (lds.dep) lds.dep[t * k + lane] = -1;
    if (gw) {
      a.r.tok_depts[t * k + lane] = -1;
      a.r.tok_dept_w[t * k + lane] = 0.f;
    }
  }
  if (gw && a.plan && exp_slots && sel) a.slot_w[(size_t)t * S + nd + lane] = p;
  if (lane == 0) {
    if (lds.nd) lds.nd[t] = nd;
    if (gw) a.r.tok_ndept[t] = nd;
    if (gw && a.plan) {
      const int ns = nd + (exp_slots ? k : 0);
      if (a.d_se > 0) a.slot_w[(size_t)t * S + ns] = 1.0f;
      a.nslot[t] = ns + (a.d_se > 0 ? 1 : 0);
    }
  }
  // the logits last: a wave may not reuse the registers of a store's data
  // until the store completes, so stores issued early would stall the
  // selection above
  if (gw && a.r.logits) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      if (e0 + s < n)
        a.r.logits[(size_t)t * n + e0 + s] = ((nanbits >> s) & 1u) ? __builtin_nanf("") : lv[s];
  }
}


// The argument block copied to LDS by the first threads of the workgroup
// (visible after the next barrier): the plan then loads each pointer where it
// uses it instead of holding all of them in scalar registers, which spilled.
template <int BT>
__device__ inline void args_to_lds(const RouteArgs &a, RouteArgs &sa) {
  static_assert(sizeof(RouteArgs) % 4 == 0 && sizeof(RouteArgs) / 4 <= BT, "argument copy");
  const int tid = threadIdx.x;
  if (tid < (int)(sizeof(RouteArgs) / 4))
    __builtin_memcpy(reinterpret_cast<char *>(&sa) + 4 * tid,
                     reinterpret_cast<const char *>(&a) + 4 * tid, 4);
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
// MT: the most tokens the plan serves (token bitmaps of MT / 32 words).
template <int MT>
struct PlanSmemT {
  static constexpr int TW = (MT + 31) / 32;
  static constexpr int MAXT = MT;
  int32_t ids[MT * kMaxK];           // [t][rank] selected expert
  int32_t dep[MT * kMaxK];           // [t][slot] departments, -1 padded
  uint32_t etok[kMaxN * TW];         // [e] token bitmap
  uint32_t dtok[kMaxM * TW];         // [j] token bitmap
  int32_t scan[kMaxM + kMaxN];       // [depts, experts] packed prefix
  int32_t nd[MT];
  int32_t tmp[64];
};
using PlanSmem = PlanSmemT<kMaxT>;

// Every thread of the workgroup (BT threads) calls it.  LDS_IN: the
// per-token results are already in sm.ids, sm.dep and sm.nd.  PS: a
// PlanSmemT; with fewer than 32 tokens per bitmap word the unit item
// prefixes must be closed forms (one token group per unit).
template <int BT, bool LDS_IN = false, class PS = PlanSmem>
__device__ __attribute__((always_inline)) void plan_body(const RouteArgs &a, PS &sm) {
  constexpr int EPT = kMaxN / BT;   // experts per thread in the per-expert loops
  constexpr int DPT = (kMaxM + BT - 1) / BT;   // departments per thread
  constexpr int kTW = PS::TW;
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
  int my_dc[DPT] = {}, my_ec[EPT] = {};
#pragma unroll
  for (int q = 0; q < DPT; ++q) {
    const int j = tid + q * BT;
    if (j < m) {
      int c = 0;
      for (int w = 0; w < tw; ++w) c += __popc(s_dtok[j * kTW + w]);
      my_dc[q] = c;
      dept_count[j] = c;
      s_scan[j] = c | ((c > 0) << 16);
    }
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
  for (int j = tid; j < m; j += BT) dept_offset[j] = doff(j);
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
  // token groups of a unit: wave_tokens per group in the gate/up stages (pair
  // A), wave_tokens_b in the separate down stages (pair B; the fused down
  // kernel takes one group, and reads the bitmaps the item scans would reuse)
  const int wt = a.wave_tokens, wtb = a.chain ? wt : a.wave_tokens_b;
  const bool multi = T > min(wt, wtb);
  auto groups = [&](int cnt) { return T > wt ? (cnt + wt - 1) / wt : 1; };
  auto groups_b = [&](int cnt) { return T > wtb ? (cnt + wtb - 1) / wtb : 1; };
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
  static_assert(PS::MAXT >= kMaxT || PS::MAXT <= kTile, "a plan for fewer tokens has one group per unit");
  if (PS::MAXT > kTile && multi) {
    lds_barrier();   // the expert bitmaps are no longer read
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
      const int j = tid + q * BT;
      if (j < m) {
        s_ia[j] = my_dc[q] > 0 ? ia_d * groups(my_dc[q]) : 0;
        s_ib[j] = my_dc[q] > 0 ? ib_d * groups_b(my_dc[q]) : 0;
      }
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      const int e = tid + q * BT;
      if (e < n) {
        const bool act = has_priv && my_ec[q] > 0;
        s_ia[m + e] = act ? ia_e * groups(my_ec[q]) : 0;
        s_ib[m + e] = act ? ib_e * groups_b(my_ec[q]) : 0;
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
  const bool scanned = PS::MAXT > kTile && multi;
  auto dbeg_a = [&](int j, int uj) { return scanned ? s_ia[j] : uj * ia_d; };
  auto dbeg_b = [&](int j, int uj) { return scanned ? s_ib[j] : uj * ib_d; };
  auto ebeg_a = [&](int e, int ui) { return scanned ? s_ia[m + e] : ud * ia_d + ui * ia_e; };
  auto ebeg_b = [&](int e, int ui) { return scanned ? s_ib[m + e] : ud * ib_d + ui * ib_e; };
  const int dept_a = scanned ? s_ia[m] : ud * ia_d;   // items of all departments
  const int dept_b = scanned ? s_ib[m] : ud * ib_d;
  const int kstep = a.w_bytes == 4 ? 64 : 128;   // K step of the weight type
  if (slice) {
    const int gd = tiles_per_item(a.d_s, dr, dk), gp = a.d_p ? tiles_per_item(a.d_p, dr, dk) : 1;
    const int gse = a.d_se ? tiles_per_item(a.d_se, dr, dk) : 1;
    const int bse = items_of(a.h, gse, dr);
    // fused down stage (T <= 32): the units' K steps are concatenated in
    // table order (departments, experts, the shared expert)
    const int sd = a.d_s / kstep, sp = a.d_p / kstep;
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
      const int j = tid + q * BT, dc = my_dc[q];
      if (j >= m || dc == 0) continue;
      const int u = s_scan[j] >> 16, off = doff(j);
      const int32_t *idx = a.r.dept_tokens + off;
      char *ao = static_cast<char *>(a.abuf_dept) + (size_t)off * a.d_s * ab;
      put_unit(glob(a.units[0]) + u, wptr(W.dept_gate, j, a.d_s, a.h), wptr(W.dept_up, j, a.d_s, a.h),
               sptr(W.scale[0], j, a.d_s, a.h), sptr(W.scale[1], j, a.d_s, a.h), x, x, idx, ao,
               nullptr, a.d_s, a.h, a.h, a.d_s, dc, dbeg_a(j, u), EPI_SWIGLU, a.act_f32);
      if (a.chain)
        put_chain(glob(a.cunits) + u, wptr(W.dept_down, j, a.h, a.d_s),
                  sptr(W.scale[2], j, a.h, a.d_s), ao, a.wdense + (size_t)j * kChainT, a.d_s,
                  s_dtok[j * kTW], u * sd);
      else
        put_unit(glob(a.units[1]) + u, wptr(W.dept_down, j, a.h, a.d_s), nullptr,
                 sptr(W.scale[2], j, a.h, a.d_s), nullptr, ao, ao, nullptr,
                 a.partial + (size_t)off * a.h, nullptr, a.h, a.d_s, a.d_s, a.h, dc,
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
        items_b += bse * groups_b(T);
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
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
      const int j = tid + q * BT, dc = my_dc[q];
      if (j >= m || dc == 0) continue;
      const int u = s_scan[j] >> 16, off = doff(j);
      const int32_t *idx = a.r.dept_tokens + off;
      char *go = static_cast<char *>(a.gbuf) + (size_t)off * d * ab;
      char *uo = static_cast<char *>(a.ubuf) + (size_t)off * d * ab;
      char *zs = static_cast<char *>(a.zsbuf) + (size_t)off * d * ab;
      put_unit(glob(a.units[0]) + u, wptr(W.dept_gate, j, d, a.h), wptr(W.dept_up, j, d, a.h),
               sptr(W.scale[0], j, d, a.h), sptr(W.scale[1], j, d, a.h), x, x, idx, go, uo, d,
               a.h, a.h, d, dc, dbeg_a(j, u), EPI_SIGMA2, a.act_f32);
      if (a.chain)   // Z already carries the routing weights: unit weight 1
        put_chain(glob(a.cunits) + u, wptr(W.dept_down, j, a.h, d), sptr(W.scale[2], j, a.h, d), zs,
                  a.wdense + (size_t)(m + n) * kChainT, d, s_dtok[j * kTW], u * (d / kstep));
      else
        put_unit(glob(a.units[3]) + u, wptr(W.dept_down, j, a.h, d), nullptr,
                 sptr(W.scale[2], j, a.h, d), nullptr, zs, zs, nullptr,
                 a.partial + (size_t)off * a.h, nullptr, a.h, d, d, a.h, dc, dbeg_b(j, u),
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
        items3 += bse * groups_b(T);
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

}  // namespace deamoe
