// Router (Eq. 2), department bookkeeping (Sec. 3.2) and the device-side plan
// of the expert stages.
//
// router_kernel: the logits W_r x as a grouped skinny product, split over KC
//   chunks of the hidden dimension so that the n x h router matrix is read by
//   many workgroups; each chunk's partial logits go to part[c][t][e].
// route_plan_kernel: one workgroup of 1024 threads.
//   phase 1, one wave per token: logits = sum of the KC partials in chunk
//     order (+ bias, one fp32 add), optional group-limited department choice,
//     top-k by (logit desc, id asc) with wavefront arg-max reductions, the
//     routing weights, and the token's distinct departments with P_{t,j};
//   phase 2: per-department and per-expert token lists in ascending token
//     order (counts by scanning, offsets by a block-wide prefix sum, no
//     atomics on any order-sensitive value);
//   phase 3: the unit tables of every expert stage (pointers, row-tile
//     prefix), the combine slots of every token, and the counts.
#include "gemm_tile.h"
#include "launch.h"

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
  U.out0 = a.part + (size_t)c * a.T * a.n;
  U.R = a.n;
  U.K = a.kchunk;
  U.ldw = a.h;
  U.ldin = a.h;
  U.ldout = a.n;
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

// ------------------------------------------------------------ route and plan

__device__ inline bool ranks_before(float va, int a, float vb, int b) {
  return va > vb || (va == vb && a < b);
}

// Order-preserving map of a float onto an unsigned int (larger float, larger key).
__device__ inline uint32_t ord_u32(float f) {
  const uint32_t u = __float_as_uint(f);
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

// Arg-max by (value desc, index asc) over the lanes' candidates; a lane with
// no candidate passes valid = false.  Returns the winning index (every lane).
__device__ inline int wave_argmax_idx(float v, int i, bool valid, float &best_v) {
  const uint64_t key = valid ? (((uint64_t)ord_u32(v) << 32) | (uint32_t)~(uint32_t)i) : 0ull;
  const uint64_t b = wave_max_u64(key);
  const uint32_t ob = (uint32_t)(b >> 32);
  best_v = __uint_as_float((ob & 0x80000000u) ? (ob & 0x7fffffffu) : ~ob);
  return (int)~(uint32_t)b;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// Order-preserving float <-> int map for integer max.
__device__ inline int ord_key(float f) {
  const int i = __float_as_int(f);
  return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ inline float ord_val(int i) { return __int_as_float(i >= 0 ? i : i ^ 0x7fffffff); }

// Exclusive prefix sum of s[0..N) in place, N <= 4 * blockDim; returns the
// total.  Every thread of the block must call it.
__device__ int block_exscan(int32_t *s, int N, int32_t *s_tmp) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int nwaves = nt / 64;
  const int per = (N + nt - 1) / nt;
  const int b = min(tid * per, N), e = min(b + per, N);
  int local = 0;
  for (int i = b; i < e; ++i) local += s[i];
  int v = local;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(v, off);
    if (lane >= off) v += o;
  }
  if (lane == 63) s_tmp[wave] = v;
  __syncthreads();
  if (wave == 0) {
    int w = lane < nwaves ? s_tmp[lane] : 0;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_up(w, off);
      if (lane >= off) w += o;
    }
    if (lane < nwaves) s_tmp[lane] = w;
  }
  __syncthreads();
  int run = (wave > 0 ? s_tmp[wave - 1] : 0) + v - local;
  for (int i = b; i < e; ++i) {
    const int x = s[i];
    s[i] = run;
    run += x;
  }
  const int total = s_tmp[nwaves - 1];
  __syncthreads();
  return total;
}

__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

constexpr int kMaxKC = 16;   // router chunks (host caps the split)

// Fill one unit of a stage table field by field (no temporary struct).
__device__ inline void put_unit(GemmUnit *U, const void *w0, const void *w1, const float *s0,
                                const float *s1, const void *in0, const void *in1,
                                const int32_t *idx, void *out0, void *out1, int R, int K, int ldin,
                                int ldout, int ntok, int tile_begin, int epi, int out_f32,
                                int tpg = 1) {
  U->w0 = w0; U->w1 = w1; U->s0 = s0; U->s1 = s1; U->in0 = in0; U->in1 = in1; U->idx = idx;
  U->out0 = out0; U->out1 = out1; U->R = R; U->K = K; U->ldw = K; U->ldin = ldin;
  U->ldout = ldout; U->ntok = ntok; U->tile_begin = tile_begin; U->epi = epi;
  U->out_f32 = out_f32; U->tpg = tpg;
}

// Row tiles per work item of a stage whose K is not split across waves: short
// contractions take several tiles so that a work item streams enough bytes.
__device__ inline int tiles_per_item(int K) { return max(1, min(8, 2048 / K)); }
__device__ inline int items_of(int R, int tpg) { return ((R + kTile - 1) / kTile + tpg - 1) / tpg; }

__device__ inline bool bit_at(const uint32_t *row, int i) { return (row[i >> 5] >> (i & 31)) & 1; }

// Number of set bits below bit i of a bitmap row.
__device__ inline int rank_below(const uint32_t *row, int i) {
  int r = 0;
  for (int w = 0; w < (i >> 5); ++w) r += __popc(row[w]);
  return r + __popc(row[i >> 5] & ((1u << (i & 31)) - 1u));
}

constexpr int kTW = kMaxT / 32;   // words of a token bitmap
constexpr int kDW = kMaxM / 32;   // words of a department bitmap

// NS: logits held per lane (n <= 64 * NS); BT: threads of the workgroup.
//
// Membership is kept as bitmaps in LDS: for every expert and department the
// set of its tokens (kTW words), for every token the set of its departments.
// A token's position in a CSR list is then the offset of the list plus the
// number of member tokens below it, so every (token, rank) pair is placed
// independently and the lists come out in ascending token order.
template <int NS, int BT>
__global__ __launch_bounds__(BT) void route_plan_kernel(RouteArgs a) {
  constexpr int EPT = kMaxN / BT;   // experts per thread in the per-expert loops
  __shared__ int32_t s_ids[kMaxTK];            // [t][rank] selected expert
  __shared__ int32_t s_dep[kMaxTK];            // [t][slot] departments, ascending
  __shared__ uint32_t s_etok[kMaxN * kTW];     // [e] token bitmap
  __shared__ uint32_t s_dtok[kMaxM * kTW];     // [j] token bitmap
  __shared__ uint32_t s_dbits[kMaxT * kDW];    // [t] department bitmap
  __shared__ int32_t s_dcnt[kMaxM + 1];
  __shared__ int32_t s_ecnt[kMaxN + 1];
  __shared__ int32_t s_nd[kMaxT];
  __shared__ int32_t s_gs[BT / 64][kMaxMGrouped];
  __shared__ int32_t s_tmp[64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T, n = a.n, m = a.m, k = a.k, E = a.E;
  const int tw = (T + 31) / 32, dwords = (m + 31) / 32;
  const bool slice = a.plan == PLAN_SLICE;
  const bool exp_slots = slice && a.d_p > 0;
  const int S = a.max_slots;
  for (int i = tid; i < n * kTW; i += BT) s_etok[i] = 0;
  for (int i = tid; i < m * kTW; i += BT) s_dtok[i] = 0;
  for (int i = tid; i < T * dwords; i += BT) s_dbits[i] = 0;
  __syncthreads();

  // ------------------------------------------------ phase 1: one wave per token
  for (int t = wave; t < T; t += BT / 64) {
    float lv[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int e = lane + 64 * s;
      const int ec = e < n ? e : n - 1;
      float l;
      if (a.logits_in) {
        l = a.logits_in[(size_t)t * n + ec];
      } else {  // partial sums of the router chunks, added in chunk order; all
                // loads are issued first (chunks past kc re-read the last one)
        float pc[kMaxKC];
#pragma unroll
        for (int c = 0; c < kMaxKC; ++c)
          pc[c] = a.part[((size_t)min(c, a.kc - 1) * T + t) * n + ec];
        l = pc[0];
#pragma unroll
        for (int c = 1; c < kMaxKC; ++c) l = c < a.kc ? l + pc[c] : l;
      }
      if (a.bias) l = l + a.bias[ec];
      if (e < n) a.r.logits[(size_t)t * n + e] = l;
      lv[s] = (e < n && l == l) ? l : -INFINITY;   // NaN ranks last
    }
    // group-limited top-k: keep the kdept departments with the largest
    // maximum logit (ties to the lower department id)
    uint64_t keep = ~0ull;
    if (a.kdept > 0) {
      if (lane < m) s_gs[wave][lane] = ord_key(-INFINITY);
      wave_lds_sync();
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int e = lane + 64 * s;
        if (e < n) atomicMax(&s_gs[wave][e / E], ord_key(lv[s]));
      }
      wave_lds_sync();
      const float gsv = lane < m ? ord_val(s_gs[wave][lane]) : -INFINITY;
      keep = 0;
      for (int r = 0; r < a.kdept; ++r) {
        float bv;
        const int bj = wave_argmax_idx(gsv, lane, lane < m && !((keep >> lane) & 1), bv);
        keep |= 1ull << (bj & 63);
      }
    }
    // top-k: k rounds of arg-max over the lane-held logits
    uint32_t taken = 0;
    int my_id = 0;
    float my_l = -INFINITY;
    for (int r = 0; r < k; ++r) {
      float bv = -INFINITY;
      int be = 0x7fffffff;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int e = lane + 64 * s;
        const bool ok = e < n && !((taken >> s) & 1) &&
                        (a.kdept == 0 || ((keep >> ((e / E) & 63)) & 1));
        if (ok && ranks_before(lv[s], e, bv, be)) { bv = lv[s]; be = e; }
      }
      be = wave_argmax_idx(bv, be, be != 0x7fffffff, bv);
      if (be < 0 || be >= n) be = 0;   // unreachable: at least k experts are always eligible
      if ((be & 63) == lane) taken |= 1u << (be >> 6);
      if (lane == r) { my_id = be; my_l = bv; }
    }
    // routing weights
    const bool sel = lane < k;
    float p;
    if (a.score == DEAMOE_SCORE_SOFTMAX) {
      float mx, den;
      if (a.renorm) {
        mx = __shfl(my_l, 0);
        den = wave_sum(sel ? expf(my_l - mx) : 0.f);
      } else {
        float lm = -INFINITY;
#pragma unroll
        for (int s = 0; s < NS; ++s) lm = fmaxf(lm, lv[s]);
        mx = wave_max(lm);
        float ls = 0.f;
#pragma unroll
        for (int s = 0; s < NS; ++s)
          if (lane + 64 * s < n) ls += expf(lv[s] - mx);
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
      a.r.topk_ids[t * k + lane] = my_id;
      a.r.topk_w[t * k + lane] = p;
      s_ids[t * k + lane] = my_id;
      atomicOr(&s_etok[my_id * kTW + (t >> 5)], 1u << (t & 31));
      atomicOr(&s_dtok[d * kTW + (t >> 5)], 1u << (t & 31));
      atomicOr(&s_dbits[t * dwords + (d >> 5)], 1u << (d & 31));
    }
    wave_lds_sync();
    // distinct departments, ascending, each with the weights of its selected
    // experts summed in rank order
    const uint32_t *drow = s_dbits + t * dwords;
    int nd = 0;
    for (int w = 0; w < dwords; ++w) nd += __popc(drow[w]);
    nd = __builtin_amdgcn_readfirstlane(nd);
    float P = 0.f;
    uint32_t eq = 0;
    for (int q = 0; q < k; ++q) {
      const int dq = __builtin_amdgcn_readlane(d, q);
      const float pq = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), q));
      if (dq == d) { P += pq; eq |= 1u << q; }
    }
    const bool first = sel && (eq & ((1u << lane) - 1u)) == 0;
    if (first) {
      const int pos = rank_below(drow, d);
      a.r.tok_depts[t * k + pos] = d;
      a.r.tok_dept_w[t * k + pos] = P;
      s_dep[t * k + pos] = d;
      if (a.plan) a.slot_w[(size_t)t * S + pos] = slice ? P : 1.0f;
    }
    if (lane >= nd && lane < k) {
      a.r.tok_depts[t * k + lane] = -1;
      a.r.tok_dept_w[t * k + lane] = 0.f;
    }
    if (a.plan && exp_slots && sel) a.slot_w[(size_t)t * S + nd + lane] = p;
    if (lane == 0) {
      a.r.tok_ndept[t] = nd;
      s_nd[t] = nd;
      if (a.plan) {
        const int ns = nd + (exp_slots ? k : 0);
        if (a.d_se > 0) a.slot_w[(size_t)t * S + ns] = 1.0f;
        a.nslot[t] = ns + (a.d_se > 0 ? 1 : 0);
      }
    }
  }
  __syncthreads();

  // ------------------------------------------------ phase 2: counts and lists
  int my_dc = 0, my_ec[EPT] = {};
  if (tid < m) {
    for (int w = 0; w < tw; ++w) my_dc += __popc(s_dtok[tid * kTW + w]);
    s_dcnt[tid] = my_dc;
    a.r.dept_count[tid] = my_dc;
  }
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = tid + q * BT;
    if (e < n) {
      int c = 0;
      for (int w = 0; w < tw; ++w) c += __popc(s_etok[e * kTW + w]);
      my_ec[q] = c;
      s_ecnt[e] = c;
      a.r.exp_count[e] = c;
    }
  }
  __syncthreads();
  const int ndp = block_exscan(s_dcnt, m, s_tmp);
  const int nep = block_exscan(s_ecnt, n, s_tmp);
  const bool has_priv = a.plan == PLAN_FACTORED || a.d_p > 0;
  const bool has_se = a.d_se > 0;
  const int nep_priv = has_priv ? nep : 0;
  if (tid < m) a.r.dept_offset[tid] = s_dcnt[tid];
  for (int e = tid; e < n; e += BT) a.r.exp_offset[e] = s_ecnt[e];
  if (tid == 0) {
    a.r.dept_offset[m] = ndp;
    a.r.exp_offset[n] = nep;
  }
  // every (token, rank) pair places itself: the expert of that rank and, for
  // ranks below the token's department count, the department of that slot
  for (int idx = tid; idx < T * k; idx += BT) {
    const int t = idx / k, q = idx - t * k;
    const int e = s_ids[idx];
    const int pe = s_ecnt[e] + rank_below(s_etok + e * kTW, t);
    a.r.exp_tokens[pe] = t;
    if (a.plan) {
      a.tok_exp_pair[idx] = pe;
      if (exp_slots) a.slot_pair[(size_t)t * S + s_nd[t] + q] = ndp + pe;
      if (a.plan == PLAN_FACTORED) {
        const int j = e / E;
        a.exp_src[pe] = s_dcnt[j] + rank_below(s_dtok + j * kTW, t);
      }
    }
    if (q < s_nd[t]) {
      const int j = s_dep[idx];
      const int pd = s_dcnt[j] + rank_below(s_dtok + j * kTW, t);
      a.r.dept_tokens[pd] = t;
      if (a.plan) a.slot_pair[(size_t)t * S + q] = pd;
    }
  }
  if (a.plan && has_se)
    for (int t = tid; t < T; t += BT)
      a.slot_pair[(size_t)t * S + s_nd[t] + (exp_slots ? k : 0)] = ndp + (slice ? nep_priv : 0) + t;
  if (!a.plan) return;
  const int my_doff = tid < m ? s_dcnt[tid] : 0;
  int my_eoff[EPT] = {};
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = tid + q * BT;
    if (e < n) my_eoff[q] = s_ecnt[e];
  }
  __syncthreads();

  // ------------------------------------------------ phase 3: stage unit tables
  // unit index of every active department / expert (prefix over active flags)
  if (tid < m) s_dcnt[tid] = my_dc > 0;
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = tid + q * BT;
    if (e < n) s_ecnt[e] = has_priv && my_ec[q] > 0;
  }
  __syncthreads();
  const int ud = block_exscan(s_dcnt, m, s_tmp);
  const int ue = block_exscan(s_ecnt, n, s_tmp);
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
  if (slice) {
    const int ta_d = (a.d_s + kTile - 1) / kTile, ta_p = (a.d_p + kTile - 1) / kTile;
    const int gd = tiles_per_item(a.d_s), gp = a.d_p ? tiles_per_item(a.d_p) : 1;
    const int gse = a.d_se ? tiles_per_item(a.d_se) : 1;
    const int bd = items_of(a.h, gd), bp = items_of(a.h, gp), bse = items_of(a.h, gse);
    if (tid < m && my_dc > 0) {
      const int j = tid, u = s_dcnt[j];
      const int32_t *idx = a.r.dept_tokens + my_doff;
      char *ao = static_cast<char *>(a.abuf_dept) + (size_t)my_doff * a.d_s * ab;
      put_unit(&a.units[0][u], wptr(W.dept_gate, j, a.d_s, a.h), wptr(W.dept_up, j, a.d_s, a.h),
               sptr(W.scale[0], j, a.d_s, a.h), sptr(W.scale[1], j, a.d_s, a.h), x, x, idx, ao,
               nullptr, a.d_s, a.h, a.h, a.d_s, my_dc, u * ta_d, EPI_SWIGLU, a.act_f32);
      put_unit(&a.units[1][u], wptr(W.dept_down, j, a.h, a.d_s), nullptr,
               sptr(W.scale[2], j, a.h, a.d_s), nullptr, ao, ao, nullptr,
               a.partial + (size_t)my_doff * a.h, nullptr, a.h, a.d_s, a.d_s, a.h, my_dc, u * bd,
               EPI_STORE, 1, gd);
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      const int e = tid + q * BT;
      if (!has_priv || e >= n || my_ec[q] == 0) continue;
      const int u = ud + s_ecnt[e];
      const int32_t *idx = a.r.exp_tokens + my_eoff[q];
      char *ao = static_cast<char *>(a.abuf_exp) + (size_t)my_eoff[q] * a.d_p * ab;
      put_unit(&a.units[0][u], wptr(W.priv_gate, e, a.d_p, a.h), wptr(W.priv_up, e, a.d_p, a.h),
               sptr(W.scale[3], e, a.d_p, a.h), sptr(W.scale[4], e, a.d_p, a.h), x, x, idx, ao,
               nullptr, a.d_p, a.h, a.h, a.d_p, my_ec[q], ud * ta_d + s_ecnt[e] * ta_p,
               EPI_SWIGLU, a.act_f32);
      put_unit(&a.units[1][u], wptr(W.priv_down, e, a.h, a.d_p), nullptr,
               sptr(W.scale[5], e, a.h, a.d_p), nullptr, ao, ao, nullptr,
               a.partial + (size_t)(ndp + my_eoff[q]) * a.h, nullptr, a.h, a.d_p, a.d_p, a.h,
               my_ec[q], ud * bd + s_ecnt[e] * bp, EPI_STORE, 1, gp);
    }
    if (tid == 0) {
      int units = ud + ue, tiles_a = ud * ta_d + ue * ta_p;
      if (has_se) {
        const int ta_se = (a.d_se + kTile - 1) / kTile;
        put_unit(&a.units[0][units], W.se_gate, W.se_up, sptr(W.scale[6], 0, a.d_se, a.h),
                 sptr(W.scale[7], 0, a.d_se, a.h), x, x, nullptr, a.abuf_se, nullptr, a.d_se, a.h,
                 a.h, a.d_se, T, tiles_a, EPI_SWIGLU, a.act_f32);
        put_unit(&a.units[1][units], W.se_down, nullptr, sptr(W.scale[8], 0, a.h, a.d_se), nullptr,
                 a.abuf_se, a.abuf_se, nullptr, a.partial + (size_t)(ndp + nep_priv) * a.h,
                 nullptr, a.h, a.d_se, a.d_se, a.h, T, ud * bd + ue * bp, EPI_STORE, 1, gse);
        tiles_a += ta_se;
        ++units;
      }
      a.counts->stage[0][0] = units;
      a.counts->stage[0][1] = tiles_a;
      a.counts->stage[1][0] = units;
      a.counts->stage[1][1] = ud * bd + ue * bp + (has_se ? bse : 0);
    }
  } else {  // PLAN_FACTORED
    const int d = a.d_s, td = (d + kTile - 1) / kTile;
    const int gd = tiles_per_item(d), gse = a.d_se ? tiles_per_item(a.d_se) : 1;
    const int bd = items_of(a.h, gd), bse = items_of(a.h, gse);
    if (tid < m && my_dc > 0) {
      const int j = tid, u = s_dcnt[j];
      const int32_t *idx = a.r.dept_tokens + my_doff;
      char *go = static_cast<char *>(a.gbuf) + (size_t)my_doff * d * ab;
      char *uo = static_cast<char *>(a.ubuf) + (size_t)my_doff * d * ab;
      char *zs = static_cast<char *>(a.zsbuf) + (size_t)my_doff * d * ab;
      put_unit(&a.units[0][u], wptr(W.dept_gate, j, d, a.h), wptr(W.dept_up, j, d, a.h),
               sptr(W.scale[0], j, d, a.h), sptr(W.scale[1], j, d, a.h), x, x, idx, go, uo, d,
               a.h, a.h, d, my_dc, u * td, EPI_SIGMA2, a.act_f32);
      put_unit(&a.units[3][u], wptr(W.dept_down, j, a.h, d), nullptr, sptr(W.scale[2], j, a.h, d),
               nullptr, zs, zs, nullptr, a.partial + (size_t)my_doff * a.h, nullptr, a.h, d, d,
               a.h, my_dc, u * bd, EPI_STORE, 1, gd);
    }
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      const int e = tid + q * BT;
      if (e >= n || my_ec[q] == 0) continue;
      const int u = s_ecnt[e];
      char *yo = static_cast<char *>(a.ybuf) + (size_t)my_eoff[q] * d * ab;
      put_unit(&a.units[1][u], wptr(W.priv_gate, e, d, d), wptr(W.priv_up, e, d, d),
               sptr(W.scale[3], e, d, d), sptr(W.scale[4], e, d, d), a.gbuf, a.ubuf,
               a.exp_src + my_eoff[q], yo, nullptr, d, d, d, d, my_ec[q], u * td, EPI_SWIGLU,
               a.act_f32);
      put_unit(&a.units[2][u], wptr(W.priv_down, e, d, d), nullptr, sptr(W.scale[5], e, d, d),
               nullptr, yo, yo, nullptr, a.zbuf + (size_t)my_eoff[q] * d, nullptr, d, d, d, d,
               my_ec[q], u * td, EPI_SIGMA, 1);
    }
    if (tid == 0) {
      int units0 = ud, tiles0 = ud * td, units3 = ud;
      if (has_se) {
        const int ta_se = (a.d_se + kTile - 1) / kTile;
        put_unit(&a.units[0][units0], W.se_gate, W.se_up, sptr(W.scale[6], 0, a.d_se, a.h),
                 sptr(W.scale[7], 0, a.d_se, a.h), x, x, nullptr, a.abuf_se, nullptr, a.d_se, a.h,
                 a.h, a.d_se, T, tiles0, EPI_SWIGLU, a.act_f32);
        put_unit(&a.units[3][units3], W.se_down, nullptr, sptr(W.scale[8], 0, a.h, a.d_se),
                 nullptr, a.abuf_se, a.abuf_se, nullptr, a.partial + (size_t)ndp * a.h, nullptr,
                 a.h, a.d_se, a.d_se, a.h, T, ud * bd, EPI_STORE, 1, gse);
        ++units0;
        tiles0 += ta_se;
        ++units3;
      }
      a.counts->stage[0][0] = units0;
      a.counts->stage[0][1] = tiles0;
      a.counts->stage[1][0] = ue;
      a.counts->stage[1][1] = ue * td;
      a.counts->stage[2][0] = ue;
      a.counts->stage[2][1] = ue * td;
      a.counts->stage[3][0] = units3;
      a.counts->stage[3][1] = ud * bd + (has_se ? bse : 0);
    }
  }
  if (tid == 0) {
    a.counts->n_dept_pairs = ndp;
    a.counts->n_exp_pairs = nep_priv;
    a.counts->n_pairs = ndp + (slice ? nep_priv : 0) + (has_se ? T : 0);
  }
}

hipError_t launch_route_plan(const RouteArgs &a, hipStream_t s) {
  // more logits per lane need more registers: half the threads from 513 experts on
  const dim3 g(1);
  if (a.n <= 64) hipLaunchKernelGGL((route_plan_kernel<1, 1024>), g, dim3(1024), 0, s, a);
  else if (a.n <= 128) hipLaunchKernelGGL((route_plan_kernel<2, 1024>), g, dim3(1024), 0, s, a);
  else if (a.n <= 256) hipLaunchKernelGGL((route_plan_kernel<4, 1024>), g, dim3(1024), 0, s, a);
  else if (a.n <= 512) hipLaunchKernelGGL((route_plan_kernel<8, 1024>), g, dim3(1024), 0, s, a);
  else if (a.n <= 1024) hipLaunchKernelGGL((route_plan_kernel<16, 512>), g, dim3(512), 0, s, a);
  else hipLaunchKernelGGL((route_plan_kernel<32, 512>), g, dim3(512), 0, s, a);
  return hipGetLastError();
}

}  // namespace deamoe
