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

// Wave-wide arg-max by (value desc, index asc); every lane gets the winner.
__device__ inline void wave_argmax(float &v, int &i) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(i, off);
    if (ranks_before(ov, oi, v, i)) { v = ov; i = oi; }
  }
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

constexpr int kSlots = kMaxN / 64;   // logits per lane (n <= 2048)

__global__ __launch_bounds__(kRouteThreads) void route_plan_kernel(RouteArgs a) {
  __shared__ int32_t s_ids[kMaxTK];
  __shared__ float s_w[kMaxTK];
  __shared__ int32_t s_dep[kMaxTK];
  __shared__ float s_dw[kMaxTK];
  __shared__ int32_t s_pair[kMaxTK];          // dept pair index of (t, dept slot)
  __shared__ uint32_t s_ebits[kMaxT * (kMaxN / 32)];
  __shared__ int32_t s_dcnt[kMaxM + 1];
  __shared__ int32_t s_ecnt[kMaxN + 1];
  __shared__ int32_t s_nd[kMaxT];
  __shared__ int32_t s_gs[kRouteThreads / 64][kMaxMGrouped];
  __shared__ int32_t s_tmp[64];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int T = a.T, n = a.n, m = a.m, k = a.k, E = a.E;
  const int nwords = (n + 31) / 32;
  for (int i = tid; i < T * nwords; i += blockDim.x) s_ebits[i] = 0;
  __syncthreads();

  // ---------------------------------------------------------------- phase 1
  for (int t = wave; t < T; t += kRouteThreads / 64) {
    float lv[kSlots];
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
      const int e = lane + 64 * s;
      lv[s] = -INFINITY;
      if (e < n) {
        float l;
        if (a.logits_in) {
          l = a.logits_in[(size_t)t * n + e];
        } else {
          l = a.part[(size_t)t * n + e];
          for (int c = 1; c < a.kc; ++c) l += a.part[((size_t)c * T + t) * n + e];
        }
        if (a.bias) l = l + a.bias[e];
        a.r.logits[(size_t)t * n + e] = l;
        lv[s] = (l != l) ? -INFINITY : l;   // NaN ranks last
      }
    }
    // group-limited top-k: keep the kdept departments with the largest
    // maximum logit (ties to the lower department id)
    uint64_t keep = ~0ull;
    if (a.kdept > 0) {
      if (lane < m) s_gs[wave][lane] = ord_key(-INFINITY);
      wave_lds_sync();
#pragma unroll
      for (int s = 0; s < kSlots; ++s) {
        const int e = lane + 64 * s;
        if (e < n) atomicMax(&s_gs[wave][e / E], ord_key(lv[s]));
      }
      wave_lds_sync();
      const float gsv = lane < m ? ord_val(s_gs[wave][lane]) : -INFINITY;
      keep = 0;
      for (int r = 0; r < a.kdept; ++r) {
        float bv = -INFINITY;
        int bj = 0x7fffffff;
        if (lane < m && !((keep >> lane) & 1)) { bv = gsv; bj = lane; }
        wave_argmax(bv, bj);
        keep |= 1ull << bj;
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
      for (int s = 0; s < kSlots; ++s) {
        const int e = lane + 64 * s;
        const bool ok = e < n && !((taken >> s) & 1) && ((keep >> ((e / E) & 63)) & 1 || a.kdept == 0);
        if (ok && ranks_before(lv[s], e, bv, be)) { bv = lv[s]; be = e; }
      }
      wave_argmax(bv, be);
      if (be >= n) be = 0;   // unreachable: at least k experts are always eligible
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
        for (int s = 0; s < kSlots; ++s) lm = fmaxf(lm, lv[s]);
        mx = wave_max(lm);
        float ls = 0.f;
#pragma unroll
        for (int s = 0; s < kSlots; ++s)
          if (lane + 64 * s < n) ls += expf(lv[s] - mx);
        den = wave_sum(ls);
      }
      p = expf(my_l - mx) / den;
    } else {
      const float sg = 1.0f / (1.0f + expf(-my_l));
      if (a.renorm) {
        const float den = wave_sum(sel ? sg : 0.f);
        p = sg / den;
      } else {
        p = sg;
      }
    }
    p *= a.route_scale;
    if (sel) {
      a.r.topk_ids[t * k + lane] = my_id;
      a.r.topk_w[t * k + lane] = p;
      s_ids[t * k + lane] = my_id;
      s_w[t * k + lane] = p;
      atomicOr(&s_ebits[t * nwords + (my_id >> 5)], 1u << (my_id & 31));
    }
    // distinct departments, ascending, with the summed weight in rank order
    const int d = sel ? my_id / E : 0x7fffffff;
    uint32_t eq = 0;
    for (int q = 0; q < k; ++q) eq |= (uint32_t)(__shfl(d, q) == d) << q;
    const bool first = sel && (eq & ((1u << lane) - 1u)) == 0;   // no earlier rank in d
    int pos = 0;
    float P = 0.f;
    for (int q = 0; q < k; ++q) {
      const int dq = __shfl(d, q);
      const bool fq = __shfl((int)first, q) != 0;
      const float pq = __shfl(p, q);
      pos += (fq && dq < d) ? 1 : 0;
      if (dq == d) P += pq;
    }
    const int nd = __popcll(__ballot(first));
    if (first) {
      a.r.tok_depts[t * k + pos] = d;
      a.r.tok_dept_w[t * k + pos] = P;
      s_dep[t * k + pos] = d;
      s_dw[t * k + pos] = P;
    }
    if (lane >= nd && lane < k) {
      a.r.tok_depts[t * k + lane] = -1;
      a.r.tok_dept_w[t * k + lane] = 0.f;
    }
    if (lane == 0) {
      a.r.tok_ndept[t] = nd;
      s_nd[t] = nd;
    }
  }
  __syncthreads();

  // ---------------------------------------------------------------- phase 2
  // counts: department j is touched by token t when j is among its departments
  int my_dc = 0, my_ec[2] = {0, 0};
  if (tid < m) {
    for (int t = 0; t < T; ++t)
      for (int r = 0; r < s_nd[t]; ++r) my_dc += s_dep[t * k + r] == tid;
    s_dcnt[tid] = my_dc;
    a.r.dept_count[tid] = my_dc;
  }
  for (int q = 0; q < 2; ++q) {
    const int e = tid + q * kRouteThreads;
    if (e < n) {
      int c = 0;
      for (int t = 0; t < T; ++t) c += (s_ebits[t * nwords + (e >> 5)] >> (e & 31)) & 1;
      my_ec[q] = c;
      s_ecnt[e] = c;
      a.r.exp_count[e] = c;
    }
  }
  __syncthreads();
  const int ndp = block_exscan(s_dcnt, m, s_tmp);
  const int nep = block_exscan(s_ecnt, n, s_tmp);
  if (tid < m) a.r.dept_offset[tid] = s_dcnt[tid];
  for (int e = tid; e < n; e += kRouteThreads) a.r.exp_offset[e] = s_ecnt[e];
  if (tid == 0) {
    a.r.dept_offset[m] = ndp;
    a.r.exp_offset[n] = nep;
  }
  // department token lists (ascending t); remember each (t, dept slot)'s pair
  const int my_doff = tid < m ? s_dcnt[tid] : 0;
  if (tid < m) {
    int pos = my_doff;
    for (int t = 0; t < T; ++t)
      for (int r = 0; r < s_nd[t]; ++r)
        if (s_dep[t * k + r] == tid) {
          a.r.dept_tokens[pos] = t;
          s_pair[t * k + r] = pos;
          ++pos;
        }
  }
  __syncthreads();
  int my_eoff[2] = {0, 0};
  for (int q = 0; q < 2; ++q) {
    const int e = tid + q * kRouteThreads;
    if (e >= n) continue;
    my_eoff[q] = s_ecnt[e];
    int pos = my_eoff[q];
    for (int t = 0; t < T; ++t) {
      if (!((s_ebits[t * nwords + (e >> 5)] >> (e & 31)) & 1)) continue;
      a.r.exp_tokens[pos] = t;
      int r = 0;
      while (r < k - 1 && s_ids[t * k + r] != e) ++r;
      if (a.plan) {
        a.tok_exp_pair[t * k + r] = pos;
        if (a.plan == PLAN_FACTORED) {
          int q2 = 0;
          while (q2 < s_nd[t] - 1 && s_dep[t * k + q2] != e / E) ++q2;
          a.exp_src[pos] = s_pair[t * k + q2];
        }
      }
      ++pos;
    }
  }
  if (!a.plan) return;
  __syncthreads();

  // ---------------------------------------------------------------- phase 3
  const bool has_priv = a.plan == PLAN_FACTORED || a.d_p > 0;
  const bool has_se = a.d_se > 0;
  // unit index of every active department / expert (prefix over active flags)
  if (tid < m) s_dcnt[tid] = my_dc > 0;
  for (int q = 0; q < 2; ++q) {
    const int e = tid + q * kRouteThreads;
    if (e < n) s_ecnt[e] = has_priv && my_ec[q] > 0;
  }
  __syncthreads();
  const int ud = block_exscan(s_dcnt, m, s_tmp);
  const int ue = block_exscan(s_ecnt, n, s_tmp);
  const int th = (a.h + kTile - 1) / kTile;
  const int nep_priv = has_priv ? nep : 0;
  const int wb = a.w_bytes, ab = a.act_f32 ? 4 : 2;
  const char *x = static_cast<const char *>(a.x);
  auto wptr = [&](const void *base, int idx, int R, int C) {
    return static_cast<const char *>(base) + (size_t)idx * R * C * wb;
  };
  auto sptr = [&](const float *base, int idx, int R, int C) -> const float * {
    if (!a.fp8) return nullptr;
    return base + (size_t)idx * ((R + 127) / 128) * (C / 128);
  };
  auto make = [&](const void *w0, const void *w1, const float *s0, const float *s1, const void *in0,
                  const void *in1, const int32_t *idx, void *out0, void *out1, int R, int K,
                  int ldin, int ldout, int ntok, int tile_begin, int epi, int out_f32) {
    GemmUnit U;
    U.w0 = w0; U.w1 = w1; U.s0 = s0; U.s1 = s1; U.in0 = in0; U.in1 = in1; U.idx = idx;
    U.out0 = out0; U.out1 = out1; U.R = R; U.K = K; U.ldw = K; U.ldin = ldin; U.ldout = ldout;
    U.ntok = ntok; U.tile_begin = tile_begin; U.epi = epi; U.out_f32 = out_f32; U.pad_ = 0;
    return U;
  };
  const deamoe_weights &W = a.w;
  if (a.plan == PLAN_SLICE) {
    const int ta_d = (a.d_s + kTile - 1) / kTile, ta_p = (a.d_p + kTile - 1) / kTile;
    if (tid < m && my_dc > 0) {
      const int j = tid, u = s_dcnt[j];
      const int32_t *idx = a.r.dept_tokens + my_doff;
      char *ao = static_cast<char *>(a.abuf_dept) + (size_t)my_doff * a.d_s * ab;
      a.units[0][u] = make(wptr(W.dept_gate, j, a.d_s, a.h), wptr(W.dept_up, j, a.d_s, a.h),
                           sptr(W.scale[0], j, a.d_s, a.h), sptr(W.scale[1], j, a.d_s, a.h), x, x,
                           idx, ao, nullptr, a.d_s, a.h, a.h, a.d_s, my_dc, u * ta_d, EPI_SWIGLU,
                           a.act_f32);
      a.units[1][u] = make(wptr(W.dept_down, j, a.h, a.d_s), nullptr, sptr(W.scale[2], j, a.h, a.d_s),
                           nullptr, ao, ao, nullptr, a.partial + (size_t)my_doff * a.h, nullptr,
                           a.h, a.d_s, a.d_s, a.h, my_dc, u * th, EPI_STORE, 1);
    }
    for (int q = 0; q < 2; ++q) {
      const int e = tid + q * kRouteThreads;
      if (!has_priv || e >= n || my_ec[q] == 0) continue;
      const int u = ud + s_ecnt[e];
      const int32_t *idx = a.r.exp_tokens + my_eoff[q];
      char *ao = static_cast<char *>(a.abuf_exp) + (size_t)my_eoff[q] * a.d_p * ab;
      a.units[0][u] = make(wptr(W.priv_gate, e, a.d_p, a.h), wptr(W.priv_up, e, a.d_p, a.h),
                           sptr(W.scale[3], e, a.d_p, a.h), sptr(W.scale[4], e, a.d_p, a.h), x, x,
                           idx, ao, nullptr, a.d_p, a.h, a.h, a.d_p, my_ec[q],
                           ud * ta_d + s_ecnt[e] * ta_p, EPI_SWIGLU, a.act_f32);
      a.units[1][u] = make(wptr(W.priv_down, e, a.h, a.d_p), nullptr, sptr(W.scale[5], e, a.h, a.d_p),
                           nullptr, ao, ao, nullptr, a.partial + (size_t)(ndp + my_eoff[q]) * a.h,
                           nullptr, a.h, a.d_p, a.d_p, a.h, my_ec[q], u * th, EPI_STORE, 1);
    }
    if (tid == 0) {
      int units = ud + ue, tiles_a = ud * ta_d + ue * ta_p;
      if (has_se) {
        const int ta_se = (a.d_se + kTile - 1) / kTile;
        a.units[0][units] = make(W.se_gate, W.se_up, sptr(W.scale[6], 0, a.d_se, a.h),
                                 sptr(W.scale[7], 0, a.d_se, a.h), x, x, nullptr, a.abuf_se, nullptr,
                                 a.d_se, a.h, a.h, a.d_se, T, tiles_a, EPI_SWIGLU, a.act_f32);
        a.units[1][units] = make(W.se_down, nullptr, sptr(W.scale[8], 0, a.h, a.d_se), nullptr,
                                 a.abuf_se, a.abuf_se, nullptr,
                                 a.partial + (size_t)(ndp + nep_priv) * a.h, nullptr, a.h, a.d_se,
                                 a.d_se, a.h, T, units * th, EPI_STORE, 1);
        tiles_a += ta_se;
        ++units;
      }
      a.counts->stage[0][0] = units;
      a.counts->stage[0][1] = tiles_a;
      a.counts->stage[1][0] = units;
      a.counts->stage[1][1] = units * th;
    }
  } else {  // PLAN_FACTORED
    const int d = a.d_s, td = (d + kTile - 1) / kTile;
    if (tid < m && my_dc > 0) {
      const int j = tid, u = s_dcnt[j];
      const int32_t *idx = a.r.dept_tokens + my_doff;
      char *go = static_cast<char *>(a.gbuf) + (size_t)my_doff * d * ab;
      char *uo = static_cast<char *>(a.ubuf) + (size_t)my_doff * d * ab;
      char *zs = static_cast<char *>(a.zsbuf) + (size_t)my_doff * d * ab;
      a.units[0][u] = make(wptr(W.dept_gate, j, d, a.h), wptr(W.dept_up, j, d, a.h),
                           sptr(W.scale[0], j, d, a.h), sptr(W.scale[1], j, d, a.h), x, x, idx, go,
                           uo, d, a.h, a.h, d, my_dc, u * td, EPI_SIGMA2, a.act_f32);
      a.units[3][u] = make(wptr(W.dept_down, j, a.h, d), nullptr, sptr(W.scale[2], j, a.h, d),
                           nullptr, zs, zs, nullptr, a.partial + (size_t)my_doff * a.h, nullptr,
                           a.h, d, d, a.h, my_dc, u * th, EPI_STORE, 1);
    }
    for (int q = 0; q < 2; ++q) {
      const int e = tid + q * kRouteThreads;
      if (e >= n || my_ec[q] == 0) continue;
      const int u = s_ecnt[e];
      char *yo = static_cast<char *>(a.ybuf) + (size_t)my_eoff[q] * d * ab;
      a.units[1][u] = make(wptr(W.priv_gate, e, d, d), wptr(W.priv_up, e, d, d),
                           sptr(W.scale[3], e, d, d), sptr(W.scale[4], e, d, d), a.gbuf, a.ubuf,
                           a.exp_src + my_eoff[q], yo, nullptr, d, d, d, d, my_ec[q], u * td,
                           EPI_SWIGLU, a.act_f32);
      a.units[2][u] = make(wptr(W.priv_down, e, d, d), nullptr, sptr(W.scale[5], e, d, d), nullptr,
                           yo, yo, nullptr, a.zbuf + (size_t)my_eoff[q] * d, nullptr, d, d, d, d,
                           my_ec[q], u * td, EPI_SIGMA, 1);
    }
    if (tid == 0) {
      int units0 = ud, tiles0 = ud * td, units3 = ud;
      if (has_se) {
        const int ta_se = (a.d_se + kTile - 1) / kTile;
        a.units[0][units0] = make(W.se_gate, W.se_up, sptr(W.scale[6], 0, a.d_se, a.h),
                                  sptr(W.scale[7], 0, a.d_se, a.h), x, x, nullptr, a.abuf_se,
                                  nullptr, a.d_se, a.h, a.h, a.d_se, T, tiles0, EPI_SWIGLU,
                                  a.act_f32);
        a.units[3][units3] = make(W.se_down, nullptr, sptr(W.scale[8], 0, a.h, a.d_se), nullptr,
                                  a.abuf_se, a.abuf_se, nullptr, a.partial + (size_t)ndp * a.h,
                                  nullptr, a.h, a.d_se, a.d_se, a.h, T, units3 * th, EPI_STORE, 1);
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
      a.counts->stage[3][1] = units3 * th;
    }
  }
  if (tid == 0) {
    a.counts->n_dept_pairs = ndp;
    a.counts->n_exp_pairs = nep_priv;
    a.counts->n_pairs = ndp + (a.plan == PLAN_SLICE ? nep_priv : 0) + (has_se ? T : 0);
  }
  // combine slots of every token: its departments (ascending), then (SLICE)
  // its experts in rank order, then the shared expert
  for (int t = tid; t < T; t += kRouteThreads) {
    int ns = 0;
    int32_t *sp = a.slot_pair + (size_t)t * a.max_slots;
    float *sw = a.slot_w + (size_t)t * a.max_slots;
    for (int r = 0; r < s_nd[t]; ++r) {
      sp[ns] = s_pair[t * k + r];
      sw[ns] = a.plan == PLAN_SLICE ? s_dw[t * k + r] : 1.0f;
      ++ns;
    }
    if (a.plan == PLAN_SLICE && a.d_p > 0)
      for (int r = 0; r < k; ++r) {
        sp[ns] = ndp + a.tok_exp_pair[t * k + r];
        sw[ns] = s_w[t * k + r];
        ++ns;
      }
    if (has_se) {
      sp[ns] = ndp + (a.plan == PLAN_SLICE ? nep_priv : 0) + t;
      sw[ns] = 1.0f;
      ++ns;
    }
    a.nslot[t] = ns;
  }
}

hipError_t launch_route_plan(const RouteArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(route_plan_kernel, dim3(1), dim3(kRouteThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace deamoe
