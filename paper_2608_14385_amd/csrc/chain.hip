// Down projections fused with the weighted combine of Eq. 3, for batches of
// at most 32 tokens (one or two token tiles of 16).
//
// For every active unit u (department, expert, shared expert) the gate/up
// stage has stored a_{t,u} = SiLU(G_u x_t) * (U_u x_t) for the unit's tokens,
// one row per member token in ascending token order.  The layer output is
//
//   y_t = sum_u p_{t,u} W_u a_{t,u}
//
// (P_{t,j} for a department, Sec. 3.2), one product over the concatenated K
// steps of all units in which token t's column carries the weight p_{t,u}
// and zero for units it does not use.  A workgroup owns 32 rows of y (two
// 16-row halves sharing the token operand; 16 rows on narrow layers) and
// splits the concatenated K
// steps into KSC contiguous ranges, one per wave, so that every wave streams
// one long run of weight rows; each K step's product is added to the
// accumulator with the lane's token weight (times the fp8 block scale), and
// the partial tiles are summed through LDS in wave order and rounded once.
// No fp32 partial rows and no combine launch.  The FACTORED department down
// projections (W_d^T Z) are the same product over the departments, with the
// routing weights already inside Z and unit weights here.
#include "gemm_tile.h"
#include "launch.h"

namespace deamoe {

// One K step of every half: the step's products start from zero and are
// added with the per-lane factor f (the token's weight, times the fp8 scale).
template <int WT, int NW, int NTT>
__device__ inline void chain_mma(const u32x4 (&a)[NW][4], const u32x4 (&b)[4], float f,
                                 f32x4 (&acc)[NW][NTT], int tt) {
#pragma unroll
  for (int n = 0; n < NW; ++n) {
    f32x4 t = {0.f, 0.f, 0.f, 0.f};
    if constexpr (WT == WT_F32) {
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          t = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[n][m][e]),
                                                   __uint_as_float(b[m][e]), t, 0, 0, 0);
    } else {
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const bf16x8 w = WT == WT_FP8 ? fp8x8_to_bf16(a[n][m][0], a[n][m][1]) : as_bf16x8(a[n][m]);
        t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, as_bf16x8(b[m]), t, 0, 0, 0);
      }
    }
    acc[n][tt] += f * t;
  }
}

// A 64-bit pointer every lane holds alike, moved to scalar registers.
template <class P>
__device__ inline P *uniform_ptr(P *p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<P *>(((uint64_t)hi << 32) | lo);
}

// NW: 16-row halves of y per workgroup (1 or 2; two share the token operand).
template <int WT, int NW, int NTT, int KSC, int PF>
__global__ __launch_bounds__(KSC * kWave) void chain_down_kernel(ChainArgs a) {
  using Tr = WTraits<WT>;
  using LD = WLoad<WT>;
  constexpr int TR = NW * kTile;   // rows of y per workgroup
  constexpr int NB = PF + 1;       // load groups per wave: PF in flight, one multiplied
  constexpr int ASEG = Tr::K_STEP * Tr::A_BYTES;
  constexpr int STAGE = NW * LD::REGION;
  constexpr int RED = NW * NTT * kWave * 16;
  constexpr int WB = STAGE > RED ? STAGE : RED;
  __shared__ __attribute__((aligned(16))) char s_buf[KSC][WB];
  __shared__ ChainUnit s_u[kMaxChainUnits];
  const int n_units = uniform(a.counts[0]), S = uniform(a.counts[1]);
  {
    const uint32_t *src = reinterpret_cast<const uint32_t *>(a.units);
    uint32_t *dst = reinterpret_cast<uint32_t *>(s_u);
    const int nd = n_units * (int)(sizeof(ChainUnit) / 4);
    for (int i = threadIdx.x; i < nd; i += blockDim.x) dst[i] = src[i];
  }
  __syncthreads();
  const int wave = uniform(threadIdx.x / kWave), lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int T = a.T, R = a.h, rt = blockIdx.x;
  const int lrow = lane / LD::LPR, lchunk = lane % LD::LPR;
  const int rmax = R - 1 - (NW - 1) * kTile;   // last row the first half may read
  const int s_lo = uniform((int)((int64_t)S * wave / KSC));
  const int total = uniform((int)((int64_t)S * (wave + 1) / KSC)) - s_lo;
  char *lds = s_buf[wave];
  // acc[n][tt]: rows of half n, tokens 16 * tt + (lane % 16)
  f32x4 acc[NW][NTT];
#pragma unroll
  for (int n = 0; n < NW; ++n)
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt) acc[n][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (total > 0) {
    // the unit holding step s_lo: the last one whose first step is <= s_lo
    int lo = 0, hi = n_units - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (uniform(s_u[mid].step0) <= s_lo) lo = mid; else hi = mid - 1;
    }
    int cu = uniform(lo);
    // issue cursor: unit cu, its K step ck of nk; the unit's per-lane state
    int ck = s_lo - uniform(s_u[cu].step0), nk = 0, ldw = 0;
    const char *w0 = nullptr, *bp[NTT];
    const float *sp = nullptr, *pp[NTT];
    uint64_t mm[NTT];   // per token tile: lanes whose token is a member of the unit
    const uint32_t tmask = T >= 32 ? 0xffffffffu : (1u << T) - 1u;
    auto load_unit = [&](int u) {
      ldw = uniform(s_u[u].K);
      nk = ldw / Tr::K_STEP;
      w0 = static_cast<const char *>(uniform_ptr(s_u[u].w)) + lchunk * 16;
      const uint32_t m32 = (uint32_t)uniform((int)s_u[u].mask) & tmask;
      const char *in = static_cast<const char *>(uniform_ptr(s_u[u].in));
      const float *pw = uniform_ptr(s_u[u].pw);
#pragma unroll
      for (int tt = 0; tt < NTT; ++tt) {
        const uint32_t m16 = (m32 >> (kTile * tt)) & 0xffffu;
        mm[tt] = (uint64_t)m16 * 0x0001000100010001ull;
        // a member's row is its rank among the members; other lanes read the
        // first member's row (their weight is zero), so each load touches
        // only the unit's rows
        const int tok = kTile * tt + j;
        const int rank = (m16 >> j) & 1 ? __popc(m32 & ((1u << tok) - 1u)) : 0;
        bp[tt] = in + (size_t)rank * ldw * Tr::A_BYTES;
        pp[tt] = pw + tok;
      }
      if constexpr (WT == WT_FP8)   // the tile's 32 rows lie in one scale row
        sp = uniform_ptr(s_u[u].s) + (size_t)((rt * TR) / 128) * (ldw / 128);
    };
    load_unit(cu);
    // loads past the wave's range read cache-resident data of the first unit
    const char *dummy = bp[0] + (lane & 15) * 16;
    const char *dummy_b = bp[0];
    const float *dummy_s = sp, *dummy_p = pp[0];
    u32x4 G[NB][NW][LD::NQ];
    u32x4 B[NB][NTT][4];
    uint64_t MM[NB][NTT];
    float SC[NB], P[NB][NTT];
    auto issue = [&](u32x4(&Gb)[NW][LD::NQ], u32x4(&Bb)[NTT][4], uint64_t(&mms)[NTT], float &sc,
                     float(&pw)[NTT], int v) {
      const bool ok = v < total;
      if (ok && ck == nk) {   // the previous step ended a unit
        ++cu;
        ck = 0;
        load_unit(cu);
      }
#pragma unroll
      for (int q = 0; q < LD::NQ; ++q) {
        const int row = min(rt * TR + q * LD::RPI + lrow, rmax);
        const size_t woff = (size_t)row * ldw * Tr::W_BYTES + (size_t)ck * LD::WSEG;
        const size_t half = (size_t)kTile * ldw * Tr::W_BYTES;
        Gb[0][q] = __builtin_nontemporal_load(gptr(ok ? w0 + woff : dummy));
        if constexpr (NW == 2)
          Gb[1][q] = __builtin_nontemporal_load(gptr(ok ? w0 + woff + half : dummy));
      }
#pragma unroll
      for (int tt = 0; tt < NTT; ++tt) {
        const char *b = ok ? bp[tt] + (size_t)ck * ASEG : dummy_b;
#pragma unroll
        for (int q = 0; q < 4; ++q) Bb[tt][q] = *gptr(b + b_chunk_offset(g, q));
        pw[tt] = *gfptr(ok ? pp[tt] : dummy_p);
        mms[tt] = mm[tt];
      }
      if constexpr (WT == WT_FP8) sc = *gfptr(ok ? sp + ck : dummy_s);
      if (ok) ++ck;
    };
#pragma unroll
    for (int p = 0; p < PF; ++p) issue(G[p], B[p], MM[p], SC[p], P[p], p);
    for (int v = 0;;) {
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        const int qn = (q + NB - 1) % NB;   // the buffer consumed one step ago
        issue(G[qn], B[qn], MM[qn], SC[qn], P[qn], v + PF);
        __builtin_amdgcn_sched_barrier(0);
        u32x4 w[NW][4];
        stage_weights<WT, NW>(lds, G[q], w);
#pragma unroll
        for (int tt = 0; tt < NTT; ++tt) {
          // tokens outside the unit have weight zero (their operand is a
          // member's row, so the product is finite)
          const float f0 = (MM[q][tt] >> lane) & 1 ? P[q][tt] : 0.f;
          chain_mma<WT, NW>(w, B[q][tt], WT == WT_FP8 ? f0 * SC[q] : f0, acc, tt);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (++v >= total) goto streamed;
      }
    }
  }
streamed:
  // partial tiles summed in wave order; wave 0 rounds and stores
  __syncthreads();   // every wave is done with its staging region
  f32x4 *red = reinterpret_cast<f32x4 *>(s_buf[wave]);
  if (wave > 0) {
#pragma unroll
    for (int n = 0; n < NW; ++n)
#pragma unroll
      for (int tt = 0; tt < NTT; ++tt) red[(n * NTT + tt) * kWave + lane] = acc[n][tt];
  }
  __syncthreads();
  if (wave == 0) {
    for (int q = 1; q < KSC; ++q) {
      const f32x4 *r = reinterpret_cast<const f32x4 *>(s_buf[q]);
#pragma unroll
      for (int n = 0; n < NW; ++n)
#pragma unroll
        for (int tt = 0; tt < NTT; ++tt) acc[n][tt] += r[(n * NTT + tt) * kWave + lane];
    }
    const int row0 = rt * TR + 4 * g, row1 = row0 + kTile;
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt) {
      const int tok = kTile * tt + j;
      if (tok < T) {
        const size_t off = (size_t)tok * R + row0;
        if (row0 < R) store4(a.y, a.act_f32, off, acc[0][tt], row0 + 3 < R, R - row0);
        if (NW == 2 && row1 < R)
          store4(a.y, a.act_f32, off + kTile, acc[NW - 1][tt], row1 + 3 < R, R - row1);
      }
    }
  }
}

template <int WT, int NW, int NTT>
static hipError_t launch_chain_wt(const ChainArgs &a, hipStream_t s) {
  const dim3 grid((a.h + NW * kTile - 1) / (NW * kTile));
  // 8 waves per workgroup, each streaming one contiguous range of the
  // concatenated K steps, one load group in flight while one is multiplied
  constexpr int KSC = 8, PF = 1;
  hipLaunchKernelGGL((chain_down_kernel<WT, NW, NTT, KSC, PF>), grid, dim3(KSC * kWave), 0, s, a);
  return hipGetLastError();
}

// Layers narrower than 5120 take one 16-row half per workgroup: twice the
// workgroups (two per CU, four waves per SIMD with one token tile) where row
// pairs leave most CUs idle.  Same-process A/B on the 2048-wide 7B-class
// layer: 36.7 -> 33.9 us per step at one token, 54.4 -> 49.3 at four; on
// the 4096-wide Qwen3 FACTORED layer 79.2 -> 76.9 at one token, 312.3 ->
// 305.1 at 16.  At 5120 (DeepSeek-V2 FACTORED: 86.6 -> 88.1 at one token,
// 389.0 -> 393.5 at 16) and at the 7168-wide DeepSeek-V3 shape (108.3 ->
// 110.4 us at one token, 525.4 -> 546.7 at 16) single halves were slower.
constexpr int kChainPairMinH = 5120;

template <int WT>
static hipError_t launch_chain_ntt(const ChainArgs &a, hipStream_t s) {
  if (a.h < kChainPairMinH)
    return a.T > kTile ? launch_chain_wt<WT, 1, 2>(a, s) : launch_chain_wt<WT, 1, 1>(a, s);
  return a.T > kTile ? launch_chain_wt<WT, 2, 2>(a, s) : launch_chain_wt<WT, 2, 1>(a, s);
}

hipError_t launch_chain(const ChainArgs &a, int wtype, hipStream_t s) {
  switch (wtype) {
    case WT_F32: return launch_chain_ntt<WT_F32>(a, s);
    case WT_BF16: return launch_chain_ntt<WT_BF16>(a, s);
    default: return launch_chain_ntt<WT_FP8>(a, s);
  }
}

}  // namespace deamoe
