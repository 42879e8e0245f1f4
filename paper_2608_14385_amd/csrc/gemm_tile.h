// Skinny grouped matrix product on gfx950 matrix cores.
//
// One wave computes a 16-row tile of one or two weight matrices (gate and up
// share the token operand) against up to 16 * NTT token rows, streaming the
// weights from HBM exactly once.  Lane l owns weight row (l % 16) of the tile
// and, in every K step, a contiguous run of K / 4 elements starting at
// k0 + (l / 16) * (K_STEP / 4); the token operand is loaded with the same
// K permutation, so the 16x16 matrix-core products sum over the whole step.
//
// Weight formats:
//   WT_F32  fp32 weights, fp32 tokens:   v_mfma_f32_16x16x4_f32,  K_STEP 64
//   WT_BF16 bf16 weights, bf16 tokens:   v_mfma_f32_16x16x32_bf16, K_STEP 128
//   WT_FP8  e4m3 weights (128x128 block scales), bf16 tokens: every code is
//           widened exactly to bf16, the step's products accumulate in a
//           fresh register tile and are added with the block scale, so each
//           K step is exactly one scale block.
#pragma once

#include "internal.h"

namespace deamoe {

enum WType : int { WT_F32 = 0, WT_BF16 = 1, WT_FP8 = 2 };

template <int WT>
struct WTraits;
template <>
struct WTraits<WT_F32> {
  static constexpr int K_STEP = 64, W_BYTES = 4, A_BYTES = 4, W_VEC = 4;
};
template <>
struct WTraits<WT_BF16> {
  static constexpr int K_STEP = 128, W_BYTES = 2, A_BYTES = 2, W_VEC = 4;
};
template <>
struct WTraits<WT_FP8> {
  static constexpr int K_STEP = 128, W_BYTES = 1, A_BYTES = 2, W_VEC = 2;
};

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// A value every lane of the wave holds alike, moved to a scalar register so
// that the control flow depending on it is scalar.
__device__ inline int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Eight e4m3 codes (two dwords) -> eight bf16 (exact: e4m3 values are bf16 values).
__device__ inline bf16x8 fp8x8_to_bf16(uint32_t lo, uint32_t hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, true);
  bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, false);
  bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, true);
  bf16x8 r = {a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
  return r;
}

typedef __attribute__((address_space(1))) const u32x4 gvec;

__device__ inline const gvec *gptr(const void *p) {
  return reinterpret_cast<const gvec *>(reinterpret_cast<uintptr_t>(p));
}

// Token-operand row of token i of a unit.
__device__ inline const char *token_row(const void *base, const int32_t *idx, int ldin, int i,
                                        int abytes) {
  const int row = idx ? idx[i] : i;
  return static_cast<const char *>(base) + (size_t)row * ldin * abytes;
}

// Byte offset, inside one K step of a token row, of the 16-byte token chunk
// that pairs with matrix-core product q (q < 4) of lane group g.
template <int WT>
__device__ inline int b_chunk_offset(int g, int q) {
  if constexpr (WT == WT_FP8) return (q >> 1) * 128 + g * 32 + (q & 1) * 16;
  return q * 64 + g * 16;
}

// Token operand of one K step for every token tile: B[tt][0..3] pairs with
// gate / single weights, B[tt][4..7] with up weights when their inputs differ.
template <int WT, int NTT, bool SPLIT>
__device__ inline void load_b(u32x4 (&B)[NTT][SPLIT ? 8 : 4], const char *const (&bp0)[NTT],
                              const char *const (&bp1)[NTT], int ntt, size_t boff, int g) {
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    if (tt > 0 && tt >= ntt) break;   // ntt >= 1
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      B[tt][q] = *gptr(bp0[tt] + boff + b_chunk_offset<WT>(g, q));
      if constexpr (SPLIT) B[tt][4 + q] = *gptr(bp1[tt] + boff + b_chunk_offset<WT>(g, q));
    }
  }
}

// The matrix-core products of one K step.
template <int WT, int NW, int NTT, bool SPLIT>
__device__ inline void step_mma(const u32x4 (&a)[NW][WTraits<WT>::W_VEC],
                                const u32x4 (&B)[NTT][SPLIT ? 8 : 4], int ntt, const float (&sc)[NW],
                                f32x4 (&acc)[NW][NTT]) {
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    if (tt > 0 && tt >= ntt) break;   // ntt >= 1
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const int bo = (SPLIT && n == 1) ? 4 : 0;
      if constexpr (WT == WT_BF16) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          acc[n][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a[n][q]),
                                                               as_bf16x8(B[tt][bo + q]), acc[n][tt],
                                                               0, 0, 0);
      } else if constexpr (WT == WT_FP8) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t lo = a[n][q >> 1][(q & 1) * 2], hi = a[n][q >> 1][(q & 1) * 2 + 1];
          t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(lo, hi),
                                                      as_bf16x8(B[tt][bo + q]), t, 0, 0, 0);
        }
        acc[n][tt] += sc[n] * t;
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[n][tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[n][v][e]),
                                                              __uint_as_float(B[tt][bo + v][e]),
                                                              acc[n][tt], 0, 0, 0);
      }
    }
  }
}

// Accumulate the wave's tile over the K steps kp, kp + ks, ... of unit U.
// Lane (j = l % 16, g = l / 16) owns weight row j of the tile; in each K step
// its v-th 16-byte chunk sits at byte v * 64 + g * 16 of the row's step
// segment, so every load instruction reads 64 contiguous bytes per row.
// Rows past R and tokens past ntok are clamped to valid ones: their products
// land only in output rows / columns that are never stored.
// Software pipeline (loads retire in issue order): the token operand of a
// step is requested before the weights two steps ahead, so waiting for it
// never waits for the prefetched weights; two weight buffers alternate.
template <int WT, int NW, int NTT, bool SPLIT>
__device__ inline void tile_loop(const GemmUnit &U, int rt, int kp, int ks, f32x4 (&acc)[NW][NTT]) {
  using Tr = WTraits<WT>;
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int row = min(rt * kTile + j, U.R - 1);
  const char *wp[NW];
  wp[0] = static_cast<const char *>(U.w0) + (size_t)row * U.ldw * Tr::W_BYTES + g * 16;
  if constexpr (NW == 2)
    wp[1] = static_cast<const char *>(U.w1) + (size_t)row * U.ldw * Tr::W_BYTES + g * 16;
  const int ntt = uniform(min(NTT, (U.ntok + kTile - 1) / kTile));
  const char *bp0[NTT];
  const char *bp1[NTT];
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    int i = tt * kTile + j;
    i = i < U.ntok ? i : 0;
    bp0[tt] = token_row(U.in0, U.idx, U.ldin, i, Tr::A_BYTES);
    bp1[tt] = SPLIT ? token_row(U.in1, U.idx, U.ldin, i, Tr::A_BYTES) : bp0[tt];
  }
  const int nsteps = uniform(U.K / Tr::K_STEP);
  constexpr int WSEG = Tr::K_STEP * Tr::W_BYTES;     // bytes of one row per K step
  constexpr int ASEG = Tr::K_STEP * Tr::A_BYTES;     // bytes of one token row per K step
  const int sblocks = U.K / 128;
  const int srow = (rt * kTile) / 128;
  if (kp >= nsteps) return;
  u32x4 A0[NW][Tr::W_VEC], A1[NW][Tr::W_VEC];
  u32x4 B[NTT][SPLIT ? 8 : 4];
  // Past the last step the prefetch reads the first token row instead (a
  // cache-resident address), so that every iteration issues the same loads.
  const char *dummy = bp0[0] + g * 16;
  auto load_w = [&](u32x4(&A)[NW][Tr::W_VEC], int step) {
    const bool ok = step < nsteps;
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const char *p = ok ? wp[n] + (size_t)step * WSEG : dummy;
#pragma unroll
      for (int v = 0; v < Tr::W_VEC; ++v) A[n][v] = __builtin_nontemporal_load(gptr(p + v * 64));
    }
  };
  auto scales = [&](float (&sc)[NW], int step) {
    if constexpr (WT == WT_FP8) {
      sc[0] = U.s0[srow * sblocks + step];
      if constexpr (NW == 2) sc[1] = U.s1[srow * sblocks + step];
    }
  };
  float sc[NW];
  // sched_barrier keeps the backend from sinking the prefetch next to its use.
  load_w(A0, kp);
  load_b<WT, NTT, SPLIT>(B, bp0, bp1, ntt, (size_t)kp * ASEG, g);
  scales(sc, kp);
  load_w(A1, kp + ks);
  __builtin_amdgcn_sched_barrier(0);
  for (int s = kp;;) {
    step_mma<WT, NW, NTT, SPLIT>(A0, B, ntt, sc, acc);
    s += ks;
    if (s >= nsteps) break;
    __builtin_amdgcn_sched_barrier(0);
    load_b<WT, NTT, SPLIT>(B, bp0, bp1, ntt, (size_t)s * ASEG, g);
    scales(sc, s);
    load_w(A0, s + ks);
    __builtin_amdgcn_sched_barrier(0);
    step_mma<WT, NW, NTT, SPLIT>(A1, B, ntt, sc, acc);
    s += ks;
    if (s >= nsteps) break;
    __builtin_amdgcn_sched_barrier(0);
    load_b<WT, NTT, SPLIT>(B, bp0, bp1, ntt, (size_t)s * ASEG, g);
    scales(sc, s);
    load_w(A1, s + ks);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int WT, int NW, int NTT>
__device__ inline void tile_compute(const GemmUnit &U, int rt, int kp, int ks,
                                    f32x4 (&acc)[NW][NTT]) {
  if (NW == 2 && U.in1 != U.in0)
    tile_loop<WT, NW, NTT, true>(U, rt, kp, ks, acc);
  else
    tile_loop<WT, NW, NTT, false>(U, rt, kp, ks, acc);
}

// Four consecutive outputs (fp32 or bf16) at element offset off; `full`
// false writes only the first `left` of them.
__device__ inline void store4(void *base, int out_f32, size_t off, f32x4 o, bool full, int left) {
  if (out_f32) {
    float *p = static_cast<float *>(base) + off;
    if (full) {
      *reinterpret_cast<f32x4 *>(p) = o;
    } else {
      for (int r = 0; r < left; ++r) p[r] = o[r];
    }
  } else {
    uint16_t *p = static_cast<uint16_t *>(base) + off;
    if (full) {
      const uint32_t lo = f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
      const uint32_t hi = f32_to_bf16(o[2]) | ((uint32_t)f32_to_bf16(o[3]) << 16);
      *reinterpret_cast<u32x2 *>(p) = u32x2{lo, hi};
    } else {
      for (int r = 0; r < left; ++r) p[r] = f32_to_bf16(o[r]);
    }
  }
}

__device__ inline float apply_sigma(float v, int sigma) {
  return sigma == DEAMOE_SIGMA_NONE ? v : silu_f(v);
}

__device__ inline f32x4 sigma4(f32x4 v, int sigma) {
  return f32x4{apply_sigma(v[0], sigma), apply_sigma(v[1], sigma), apply_sigma(v[2], sigma),
               apply_sigma(v[3], sigma)};
}

// Write the finished tile.  Lane l holds rows 4 * (l / 16) + r, r < 4, of
// the tile for token (l % 16) of each token tile.
template <int NW, int NTT>
__device__ inline void tile_epilogue(const GemmUnit &U, int rt, int sigma, const f32x4 (&acc)[NW][NTT]) {
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int R = uniform(U.R), ntok = uniform(U.ntok), epi = uniform(U.epi);
  const int out_f32 = uniform(U.out_f32), ldout = uniform(U.ldout);
  const int row0 = rt * kTile + 4 * g;
  if (row0 >= R) return;
  const bool full = row0 + 3 < R;
  const int ntt = uniform(min(NTT, (ntok + kTile - 1) / kTile));
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    if (tt > 0 && tt >= ntt) break;   // ntt >= 1
    const int i = tt * kTile + j;
    if (i >= ntok) continue;
    const size_t off = (size_t)i * ldout + row0;
    const f32x4 v0 = acc[0][tt];
    if constexpr (NW == 2) {
      const f32x4 v1 = acc[1][tt];
      if (epi == EPI_SWIGLU) {
        const f32x4 o = f32x4{silu_f(v0[0]) * v1[0], silu_f(v0[1]) * v1[1], silu_f(v0[2]) * v1[2],
                              silu_f(v0[3]) * v1[3]};
        store4(U.out0, out_f32, off, o, full, R - row0);
      } else {   // EPI_SIGMA2
        store4(U.out0, out_f32, off, sigma4(v0, sigma), full, R - row0);
        store4(U.out1, out_f32, off, sigma4(v1, sigma), full, R - row0);
      }
    } else {
      const f32x4 o = epi == EPI_SIGMA ? sigma4(v0, sigma) : v0;
      store4(U.out0, out_f32, off, o, full, R - row0);
    }
  }
}

// One workgroup of 4 waves: 4 / KS tiles, each split over KS waves along K
// (interleaved K steps), partial tiles summed in a fixed order through LDS.
template <int WT, int NW, int NTT, int KS>
struct TileRunner {
  static constexpr int TPB = 4 / KS;
  struct Smem {
    f32x4 red[KS > 1 ? 4 : 1][NW * NTT][kWave];
  };

  __device__ static void run(Smem &sm, const GemmUnit *U, int rt, bool active, int sigma) {
    const int wave = uniform(threadIdx.x / kWave), lane = lane_id();
    const int kp = uniform(wave % KS);
    rt = uniform(rt);
    f32x4 acc[NW][NTT];
#pragma unroll
    for (int n = 0; n < NW; ++n)
#pragma unroll
      for (int tt = 0; tt < NTT; ++tt) acc[n][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (active) tile_compute<WT, NW, NTT>(*U, rt, kp, KS, acc);
    if constexpr (KS > 1) {
      if (active && kp > 0) {
#pragma unroll
        for (int n = 0; n < NW; ++n)
#pragma unroll
          for (int tt = 0; tt < NTT; ++tt) sm.red[wave][n * NTT + tt][lane] = acc[n][tt];
      }
      __syncthreads();
      if (active && kp == 0) {
        for (int q = 1; q < KS; ++q)
#pragma unroll
          for (int n = 0; n < NW; ++n)
#pragma unroll
            for (int tt = 0; tt < NTT; ++tt) acc[n][tt] += sm.red[wave + q][n * NTT + tt][lane];
      }
      __syncthreads();
    }
    if (active && kp == 0) tile_epilogue<NW, NTT>(*U, rt, sigma, acc);
  }
};

}  // namespace deamoe
