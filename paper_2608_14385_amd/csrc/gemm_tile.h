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

// Token-operand row pointer of token i of a unit (nullptr: zero row).
__device__ inline const char *token_row(const void *base, const int32_t *idx, int ldin, int i,
                                        int abytes) {
  const int row = idx ? idx[i] : i;
  return static_cast<const char *>(base) + (size_t)row * ldin * abytes;
}

// Accumulate the wave's tile over the K steps kp, kp + ks, ... of unit U.
template <int WT, int NW, int NTT>
__device__ inline void tile_compute(const GemmUnit &U, int rt, int kp, int ks,
                                    f32x4 (&acc)[NW][NTT]) {
  using Tr = WTraits<WT>;
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int row = rt * kTile + j;
  const bool row_ok = row < U.R;
  const char *wp[NW];
  wp[0] = static_cast<const char *>(U.w0) + (size_t)(row_ok ? row : 0) * U.ldw * Tr::W_BYTES;
  if constexpr (NW == 2)
    wp[1] = static_cast<const char *>(U.w1) + (size_t)(row_ok ? row : 0) * U.ldw * Tr::W_BYTES;
  const int ntt = min(NTT, (U.ntok + kTile - 1) / kTile);
  const bool split_in = NW == 2 && U.in1 != U.in0;
  const char *bp0[NTT];
  const char *bp1[NTT];
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    const int i = tt * kTile + j;
    const bool ok = tt < ntt && i < U.ntok;
    bp0[tt] = ok ? token_row(U.in0, U.idx, U.ldin, i, Tr::A_BYTES) : nullptr;
    bp1[tt] = ok && split_in ? token_row(U.in1, U.idx, U.ldin, i, Tr::A_BYTES) : nullptr;
  }
  const int nsteps = U.K / Tr::K_STEP;
  const int sblocks = U.K / 128;                   // fp8: scale blocks along K
  const int srow = (rt * kTile) / 128;             // fp8: scale block row of the tile
  for (int s = kp; s < nsteps; s += ks) {
    const int kel = s * Tr::K_STEP + g * (Tr::K_STEP / 4);
    u32x4 a[NW][Tr::W_VEC];
#pragma unroll
    for (int n = 0; n < NW; ++n)
#pragma unroll
      for (int v = 0; v < Tr::W_VEC; ++v)
        a[n][v] = row_ok ? load_stream16(wp[n] + (size_t)kel * Tr::W_BYTES + v * 16) : u32x4{0, 0, 0, 0};
    float sc[NW];
    if constexpr (WT == WT_FP8) {
      sc[0] = U.s0[srow * sblocks + s];
      if constexpr (NW == 2) sc[1] = U.s1[srow * sblocks + s];
    }
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt) {
      if (tt >= ntt) break;
      u32x4 b0[4], b1[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        b0[v] = bp0[tt] ? load16(bp0[tt] + (size_t)kel * Tr::A_BYTES + v * 16) : u32x4{0, 0, 0, 0};
        if (split_in)
          b1[v] = bp1[tt] ? load16(bp1[tt] + (size_t)kel * Tr::A_BYTES + v * 16) : u32x4{0, 0, 0, 0};
        else
          b1[v] = b0[v];
      }
#pragma unroll
      for (int n = 0; n < NW; ++n) {
        const u32x4 *b = (n == 1) ? b1 : b0;
        if constexpr (WT == WT_BF16) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            acc[n][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a[n][q]), as_bf16x8(b[q]),
                                                                 acc[n][tt], 0, 0, 0);
        } else if constexpr (WT == WT_FP8) {
          f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t lo = a[n][q >> 1][(q & 1) * 2], hi = a[n][q >> 1][(q & 1) * 2 + 1];
            t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(lo, hi), as_bf16x8(b[q]), t,
                                                        0, 0, 0);
          }
          acc[n][tt] += sc[n] * t;
        } else {
#pragma unroll
          for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[n][tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __uint_as_float(a[n][v][e]), __uint_as_float(b[v][e]), acc[n][tt], 0, 0, 0);
        }
      }
    }
  }
}

__device__ inline float apply_sigma(float v, int sigma) {
  return sigma == DEAMOE_SIGMA_NONE ? v : silu_f(v);
}

// Write the finished tile.  Lane l holds rows 4 * (l / 16) + r, r < 4, of
// the tile for token (l % 16) of each token tile.
template <int NW, int NTT>
__device__ inline void tile_epilogue(const GemmUnit &U, int rt, int sigma, const f32x4 (&acc)[NW][NTT]) {
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int row0 = rt * kTile + 4 * g;
  if (row0 >= U.R) return;
  const bool full = row0 + 3 < U.R;
  const int ntt = min(NTT, (U.ntok + kTile - 1) / kTile);
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    if (tt >= ntt) break;
    const int i = tt * kTile + j;
    if (i >= U.ntok) continue;
    float o0[4] = {0.f, 0.f, 0.f, 0.f}, o1[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v0 = acc[0][tt][r];
      const float v1 = NW == 2 ? acc[NW - 1][tt][r] : 0.f;
      switch (U.epi) {
        case EPI_SWIGLU: o0[r] = silu_f(v0) * v1; break;
        case EPI_SIGMA2: o0[r] = apply_sigma(v0, sigma); o1[r] = apply_sigma(v1, sigma); break;
        case EPI_SIGMA: o0[r] = apply_sigma(v0, sigma); break;
        default: o0[r] = v0; break;
      }
    }
    const int nout = U.epi == EPI_SIGMA2 ? 2 : 1;
    for (int q = 0; q < nout; ++q) {
      const float *o = q ? o1 : o0;
      void *base = q ? U.out1 : U.out0;
      if (U.out_f32) {
        float *p = static_cast<float *>(base) + (size_t)i * U.ldout + row0;
        if (full) {
          *reinterpret_cast<f32x4 *>(p) = f32x4{o[0], o[1], o[2], o[3]};
        } else {
          for (int r = 0; row0 + r < U.R; ++r) p[r] = o[r];
        }
      } else {
        uint16_t *p = static_cast<uint16_t *>(base) + (size_t)i * U.ldout + row0;
        if (full) {
          const uint32_t lo = f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
          const uint32_t hi = f32_to_bf16(o[2]) | ((uint32_t)f32_to_bf16(o[3]) << 16);
          *reinterpret_cast<u32x2 *>(p) = u32x2{lo, hi};
        } else {
          for (int r = 0; row0 + r < U.R; ++r) p[r] = f32_to_bf16(o[r]);
        }
      }
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
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int kp = wave % KS;
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
