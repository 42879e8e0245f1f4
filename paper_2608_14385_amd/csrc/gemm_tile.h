// Skinny grouped matrix product on gfx950 matrix cores.
//
// One wave computes a 16-row tile of one or two weight matrices (gate and up
// share the token operand) against up to 16 * NTT token rows, streaming the
// weights from HBM exactly once.
//
// Weight path per K step (WSEG bytes of each of the 16 rows): the rows are
// read with whole-row-segment loads (each instruction covers RPI rows x WSEG
// contiguous bytes, the pattern HBM streams fastest), staged through a
// wave-private, padded LDS region and read back in the matrix-core operand
// layout: lane (j = l % 16, g = l / 16) takes row j, and for product m the
// bytes of k-range [32m + 8g, 32m + 8g + 8) (bf16, fp8) or the four fp32 of
// [16m + 4g, 16m + 4g + 4).  The token operand uses the same K permutation,
// so every 16x16 product sums over the whole step.
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
  static constexpr int K_STEP = 64, W_BYTES = 4, A_BYTES = 4;
};
template <>
struct WTraits<WT_BF16> {
  static constexpr int K_STEP = 128, W_BYTES = 2, A_BYTES = 2;
};
template <>
struct WTraits<WT_FP8> {
  static constexpr int K_STEP = 128, W_BYTES = 1, A_BYTES = 2;
};

// Load geometry of one K step of a 16-row tile.
template <int WT>
struct WLoad {
  static constexpr int WSEG = WTraits<WT>::K_STEP * WTraits<WT>::W_BYTES;   // bytes per row
  static constexpr int LPR = WSEG / 16;      // lanes per row (16 B each)
  static constexpr int RPI = 64 / LPR;       // rows per load instruction
  static constexpr int NQ = kTile / RPI;     // load instructions per matrix
  static constexpr int RS = WSEG + 16;       // padded LDS row stride
  static constexpr int REGION = kTile * RS;  // LDS bytes per matrix per wave
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

// Global-address-space view of a pointer.  Pointers read from a unit table
// or an LDS copy of the arguments leave the compiler without the knowledge
// that they address global memory: accesses through them would become flat
// accesses, which also count as LDS operations, so every later LDS wait
// would wait for them too (a store's full round trip).
template <class T>
using gmem = __attribute__((address_space(1))) T;
template <class T>
__device__ inline gmem<T> *glob(T *p) {
  return reinterpret_cast<gmem<T> *>(reinterpret_cast<uintptr_t>(p));
}

// A unit of a stage table, read once per work item with scalar loads: the
// table is constant while a stage runs.  The tile loop and the epilogue then
// take every field from scalar registers; a field read through the table
// pointer would be a vector load, and a vector load issued after the weight
// prefetch can only be waited for together with it.
__device__ inline GemmUnit load_unit(const GemmUnit *p) {
  const auto *c = reinterpret_cast<const __attribute__((address_space(4))) GemmUnit *>(
      reinterpret_cast<uintptr_t>(p));
  GemmUnit u;
  u.w0 = c->w0; u.w1 = c->w1; u.s0 = c->s0; u.s1 = c->s1;
  u.in0 = c->in0; u.in1 = c->in1; u.idx = c->idx; u.out0 = c->out0; u.out1 = c->out1;
  u.R = c->R; u.K = c->K; u.ldw = c->ldw; u.ldin = c->ldin; u.ldout = c->ldout;
  u.ntok = c->ntok; u.tile_begin = c->tile_begin; u.epi = c->epi; u.out_f32 = c->out_f32;
  u.tpg = c->tpg;
  return u;
}

typedef __attribute__((address_space(1))) const u32x4 gvec;
typedef __attribute__((address_space(1))) const float gfloat;

__device__ inline const gvec *gptr(const void *p) {
  return reinterpret_cast<const gvec *>(reinterpret_cast<uintptr_t>(p));
}
__device__ inline const gfloat *gfptr(const float *p) {
  return reinterpret_cast<const gfloat *>(reinterpret_cast<uintptr_t>(p));
}

// Token-operand row of token i of a unit.
// idx is a generic pointer: the small-batch kernel keeps its token lists in
// LDS, the stage tables in global memory.
__device__ inline const char *token_row(const void *base, const int32_t *idx, int ldin, int i,
                                        int abytes) {
  const int row = idx ? idx[i] : i;
  return static_cast<const char *>(base) + (size_t)row * ldin * abytes;
}

// Byte offset, inside one K step of a token row, of the 16-byte token chunk
// that pairs with matrix-core product m (m < 4) of lane group g.
__device__ inline int b_chunk_offset(int g, int m) { return m * 64 + g * 16; }

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
      B[tt][q] = *gptr(bp0[tt] + boff + b_chunk_offset(g, q));
      if constexpr (SPLIT) B[tt][4 + q] = *gptr(bp1[tt] + boff + b_chunk_offset(g, q));
    }
  }
}

// The matrix-core products of one K step; a[n][m] is the operand of product
// m (fp8: the first two dwords hold its eight codes).
template <int WT, int NW, int NTT, bool SPLIT>
__device__ inline void step_mma(const u32x4 (&a)[NW][4], const u32x4 (&B)[NTT][SPLIT ? 8 : 4],
                                int ntt, const float (&sc)[NW], f32x4 (&acc)[NW][NTT]) {
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    if (tt > 0 && tt >= ntt) break;   // ntt >= 1
#pragma unroll
    for (int n = 0; n < NW; ++n) {
      const int bo = (SPLIT && n == 1) ? 4 : 0;
      if constexpr (WT == WT_BF16) {
#pragma unroll
        for (int m = 0; m < 4; ++m)
          acc[n][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a[n][m]),
                                                               as_bf16x8(B[tt][bo + m]), acc[n][tt],
                                                               0, 0, 0);
      } else if constexpr (WT == WT_FP8) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < 4; ++m)
          t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(a[n][m][0], a[n][m][1]),
                                                      as_bf16x8(B[tt][bo + m]), t, 0, 0, 0);
        acc[n][tt] += sc[n] * t;
      } else {
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[n][tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[n][m][e]),
                                                              __uint_as_float(B[tt][bo + m][e]),
                                                              acc[n][tt], 0, 0, 0);
      }
    }
  }
}

// Rows of one staged K step (as loaded: instruction q covers rows
// q * RPI + lane / LPR, 16 bytes each) written to the wave's LDS region and
// read back in the matrix-core operand layout.
template <int WT, int NW>
__device__ inline void stage_weights(char *lds, const u32x4 (&Gb)[NW][WLoad<WT>::NQ],
                                     u32x4 (&a)[NW][4]) {
  using LD = WLoad<WT>;
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int lrow = lane / LD::LPR, lchunk = lane % LD::LPR;
#pragma unroll
  for (int n = 0; n < NW; ++n)
#pragma unroll
    for (int q = 0; q < LD::NQ; ++q)
      *reinterpret_cast<u32x4 *>(lds + n * LD::REGION + (q * LD::RPI + lrow) * LD::RS +
                                 lchunk * 16) = Gb[n][q];
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int n = 0; n < NW; ++n)
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if constexpr (WT == WT_FP8) {
        const u32x2 v = *reinterpret_cast<const u32x2 *>(lds + n * LD::REGION + j * LD::RS +
                                                           m * 32 + g * 8);
        a[n][m] = u32x4{v[0], v[1], 0u, 0u};
      } else {
        a[n][m] = *reinterpret_cast<const u32x4 *>(lds + n * LD::REGION + j * LD::RS +
                                                      b_chunk_offset(g, m));
      }
    }
}

// Stream one work item: row tiles rt0 .. rt0 + nsub - 1 of unit U, each over
// the K steps kp, kp + ks, ... (nsub > 1 only when ks == 1).  PAIR: a tile is
// 32 rows of one matrix, streamed as two 16-row halves (w0 and w0 + 16 rows)
// that share the token operand; R is then a multiple of 32.  `lds` is this
// wave's private staging region (NW * WLoad<WT>::REGION bytes).
// Rows past R and tokens past ntok are clamped to valid ones: their products
// land only in output rows / columns that are never stored.
// Software pipeline: loads retire in issue order, so the weights and the
// token operand of one K step are requested together as one group, PF
// groups ahead of the step being multiplied; waiting for a group never
// waits for a later one.  Groups past the end read a cache-resident token
// row instead of weights, so every iteration issues the same loads.
// `done(rt, acc)` is called (and acc cleared) after the last K step of
// each tile when nsub > 1; with nsub == 1 the caller finishes the tile.
// B1: the token operand is requested with the step that uses it rather than
// PF steps ahead (one buffer instead of PF + 1), before that step's weight
// prefetch, so that waiting for it never waits for the prefetch; its L2
// round trip overlaps the weights of the step in flight.  This saves the
// registers of PF token-operand buffers.
template <int WT, int NW, int NTT, bool SPLIT, int PF, bool PAIR, bool NT, bool B1, class Done>
__device__ inline void tile_loop(const GemmUnit &U, int rt0, int nsub, int kp, int ks, int tok0,
                                 char *lds, f32x4 (&acc)[NW][NTT], Done done) {
  static_assert(!PAIR || (NW == 2 && !SPLIT), "a row pair is two tiles of one matrix");
  constexpr int TR = PAIR ? 2 * kTile : kTile;   // weight rows of a tile
  using Tr = WTraits<WT>;
  using LD = WLoad<WT>;
  constexpr int NB = PF + 1;
  constexpr int BV = SPLIT ? 8 : 4;
  constexpr int ASEG = Tr::K_STEP * Tr::A_BYTES;     // bytes of one token row per K step
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int R = uniform(U.R), ldw = uniform(U.ldw);
  const int nsteps = uniform(U.K / Tr::K_STEP);
  const int nloc = kp < nsteps ? (nsteps - kp + ks - 1) / ks : 0;   // K steps of this wave per tile
  const int total = nloc * nsub;
  if (total == 0) return;
  const int ntok = uniform(U.ntok) - tok0;   // tokens of this item: tok0 .. U.ntok - 1
  const int ntt = uniform(min(NTT, (ntok + kTile - 1) / kTile));
  const char *bp0[NTT];
  const char *bp1[NTT];
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    int i = tt * kTile + j;
    i = tok0 + (i < ntok ? i : 0);
    bp0[tt] = token_row(U.in0, U.idx, U.ldin, i, Tr::A_BYTES);
    bp1[tt] = SPLIT ? token_row(U.in1, U.idx, U.ldin, i, Tr::A_BYTES) : bp0[tt];
  }
  // ROWS: the token operand of two or more tiles is loaded like the weights,
  // as whole 256-byte row segments (instruction q of tile tt covers tokens
  // 4q + lane / 16, 16 bytes each), and transposed through this wave's LDS
  // region one tile at a time.  That touches half the cache lines per load
  // instruction of the operand layout's 16 rows x 64 bytes.  fp8 stages take
  // it with the operand requested per step (B1): their double-buffered
  // three-wave instantiations would spill the row offsets.
  constexpr bool ROWS = (WT == WT_BF16 || (WT == WT_FP8 && B1)) && !SPLIT && NTT >= 2;
  using LB = WLoad<WT_BF16>;   // token rows are bf16
  static_assert(!ROWS || (ASEG == LB::WSEG && LB::NQ == 4 && NW * LD::REGION >= LB::REGION),
                "a token tile is staged like one bf16 weight tile");
  // byte offsets from in0 of the rows this lane loads: below 2^32, as a stage
  // reads at most one row per (token, selected expert) pair, of at most
  // DEAMOE_MAX_WIDTH bf16 columns
  static_assert((int64_t)DEAMOE_MAX_TOKENS * DEAMOE_MAX_TOPK * DEAMOE_MAX_WIDTH * 2 <
                    (int64_t{1} << 32),
                "32-bit row offsets");
  uint32_t boffs[ROWS ? NTT : 1][4];
  if constexpr (ROWS) {
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int i = tt * kTile + q * LB::RPI + lane / LB::LPR;
        i = tok0 + (i < ntok ? i : 0);
        boffs[tt][q] = (uint32_t)(token_row(U.in0, U.idx, U.ldin, i, Tr::A_BYTES) -
                                  static_cast<const char *>(U.in0)) +
                       (lane % LB::LPR) * 16;
      }
  }
  // the token operand of K step kstep in the load layout (ROWS) or the operand layout
  auto load_tok = [&](u32x4(&Bb)[NTT][BV], int kstep) {
    if constexpr (ROWS) {
      const char *base = static_cast<const char *>(U.in0) + (size_t)kstep * ASEG;
#pragma unroll
      for (int tt = 0; tt < NTT; ++tt) {
        if (tt > 0 && tt >= ntt) break;   // ntt >= 1
#pragma unroll
        for (int q = 0; q < 4; ++q) Bb[tt][q] = *gptr(base + boffs[tt][q]);
      }
    } else {
      load_b<WT, NTT, SPLIT>(Bb, bp0, bp1, ntt, (size_t)kstep * ASEG, g);
    }
  };
  // load pattern: instruction q covers rows q * RPI + lane / LPR, 16 bytes each
  const int lrow = lane / LD::LPR, lchunk = lane % LD::LPR;
  const char *w0 = static_cast<const char *>(U.w0) + lchunk * 16;
  const char *w1 = PAIR ? w0 + (size_t)kTile * ldw * Tr::W_BYTES
                        : NW == 2 ? static_cast<const char *>(U.w1) + lchunk * 16 : w0;
  const int rmax = R - 1 - (PAIR ? kTile : 0);   // last row the first matrix may read
  const char *dummy = bp0[0] + (lane & 15) * 16;
  // fp8 block scales.  The scale rows of this item's tiles are read once, as a
  // window of 64 entries of the [R/128, K/128] table starting at the first
  // tile's scale row: lane l holds entry l.  A K step then takes its scale
  // with one lane read instead of a load.  The window covers the item: a
  // single tile lies in one scale row (TR divides 128) and K / 128 <= 64; a
  // multi-tile item spans at most 32768 / K rows with K <= 1024, at most
  // 2 + K / 64 <= 18 entries.
  const int sblocks = U.K / 128;
  float scw[NW];
  const int srow0 = (rt0 * TR) / 128;
  if constexpr (WT == WT_FP8) {
    const int base = srow0 * sblocks, nsc = ((R + 127) / 128) * sblocks;
    const int e = base + lane < nsc ? base + lane : base;
    scw[0] = gfptr(U.s0)[e];
    if constexpr (NW == 2) scw[1] = gfptr(PAIR ? U.s0 : U.s1)[e];
  }
  u32x4 G[NB][NW][LD::NQ];
  u32x4 B[B1 ? 1 : NB][NTT][BV];
  int SC[NB];   // fp8: window entry of the group's scales
  // K step of virtual step v (tile v / nloc, K step kp + (v % nloc) * ks)
  auto kstep_of = [&](int v) {
    const bool ok = v < total;
    const int sub = ok ? v / nloc : 0;
    return ok ? kp + (v - sub * nloc) * ks : 0;
  };
  // issue the weight loads (and, without B1, the token operand) of virtual step v
  auto issue = [&](u32x4(&Gb)[NW][LD::NQ], u32x4(&Bb)[NTT][BV], int &sc, int v) {
    const bool ok = v < total;
    const int sub = ok ? v / nloc : 0;
    const int kstep = kstep_of(v);
#pragma unroll
    for (int q = 0; q < LD::NQ; ++q) {
      const int row = min((rt0 + sub) * TR + q * LD::RPI + lrow, rmax);
      const size_t woff = (size_t)row * ldw * Tr::W_BYTES + (size_t)kstep * LD::WSEG;
#pragma unroll
      for (int n = 0; n < NW; ++n)
        Gb[n][q] = NT ? __builtin_nontemporal_load(gptr(ok ? (n ? w1 : w0) + woff : dummy))
                      : *gptr(ok ? (n ? w1 : w0) + woff : dummy);
    }
    if constexpr (!B1) load_tok(Bb, kstep);
    if constexpr (WT == WT_FP8)   // a row pair lies in one scale row
      sc = uniform((((rt0 + sub) * TR) / 128 - srow0) * sblocks + kstep);
  };
  auto stage = [&](const u32x4(&Gb)[NW][LD::NQ], u32x4(&a)[NW][4]) {
    stage_weights<WT, NW>(lds, Gb, a);
  };
#pragma unroll
  for (int p = 0; p < PF; ++p) issue(G[p], B[B1 ? 0 : p], SC[p], p);
  for (int v = 0;;) {
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int qn = (q + NB - 1) % NB;   // the buffer consumed one step ago
      if constexpr (B1) {
        load_tok(B[0], kstep_of(v));
        __builtin_amdgcn_sched_barrier(0);
      }
      issue(G[qn], B[B1 ? 0 : qn], SC[qn], v + PF);
      __builtin_amdgcn_sched_barrier(0);
      u32x4 a[NW][4];
      stage(G[q], a);
      if constexpr (ROWS) {   // after the weights' reads, in the same region
        u32x4(&Bq)[NTT][BV] = B[B1 ? 0 : q];
#pragma unroll
        for (int tt = 0; tt < NTT; ++tt) {
          if (tt > 0 && tt >= ntt) break;
          stage_weights<WT_BF16, 1>(lds, reinterpret_cast<const u32x4(&)[1][4]>(Bq[tt]),
                                    reinterpret_cast<u32x4(&)[1][4]>(Bq[tt]));
        }
      }
      float sc[NW];
      if constexpr (WT == WT_FP8) {
#pragma unroll
        for (int n = 0; n < NW; ++n)
          sc[n] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(scw[n]), SC[q]));
      }
      step_mma<WT, NW, NTT, SPLIT>(a, B[B1 ? 0 : q], ntt, sc, acc);
      __builtin_amdgcn_sched_barrier(0);
      ++v;
      if (nsub > 1 && v % nloc == 0) {   // a tile of a multi-tile work item is complete
        done(rt0 + v / nloc - 1, acc);
#pragma unroll
        for (int n = 0; n < NW; ++n)
#pragma unroll
          for (int tt = 0; tt < NTT; ++tt) acc[n][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
      if (v >= total) return;
    }
  }
}

// Four consecutive outputs (fp32 or bf16) at element offset off; `full`
// false writes only the first `left` of them.
__device__ inline void store4(void *base, int out_f32, size_t off, f32x4 o, bool full, int left) {
  if (out_f32) {
    gmem<float> *p = glob(static_cast<float *>(base)) + off;
    if (full) {
      *reinterpret_cast<gmem<f32x4> *>(p) = o;
    } else {
      for (int r = 0; r < left; ++r) p[r] = o[r];
    }
  } else {
    gmem<uint16_t> *p = glob(static_cast<uint16_t *>(base)) + off;
    if (full) {
      const uint32_t lo = f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
      const uint32_t hi = f32_to_bf16(o[2]) | ((uint32_t)f32_to_bf16(o[3]) << 16);
      *reinterpret_cast<gmem<u32x2> *>(p) = u32x2{lo, hi};
    } else {
      for (int r = 0; r < left; ++r) p[r] = f32_to_bf16(o[r]);
    }
  }
}

// Element-wise part of sigma.  RMSNorm needs the whole d-vector: its stages
// store the raw value and a row pass (rownorm_kernel, zsum_kernel) divides
// by the root mean square.
__device__ inline float apply_sigma(float v, int sigma) {
  return sigma == DEAMOE_SIGMA_SILU ? silu_f(v) : sigma == DEAMOE_SIGMA_GELU ? gelu_f(v) : v;
}

__device__ inline f32x4 sigma4(f32x4 v, int sigma) {
  return f32x4{apply_sigma(v[0], sigma), apply_sigma(v[1], sigma), apply_sigma(v[2], sigma),
               apply_sigma(v[3], sigma)};
}

// Write the finished tile.  Lane l holds rows 4 * (l / 16) + r, r < 4, of
// the tile for token (l % 16) of each token tile.  PAIR: the second
// accumulator holds the 16 rows after the first (same epilogue, one matrix).
template <int NW, int NTT, bool PAIR>
__device__ inline void tile_epilogue(const GemmUnit &U, int rt, int tok0, int sigma,
                                     const f32x4 (&acc)[NW][NTT]) {
  constexpr int TR = PAIR ? 2 * kTile : kTile;
  const int lane = lane_id();
  const int g = lane >> 4, j = lane & 15;
  const int R = uniform(U.R), ntok = uniform(U.ntok) - tok0, epi = uniform(U.epi);
  const int out_f32 = uniform(U.out_f32), ldout = uniform(U.ldout);
  const int row0 = rt * TR + 4 * g;
  if (row0 >= R) return;
  const bool full = row0 + 3 < R;
  const int ntt = uniform(min(NTT, (ntok + kTile - 1) / kTile));
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    if (tt > 0 && tt >= ntt) break;   // ntt >= 1
    const int i = tt * kTile + j;
    if (i >= ntok) continue;
    const size_t off = (size_t)(tok0 + i) * ldout + row0;
    const f32x4 v0 = acc[0][tt];
    if constexpr (PAIR) {
      const f32x4 v1 = acc[1][tt];
      const int row1 = row0 + kTile;
      store4(U.out0, out_f32, off, epi == EPI_SIGMA ? sigma4(v0, sigma) : v0, full, R - row0);
      if (row1 < R)
        store4(U.out0, out_f32, off + kTile, epi == EPI_SIGMA ? sigma4(v1, sigma) : v1,
               row1 + 3 < R, R - row1);
    } else if constexpr (NW == 2) {
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

// One workgroup of 4 waves: 4 / KS work items, each split over KS waves
// along K (interleaved K steps, partial tiles summed in a fixed order
// through LDS; work items of one tile), or with KS == 1 one work item of
// `tpg` tiles per wave.  A unit with more than 16 * NTT tokens has one work
// item per token group of 16 * NTT tokens and tile item; the items of one
// tile item are 8 * TPB apart, in workgroups on the same XCD.
// SPLIT: the two matrices read different token operands (in0 / in1).
// B1: the token operand is requested per step (see tile_loop), which lets
// stages with two token tiles fit three waves per SIMD.
template <int WT, int NW, int NTT, int KS, bool SPLIT = false, bool PAIR = false, bool B1 = false>
struct TileRunner {
  static constexpr int TR = PAIR ? 2 * kTile : kTile;   // weight rows of a tile
  static constexpr int TPB = 4 / KS;
  // load groups in flight per wave while one is multiplied
  static constexpr int PF = 1;
  static constexpr int STAGE_BYTES = NW * WLoad<WT>::REGION;   // per wave
  static constexpr int RED_BYTES = KS > 1 ? NW * NTT * kWave * 16 : 0;   // per wave
  static constexpr int WAVE_BYTES = STAGE_BYTES > RED_BYTES ? STAGE_BYTES : RED_BYTES;
  struct Smem {
    alignas(16) char buf[4][WAVE_BYTES];   // staging, then (KS > 1) partial tiles
  };

  // U: the unit in registers (load_unit for a table entry).
  __device__ __attribute__((always_inline)) static void run(Smem &sm, const GemmUnit *U, int item,
                                                            bool active, int sigma) {
    const int wave = uniform(threadIdx.x / kWave), lane = lane_id();
    const int kp = uniform(wave % KS);
    item = uniform(item);
    f32x4 acc[NW][NTT];
#pragma unroll
    for (int n = 0; n < NW; ++n)
#pragma unroll
      for (int tt = 0; tt < NTT; ++tt) acc[n][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
    int rt0 = 0, nsub = 1, tok0 = 0;
    if (active) {
      constexpr int GT = kTile * NTT;   // tokens of a group
      const int groups = (uniform(U->ntok) + GT - 1) / GT;
      const int tpg = KS == 1 ? uniform(U->tpg) : 1;
      const int ntiles = (uniform(U->R) + TR - 1) / TR;
      if (groups > 1) {
        // The token groups of one tile item stream the same weight rows.
        // Items S apart run in workgroups 8 apart, which the dispatcher puts
        // on the same XCD, so a tile's groups are numbered S apart (blocks of
        // S tile items, group-major inside a block; the last block holds the
        // r remaining tile items): the later groups' reads find the rows in
        // that XCD's L2.
        constexpr int S = 8 * TPB;
        const int nti = (ntiles + tpg - 1) / tpg;   // tile items of the unit
        const int full = nti / S;
        int g, ti;
        if (item < full * S * groups) {
          const int b = item / (S * groups), w = item - b * (S * groups);
          g = w / S;
          ti = b * S + (w - g * S);
        } else {
          const int r = nti - full * S, w = item - full * S * groups;
          g = w / r;
          ti = full * S + (w - g * r);
        }
        tok0 = uniform(g) * GT;
        item = uniform(ti);
      }
      rt0 = item * tpg;
      nsub = min(tpg, ntiles - rt0);
      auto done = [&](int rt, const f32x4 (&a)[NW][NTT]) {
        tile_epilogue<NW, NTT, PAIR>(*U, rt, tok0, sigma, a);
      };
      // A unit with several token groups streams its weight rows once per
      // group: those loads stay in the caches for the other groups (the
      // groups of a tile item run on one XCD at about the same time); every
      // other weight row is read once and streams past them.
      if (groups > 1)
        tile_loop<WT, NW, NTT, SPLIT, PF, PAIR, false, B1>(*U, rt0, nsub, kp, KS, tok0, sm.buf[wave],
                                                       acc, done);
      else
        tile_loop<WT, NW, NTT, SPLIT, PF, PAIR, true, B1>(*U, rt0, nsub, kp, KS, tok0, sm.buf[wave],
                                                      acc, done);
    }
    if constexpr (KS > 1) {
      f32x4 *red = reinterpret_cast<f32x4 *>(sm.buf[wave]);
      if (active && kp > 0) {
#pragma unroll
        for (int n = 0; n < NW; ++n)
#pragma unroll
          for (int tt = 0; tt < NTT; ++tt) red[(n * NTT + tt) * kWave + lane] = acc[n][tt];
      }
      __syncthreads();
      if (active && kp == 0) {
        for (int q = 1; q < KS; ++q) {
          const f32x4 *r = reinterpret_cast<const f32x4 *>(sm.buf[wave + q]);
#pragma unroll
          for (int n = 0; n < NW; ++n)
#pragma unroll
            for (int tt = 0; tt < NTT; ++tt) acc[n][tt] += r[(n * NTT + tt) * kWave + lane];
        }
      }
      __syncthreads();
    }
    if (active && kp == 0 && nsub == 1) tile_epilogue<NW, NTT, PAIR>(*U, rt0, tok0, sigma, acc);
  }
};

}  // namespace deamoe
