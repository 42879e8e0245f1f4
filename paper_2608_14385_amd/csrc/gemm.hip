// Grouped skinny GEMM over a device-built list of units (one launch per
// stage).  The number of units and row tiles is only known on the device, so
// the grid is fixed on the host and every workgroup walks tiles
// blockIdx.x * TPB, + gridDim.x * TPB, ...; tiles past the end do nothing.
#include "gemm_tile.h"
#include "launch.h"

namespace deamoe {

constexpr int kMaxUnitsCached = 4096;

template <int WT, int NW, int NTT, int KS, bool SPLIT, bool PAIR, bool B1>
__device__ __attribute__((always_inline)) void grouped_gemm_body(const GemmStage &st) {
  using Run = TileRunner<WT, NW, NTT, KS, SPLIT, PAIR, B1>;
  __shared__ typename Run::Smem sm;
  __shared__ int32_t s_begin[kMaxUnitsCached];
  const int n_units = st.counts[0], n_tiles = st.counts[1];
  if (blockIdx.x * Run::TPB >= n_tiles) return;   // the grid is sized for the most work a step can have
  for (int u = threadIdx.x; u < n_units; u += blockDim.x) s_begin[u] = st.units[u].tile_begin;
  __syncthreads();
  const int wave = uniform(threadIdx.x / kWave);
  for (int base = blockIdx.x * Run::TPB; base < n_tiles; base += gridDim.x * Run::TPB) {
    const int tile = base + wave / KS;
    const bool active = tile < n_tiles;
    int u = 0;
    if (active) {  // last unit whose first tile is <= tile
      int lo = 0, hi = n_units - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (uniform(s_begin[mid]) <= tile) lo = mid; else hi = mid - 1;
      }
      u = lo;
    }
    u = uniform(u);
    const GemmUnit U = load_unit(st.units + u);
    Run::run(sm, &U, active ? tile - uniform(s_begin[u]) : 0, active, st.sigma);
  }
}

template <int WT, int NW, int NTT, int KS, bool SPLIT, bool PAIR>
__global__ __launch_bounds__(256) void grouped_gemm_kernel(GemmStage st) {
  grouped_gemm_body<WT, NW, NTT, KS, SPLIT, PAIR, false>(st);
}

// The same at three waves per SIMD (at most 168 registers), for the
// instantiations that fit them without spilling:
//  - the split-operand stage with one token tile (the FACTORED private
//    gate/up), its two token operands requested per step (B1): 138
//    registers, where both operands double-buffered took 166 at two waves
//    per SIMD, or 168 and a 24-byte spill at three.  Same-process A/B
//    against the latter (outputs bit-identical): 745.6 -> 704.4 us per step
//    at 16 tokens on the DeepSeek-V3 FACTORED layer (the stage 405.0 ->
//    364.3), 2071.8 -> 1977.4 at 64, 148.4 -> 145.3 at one token; Kimi-K2
//    879.6 -> 839.6, DeepSeek-V2 406.2 -> 391.6, Qwen3 330.8 -> 319.5 at 16;
//  - fp8 stages with two token tiles: with the token operand requested per
//    step (B1) and loaded as whole row segments for row pairs and for gate/up
//    pairs with a K split over 2 waves (above 32 tokens; same-process A/B at
//    the DeepSeek-V3 shape, us per step: 477.6 -> 458.4 at 64 tokens, 631.0
//    -> 569.1 at 128), double-buffered at 17-32 tokens (348.5 -> 351.4 at 24
//    with B1);
//  - bf16 and fp32 stages with two token tiles whose token operand is
//    requested per step (B1): row pairs (same-process A/B at the DeepSeek-V3
//    shape, down stage at 128 tokens 378.3 -> 370.0 us, skewed 178.9 ->
//    172.8), and gate/up pairs of layers narrower than 4096 (the 7B-class
//    layer 48.5 -> 44.9 us at 32 tokens, 52.3 -> 48.5 at 64; at the
//    DeepSeek-V3 shape they were 0-2 % slower, so two waves stay there).
template <int WT, int NW, int NTT, int KS, bool SPLIT, bool PAIR, bool B1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
void grouped_gemm_occ3_kernel(GemmStage st) {
  grouped_gemm_body<WT, NW, NTT, KS, SPLIT, PAIR, B1>(st);
}

// Four token tiles per wave (64 tokens), for the gate/up stage of wide
// layers above 64 tokens (fp8: above 96) and the bf16 down stage's row pairs
// there: a unit with many tokens streams its rows once per 64 tokens instead
// of once per 32.  The token operand is requested per step (B1);
// two waves per SIMD.
template <int WT, int NW, int NTT, int KS, bool PAIR>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
void grouped_gemm_wide_kernel(GemmStage st) {
  grouped_gemm_body<WT, NW, NTT, KS, false, PAIR, true>(st);
}

// mode: GemmMode; row pairs exist for NTT <= 2 only (the host picks them so).
// narrow: two-token-tile gate/up pairs run at three waves per SIMD.
template <int WT, int NW, int NTT, int KS>
static hipError_t launch_gemm(const GemmStage &st, int mode, int max_tiles, int grid_cap,
                              bool narrow, hipStream_t s) {
  constexpr int TPB = 4 / KS;
  int grid = (max_tiles + TPB - 1) / TPB;
  grid = grid < 1 ? 1 : (grid > grid_cap ? grid_cap : grid);
  constexpr bool FP8 = WT == WT_FP8;
  auto plain = [&](auto k) {
    hipLaunchKernelGGL(k, dim3(grid), dim3(256), 0, s, st);
    return hipGetLastError();
  };
  if constexpr (NTT == 4) {   // four tiles: gate/up with a two-wave K split, row pairs without
    if constexpr (KS == 2) {
      if (mode == GEMM_PLAIN) return plain(grouped_gemm_wide_kernel<WT, NW, NTT, KS, false>);
    } else if constexpr (KS == 1 && WT != WT_FP8) {
      if (mode == GEMM_PAIR) return plain(grouped_gemm_wide_kernel<WT, NW, NTT, KS, true>);
    }
    return hipErrorInvalidValue;
  }
  if constexpr (NW == 2) {
    if (mode == GEMM_SPLIT) {
      if constexpr (NTT == 1)
        return plain(grouped_gemm_occ3_kernel<WT, NW, NTT, KS, true, false, true>);
      else   // two token tiles would spill at three waves per SIMD (no stage uses them)
        return plain(grouped_gemm_kernel<WT, NW, NTT, KS, true, false>);
    }
    if (mode == GEMM_PAIR) {
      if constexpr (NTT == 2)
        return plain(grouped_gemm_occ3_kernel<WT, NW, NTT, KS, false, true, true>);
      else if constexpr (NTT == 1)
        return plain(grouped_gemm_kernel<WT, NW, NTT, KS, false, true>);
      return hipErrorInvalidValue;   // row pairs are built for up to two token tiles
    }
    if constexpr (NTT == 2 && KS > 1) {
      if constexpr (FP8)
        return plain(grouped_gemm_occ3_kernel<WT, NW, NTT, KS, false, false, KS == 2>);
      else if (narrow)
        return plain(grouped_gemm_occ3_kernel<WT, NW, NTT, KS, false, false, true>);
    }
  }
  return plain(grouped_gemm_kernel<WT, NW, NTT, KS, false, false>);
}

// Token tiles per wave: 1, 2, or 4 with a K split over 2 waves (larger
// token sets are split into groups).
template <int WT, int NW, int KS>
static hipError_t dispatch_ntt(const GemmStage &st, int mode, int ntt, int max_tiles, int cap,
                               bool narrow, hipStream_t s) {
  switch (ntt) {
    case 1: return launch_gemm<WT, NW, 1, KS>(st, mode, max_tiles, cap, narrow, s);
    case 2: return launch_gemm<WT, NW, 2, KS>(st, mode, max_tiles, cap, narrow, s);
    case 4:   // gate/up with a K split over 2 waves, row pairs without one
      if constexpr (KS <= 2) return launch_gemm<WT, NW, 4, KS>(st, mode, max_tiles, cap, narrow, s);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <int WT, int NW>
static hipError_t dispatch_ks(const GemmStage &st, int mode, int ntt, int ks, int max_tiles,
                              int cap, bool narrow, hipStream_t s) {
  switch (ks) {
    case 1: return dispatch_ntt<WT, NW, 1>(st, mode, ntt, max_tiles, cap, narrow, s);
    case 2: return dispatch_ntt<WT, NW, 2>(st, mode, ntt, max_tiles, cap, narrow, s);
    default: return dispatch_ntt<WT, NW, 4>(st, mode, ntt, max_tiles, cap, narrow, s);
  }
}

hipError_t launch_grouped_gemm(const GemmStage &st, int wtype, int nw, int mode, int ntt,
                               int ks, int max_tiles, int grid_cap, hipStream_t s, bool narrow) {
  if (nw != 2) return hipErrorInvalidValue;   // every stage streams two matrices or a row pair
  switch (wtype) {
    case WT_F32: return dispatch_ks<WT_F32, 2>(st, mode, ntt, ks, max_tiles, grid_cap, narrow, s);
    case WT_BF16: return dispatch_ks<WT_BF16, 2>(st, mode, ntt, ks, max_tiles, grid_cap, narrow, s);
    default: return dispatch_ks<WT_FP8, 2>(st, mode, ntt, ks, max_tiles, grid_cap, narrow, s);
  }
}

}  // namespace deamoe
