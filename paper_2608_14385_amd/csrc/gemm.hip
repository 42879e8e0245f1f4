// Grouped skinny GEMM over a device-built list of units (one launch per
// stage).  The number of units and row tiles is only known on the device, so
// the grid is fixed on the host and every workgroup walks tiles
// blockIdx.x * TPB, + gridDim.x * TPB, ...; tiles past the end do nothing.
#include "gemm_tile.h"
#include "launch.h"

namespace deamoe {

constexpr int kMaxUnitsCached = 4096;

template <int WT, int NW, int NTT, int KS, bool SPLIT, bool PAIR>
__device__ __attribute__((always_inline)) void grouped_gemm_body(const GemmStage &st) {
  using Run = TileRunner<WT, NW, NTT, KS, SPLIT, PAIR>;
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
    const GemmUnit *U = st.units + u;
    Run::run(sm, U, active ? tile - uniform(s_begin[u]) : 0, active, st.sigma);
  }
}

template <int WT, int NW, int NTT, int KS, bool SPLIT, bool PAIR>
__global__ __launch_bounds__(256) void grouped_gemm_kernel(GemmStage st) {
  grouped_gemm_body<WT, NW, NTT, KS, SPLIT, PAIR>(st);
}

// The same at three waves per SIMD (at most 168 registers).  Left alone the
// compiler gives two-matrix stages with split token operands (the FACTORED
// private gate/up) 166 registers, two waves per SIMD; with one token tile,
// three (no spills) keep the 640 workgroups of a one-token step resident in
// one round.
template <int WT, int NW, int NTT, int KS, bool SPLIT, bool PAIR>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
void grouped_gemm_occ3_kernel(GemmStage st) {
  grouped_gemm_body<WT, NW, NTT, KS, SPLIT, PAIR>(st);
}

// fp8 stages with two token tiles also fit three waves without spilling
// (bf16 ones would spill, which costs far more than the occupancy gains).
template <int WT, int NTT>
constexpr bool occ3_two_tiles() { return NTT == 2 && WT == WT_FP8; }

// mode: GemmMode; row pairs exist for NTT <= 2 only (the host picks them so)
template <int WT, int NW, int NTT, int KS>
static hipError_t launch_gemm(const GemmStage &st, int mode, int max_tiles, int grid_cap,
                              hipStream_t s) {
  constexpr int TPB = 4 / KS;
  int grid = (max_tiles + TPB - 1) / TPB;
  grid = grid < 1 ? 1 : (grid > grid_cap ? grid_cap : grid);
  if constexpr (NW == 2) {
    if (mode == 1) {
      if constexpr (NTT == 1 && KS > 1)
        hipLaunchKernelGGL((grouped_gemm_occ3_kernel<WT, NW, NTT, KS, true, false>), dim3(grid),
                           dim3(256), 0, s, st);
      else   // two token tiles (or no K split) would spill at three waves per SIMD
        hipLaunchKernelGGL((grouped_gemm_kernel<WT, NW, NTT, KS, true, false>), dim3(grid),
                           dim3(256), 0, s, st);
      return hipGetLastError();
    }
    if (mode == 2) {
      if constexpr (NTT <= 2) {   // row pairs are built for up to two token tiles
        if constexpr (occ3_two_tiles<WT, NTT>())
          hipLaunchKernelGGL((grouped_gemm_occ3_kernel<WT, NW, NTT, KS, false, true>), dim3(grid),
                             dim3(256), 0, s, st);
        else
          hipLaunchKernelGGL((grouped_gemm_kernel<WT, NW, NTT, KS, false, true>), dim3(grid),
                             dim3(256), 0, s, st);
        return hipGetLastError();
      }
      return hipErrorInvalidValue;
    }
  }
  if constexpr (NW == 2 && occ3_two_tiles<WT, NTT>())
    hipLaunchKernelGGL((grouped_gemm_occ3_kernel<WT, NW, NTT, KS, false, false>), dim3(grid),
                       dim3(256), 0, s, st);
  else
    hipLaunchKernelGGL((grouped_gemm_kernel<WT, NW, NTT, KS, false, false>), dim3(grid),
                       dim3(256), 0, s, st);
  return hipGetLastError();
}

// Token tiles per wave: 1 or 2 (larger token sets are split into groups).
template <int WT, int NW, int KS>
static hipError_t dispatch_ntt(const GemmStage &st, int mode, int ntt, int max_tiles, int cap,
                               hipStream_t s) {
  switch (ntt) {
    case 1: return launch_gemm<WT, NW, 1, KS>(st, mode, max_tiles, cap, s);
    case 2: return launch_gemm<WT, NW, 2, KS>(st, mode, max_tiles, cap, s);
    default: return hipErrorInvalidValue;
  }
}

template <int WT, int NW>
static hipError_t dispatch_ks(const GemmStage &st, int mode, int ntt, int ks, int max_tiles,
                              int cap, hipStream_t s) {
  switch (ks) {
    case 1: return dispatch_ntt<WT, NW, 1>(st, mode, ntt, max_tiles, cap, s);
    case 2: return dispatch_ntt<WT, NW, 2>(st, mode, ntt, max_tiles, cap, s);
    default: return dispatch_ntt<WT, NW, 4>(st, mode, ntt, max_tiles, cap, s);
  }
}

hipError_t launch_grouped_gemm(const GemmStage &st, int wtype, int nw, int mode, int ntt,
                               int ks, int max_tiles, int grid_cap, hipStream_t s) {
  if (nw != 2) return hipErrorInvalidValue;   // every stage streams two matrices or a row pair
  switch (wtype) {
    case WT_F32: return dispatch_ks<WT_F32, 2>(st, mode, ntt, ks, max_tiles, grid_cap, s);
    case WT_BF16: return dispatch_ks<WT_BF16, 2>(st, mode, ntt, ks, max_tiles, grid_cap, s);
    default: return dispatch_ks<WT_FP8, 2>(st, mode, ntt, ks, max_tiles, grid_cap, s);
  }
}

}  // namespace deamoe
