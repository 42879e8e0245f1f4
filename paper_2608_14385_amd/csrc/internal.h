// Internal types and device helpers of libdeamoe (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/deamoe.h"

namespace deamoe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kTile = 16;   // MFMA tile edge: 16 weight rows x 16 tokens

// Epilogue of one grouped-GEMM unit.
enum Epilogue : int32_t {
  EPI_SWIGLU = 0,   // out0 = SiLU(acc0) * acc1                       (two matrices)
  EPI_SIGMA2 = 1,   // out0 = sigma(acc0), out1 = sigma(acc1)          (two matrices)
  EPI_SIGMA = 2,    // out0 = sigma(acc0)                              (one matrix)
  EPI_STORE = 3,    // out0 = acc0                                     (one matrix)
};

// One weight matrix (or gate/up pair) applied to a group of token rows.
// A work item is `tpg` consecutive 16-row tiles of the unit.
// Row r of the weights is at w + r * ldw (elements of the weight type).  The
// B operand row of token i is at in + idx[i] * ldin (idx == NULL: row i).
// Output row of token i is at out + i * ldout (act type or fp32).
struct GemmUnit {
  const void *w0, *w1;
  const float *s0, *s1;     // fp8: block scales of this matrix, [ceil(R/128), K/128]
  const void *in0, *in1;
  const int32_t *idx;
  void *out0, *out1;
  int32_t R, K, ldw, ldin, ldout, ntok;
  int32_t tile_begin;       // exclusive prefix of work items over the units of a stage
  int32_t epi;              // Epilogue
  int32_t out_f32;          // 1: outputs are fp32, 0: act dtype
  int32_t tpg;              // row tiles per work item (1 unless the K split is 1)
};

// One unit of the fused down projection and combine (at most 32 tokens): the
// [R, K] down matrix w (fp8: block scales s) applied to
// the unit's gate/up outputs `in` ([members, K], one row per member token in
// ascending token order), each token's product weighted by pw[t].  The K
// steps of all units form one concatenation.
struct ChainUnit {
  const void *w;
  const float *s;
  const void *in;
  const float *pw;          // routing weight of token t at pw[t] (members only)
  int32_t K;
  uint32_t mask;            // member tokens, bit t
  int32_t step0;            // first K step of the unit in the concatenation
  int32_t pad_;
};

struct GemmStage {
  const GemmUnit *units;
  const int32_t *counts;    // [0] = number of units, [1] = number of row tiles
  int32_t sigma;            // DEAMOE_SIGMA_*
};

// Device-side plan written by the route kernel and consumed by the later ones.
constexpr int kMaxStages = 4;
struct PlanCounts {
  int32_t stage[kMaxStages][2];  // units, tiles per stage
  int32_t n_dept_pairs, n_exp_pairs, n_pairs, pad_;
};

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round-to-nearest-even fp32 -> bf16 (finite inputs).
__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffff) ? 0x40 : 0));
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float silu_f(float v) { return v / (1.0f + __expf(-v)); }
// GeLU in its exact form v * Phi(v) = v / 2 * (1 + erf(v / sqrt 2)).
__device__ inline float gelu_f(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }
// RMSNorm form of sigma: v / sqrt(mean(v^2) + kRmsEps) over a d-vector, unit gain.
constexpr float kRmsEps = 1e-6f;

__device__ inline int lane_id() { return __lane_id(); }

// Streaming 16-byte load that should not displace reusable lines in the caches.
__device__ inline u32x4 load_stream16(const void *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
__device__ inline u32x4 load16(const void *p) { return *reinterpret_cast<const u32x4 *>(p); }

}  // namespace deamoe
