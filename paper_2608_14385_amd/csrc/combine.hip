// Weighted combine (Eq. 3) and, for the FACTORED form, the collection of the
// experts' Z rows per (department, token) before the department's down
// projection (Sec. 3.2).
#include "launch.h"

namespace deamoe {

// y[t, c] = sum over the token's slots, in slot order, of w * partial[pair, c];
// rounded once to the output type.  One thread per 4 consecutive columns;
// the slots are taken in batches whose loads are all issued before the
// batch is summed (selects, not branches, so that they are not serialized).
__global__ __launch_bounds__(64) void combine_kernel(CombineArgs a) {
  constexpr int U = 8;
  const int t = blockIdx.y;
  const int c = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (c >= a.h) return;
  const int ns = a.nslot[t];
  const int32_t *sp = a.slot_pair + (size_t)t * a.max_slots;
  const float *sw = a.slot_w + (size_t)t * a.max_slots;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < ns; s0 += U) {
    f32x4 v[U];
    float w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = min(s0 + u, ns - 1);
      w[u] = sw[s];
      v[u] = *reinterpret_cast<const f32x4 *>(a.partial + (size_t)sp[s] * a.h + c);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const f32x4 nx = acc + w[u] * v[u];
      acc = s0 + u < ns ? nx : acc;
    }
  }
  if (a.act_f32) {
    *reinterpret_cast<f32x4 *>(static_cast<float *>(a.y) + (size_t)t * a.h + c) = acc;
  } else {
    const uint32_t lo = f32_to_bf16(acc[0]) | ((uint32_t)f32_to_bf16(acc[1]) << 16);
    const uint32_t hi = f32_to_bf16(acc[2]) | ((uint32_t)f32_to_bf16(acc[3]) << 16);
    *reinterpret_cast<u32x2 *>(static_cast<uint16_t *>(a.y) + (size_t)t * a.h + c) = u32x2{lo, hi};
  }
}

hipError_t launch_combine(const CombineArgs &a, hipStream_t s) {
  dim3 grid((a.h / 4 + 63) / 64, a.T);
  hipLaunchKernelGGL(combine_kernel, grid, dim3(64), 0, s, a);
  return hipGetLastError();
}

// Zs[q] = sum over the token's experts i in department j (rank order) of
// p_i * Z[(i, t)], for the department pair q = (j, t).  One workgroup per
// department pair (pairs past the step's count return at once): the pair's
// experts and weights go to LDS first, then each thread sums 4 columns with
// all of a batch's loads issued before it is summed.
__global__ __launch_bounds__(256) void zsum_kernel(ZsumArgs a) {
  constexpr int U = 4;
  __shared__ int32_t s_pair[DEAMOE_MAX_TOPK];
  __shared__ float s_w[DEAMOE_MAX_TOPK];
  __shared__ int32_t s_n;
  const int q = blockIdx.x;
  if (q >= a.counts->n_dept_pairs) return;
  const int j = a.pair_dept[q], t = a.dept_tokens[q];
  if (threadIdx.x < 64) {   // wave 0 gathers the token's experts of department j in rank order
    const int r = threadIdx.x;
    const bool in = r < a.k && a.topk_ids[t * a.k + r] / a.E == j;
    const uint64_t m = __ballot(in);
    if (in) {
      const int pos = __popcll(m & ((1ull << r) - 1ull));
      s_pair[pos] = a.tok_exp_pair[t * a.k + r];
      s_w[pos] = a.topk_w[t * a.k + r];
    }
    if (r == 0) s_n = __popcll(m);
  }
  __syncthreads();
  const int n = s_n;
  for (int c = threadIdx.x * 4; c < a.d; c += blockDim.x * 4) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < n; s0 += U) {
      f32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        v[u] = *reinterpret_cast<const f32x4 *>(a.z + (size_t)s_pair[min(s0 + u, n - 1)] * a.d + c);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const f32x4 nx = acc + s_w[min(s0 + u, n - 1)] * v[u];
        acc = s0 + u < n ? nx : acc;
      }
    }
    if (a.act_f32) {
      *reinterpret_cast<f32x4 *>(static_cast<float *>(a.zs) + (size_t)q * a.d + c) = acc;
    } else {
      const uint32_t lo = f32_to_bf16(acc[0]) | ((uint32_t)f32_to_bf16(acc[1]) << 16);
      const uint32_t hi = f32_to_bf16(acc[2]) | ((uint32_t)f32_to_bf16(acc[3]) << 16);
      *reinterpret_cast<u32x2 *>(static_cast<uint16_t *>(a.zs) + (size_t)q * a.d + c) =
          u32x2{lo, hi};
    }
  }
}

hipError_t launch_zsum(const ZsumArgs &a, int max_dept_pairs, hipStream_t s) {
  hipLaunchKernelGGL(zsum_kernel, dim3(max_dept_pairs > 0 ? max_dept_pairs : 1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace deamoe
