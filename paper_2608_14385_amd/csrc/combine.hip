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
// department pair; pairs past the step's count return at once.
__global__ __launch_bounds__(256) void zsum_kernel(ZsumArgs a) {
  const int q = blockIdx.x;
  if (q >= a.counts->n_dept_pairs) return;
  int lo = 0, hi = a.m - 1;   // department of pair q: last j with offset[j] <= q
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.dept_offset[mid] <= q) lo = mid; else hi = mid - 1;
  }
  const int j = lo, t = a.dept_tokens[q];
  for (int c = threadIdx.x; c < a.d; c += blockDim.x) {
    float acc = 0.f;
    for (int r = 0; r < a.k; ++r) {
      const int e = a.topk_ids[t * a.k + r];
      if (e / a.E != j) continue;
      acc += a.topk_w[t * a.k + r] * a.z[(size_t)a.tok_exp_pair[t * a.k + r] * a.d + c];
    }
    if (a.act_f32)
      static_cast<float *>(a.zs)[(size_t)q * a.d + c] = acc;
    else
      static_cast<uint16_t *>(a.zs)[(size_t)q * a.d + c] = f32_to_bf16(acc);
  }
}

hipError_t launch_zsum(const ZsumArgs &a, int max_dept_pairs, hipStream_t s) {
  hipLaunchKernelGGL(zsum_kernel, dim3(max_dept_pairs > 0 ? max_dept_pairs : 1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace deamoe
