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
  if (a.rms) {   // RMSNorm sigma: fold 1 / rms of each Z row into its weight
    const int wv = threadIdx.x / 64, lane = threadIdx.x % 64;
    for (int s = wv; s < n; s += blockDim.x / 64) {
      const float *zr = a.z + (size_t)s_pair[s] * a.d;
      float ss = 0.f;
      for (int c = lane * 4; c < a.d; c += 256) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(zr + c);
        ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
      if (lane == 0) s_w[s] = s_w[s] / sqrtf(ss / (float)a.d + kRmsEps);
    }
    __syncthreads();
  }
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

// One workgroup per department pair (pairs past the step's count return at
// once): the sum of squares of the pair's g and u rows, then both rows
// rescaled in place.
__global__ __launch_bounds__(256) void rownorm_kernel(RowNormArgs a) {
  __shared__ float s_part[2][4];
  const int q = blockIdx.x;
  if (q >= a.counts->n_dept_pairs) return;
  const int wv = threadIdx.x / 64, lane = threadIdx.x % 64;
  const size_t base = (size_t)q * a.d;
  auto at = [&](const void *p, int c) {
    return a.act_f32 ? static_cast<const float *>(p)[base + c]
                     : bf16_to_f32(static_cast<const uint16_t *>(p)[base + c]);
  };
  float sg = 0.f, su = 0.f;
  for (int c = threadIdx.x; c < a.d; c += blockDim.x) {
    const float g = at(a.g, c), u = at(a.u, c);
    sg += g * g;
    su += u * u;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    sg += __shfl_xor(sg, off);
    su += __shfl_xor(su, off);
  }
  if (lane == 0) {
    s_part[0][wv] = sg;
    s_part[1][wv] = su;
  }
  __syncthreads();
  float tg = 0.f, tu = 0.f;
  for (int w = 0; w < (int)blockDim.x / 64; ++w) {
    tg += s_part[0][w];
    tu += s_part[1][w];
  }
  const float ig = 1.0f / sqrtf(tg / (float)a.d + kRmsEps);
  const float iu = 1.0f / sqrtf(tu / (float)a.d + kRmsEps);
  for (int c = threadIdx.x; c < a.d; c += blockDim.x) {
    const float g = at(a.g, c) * ig, u = at(a.u, c) * iu;
    if (a.act_f32) {
      static_cast<float *>(a.g)[base + c] = g;
      static_cast<float *>(a.u)[base + c] = u;
    } else {
      static_cast<uint16_t *>(a.g)[base + c] = f32_to_bf16(g);
      static_cast<uint16_t *>(a.u)[base + c] = f32_to_bf16(u);
    }
  }
}

hipError_t launch_rownorm(const RowNormArgs &a, int max_dept_pairs, hipStream_t s) {
  hipLaunchKernelGGL(rownorm_kernel, dim3(max_dept_pairs > 0 ? max_dept_pairs : 1), dim3(256), 0,
                     s, a);
  return hipGetLastError();
}

hipError_t launch_zsum(const ZsumArgs &a, int max_dept_pairs, hipStream_t s) {
  hipLaunchKernelGGL(zsum_kernel, dim3(max_dept_pairs > 0 ? max_dept_pairs : 1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace deamoe
