// Router (Eq. 2), department bookkeeping (Sec. 3.2) and the device-side plan
// of the expert stages.
//
// router_kernel: the logits W_r x as a grouped skinny product, split over KC
//   chunks of the hidden dimension so that the n x h router matrix is read by
//   many workgroups; each chunk's partial logits go to part[c][t][e] (rows
//   padded to 64 * NS values).
// route_token_kernel: one wave per token: logits = sum of the KC partials in
//   chunk order (+ bias, one fp32 add), optional group-limited department
//   choice, top-k by (logit desc, id asc), the routing weights, and the
//   token's distinct departments with P_{t,j}.
// plan_kernel: one workgroup: per-department and per-expert token lists in
//   ascending token order (no atomics on any order-sensitive value), the
//   unit tables of every expert stage (pointers, row-tile prefix), the
//   combine slots of every token, and the counts.
// route_plan_kernel: both of the above in one workgroup for batches of up
//   to four tokens, the per-token results passed on through LDS.
#include "route_dev.h"

namespace deamoe {

// --------------------------------------------------------------- router GEMV

template <int WT, int NTT>
__global__ __launch_bounds__(256) void router_kernel(RouterArgs a) {
  using Run = TileRunner<WT, 1, NTT, 4>;
  __shared__ typename Run::Smem sm;
  using Tr = WTraits<WT>;
  const int rt = blockIdx.x % a.tiles, c = blockIdx.x / a.tiles;
  GemmUnit U = {};
  U.w0 = static_cast<const char *>(a.w) + (size_t)c * a.kchunk * Tr::W_BYTES;
  U.in0 = U.in1 = static_cast<const char *>(a.x) + (size_t)c * a.kchunk * Tr::A_BYTES;
  U.idx = nullptr;
  U.out0 = a.part + (size_t)c * a.T * a.ldp;
  U.R = a.n;
  U.K = a.kchunk;
  U.ldw = a.h;
  U.ldin = a.h;
  U.ldout = a.ldp;
  U.ntok = a.T;
  U.epi = EPI_STORE;
  U.out_f32 = 1;
  U.tpg = 1;
  Run::run(sm, &U, rt, true, DEAMOE_SIGMA_NONE);
}

template <int WT>
static hipError_t router_ntt(const RouterArgs &a, int ntt, int kc, hipStream_t s) {
  dim3 grid(a.tiles * kc);
  switch (ntt) {
    case 1: hipLaunchKernelGGL((router_kernel<WT, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((router_kernel<WT, 2>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((router_kernel<WT, 4>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((router_kernel<WT, 8>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_router(const RouterArgs &a, int wtype, int ntt, int kc, hipStream_t s) {
  return wtype == WT_F32 ? router_ntt<WT_F32>(a, ntt, kc, s) : router_ntt<WT_BF16>(a, ntt, kc, s);
}

template <int NS>
__global__ __launch_bounds__(64) void route_token_kernel(RouteArgs a) {
  __shared__ TokSmem sm;
  route_one<NS>(a, blockIdx.x, threadIdx.x, sm);
}

template <int BT>
__global__ __launch_bounds__(BT) void plan_kernel(RouteArgs a) {
  __shared__ PlanSmem sm;
  __shared__ RouteArgs sa;
  args_to_lds<BT>(a, sa);
  lds_barrier();
  plan_body<BT>(sa, sm);
}

// Batches of at most kFusedMaxT tokens (and no more than the workgroup has
// waves) route and plan in one workgroup: wave t routes token t and leaves
// its results in LDS as well, and the plan starts after a barrier that waits
// for LDS only (the results' global stores complete in the background).
// Larger batches route in a workgroup per token, which spreads the routing
// over as many CUs.  Wider routers (more experts per lane) take fewer waves
// for the plan, which leaves each wave more registers.  Same-process A/B of
// one workgroup against the two kernels, us per step: the DeepSeek-V3 shape
// 358.4 -> 357.0 at 6 tokens and 410.9 -> 409.8 at 8; fp8 182.1 -> 180.7 at
// 5; the 7B-class layer 72.2 -> 70.9 and Qwen3 209.6 -> 208.4 at 8; routers
// of 16 experts per lane even.
constexpr int kFusedMaxT = 8;
template <int NS>
constexpr int fused_waves() { return NS <= 4 ? 16 : NS <= 16 ? 8 : 4; }

template <int NS>
__global__ __launch_bounds__(fused_waves<NS>() * 64) void route_plan_kernel(RouteArgs a) {
  __shared__ TokSmem tsm[fused_waves<NS>()];
  __shared__ PlanSmem psm;
  __shared__ RouteArgs sa;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  args_to_lds<fused_waves<NS>() * 64>(a, sa);
  if (w < a.T) route_one<NS>(a, w, lane, tsm[w], PlanIn{psm.ids, psm.dep, psm.nd, nullptr});
  lds_barrier();
  plan_body<fused_waves<NS>() * 64, true>(sa, psm);
}

template <int NS>
static hipError_t launch_route_ns(const RouteArgs &a, hipStream_t s) {
  if (a.T <= kFusedMaxT && a.T <= fused_waves<NS>()) {
    hipLaunchKernelGGL((route_plan_kernel<NS>), dim3(1), dim3(fused_waves<NS>() * 64), 0, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((route_token_kernel<NS>), dim3(a.T), dim3(64), 0, s, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((plan_kernel<1024>), dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_route(const RouteArgs &a, hipStream_t s) {
  switch (route_ns(a.n)) {
    case 1: return launch_route_ns<1>(a, s);
    case 2: return launch_route_ns<2>(a, s);
    case 4: return launch_route_ns<4>(a, s);
    case 8: return launch_route_ns<8>(a, s);
    case 16: return launch_route_ns<16>(a, s);
    default: return launch_route_ns<32>(a, s);
  }
}

}  // namespace deamoe
