// Read-bandwidth probe for the benchmark: the practical streaming-read rate
// of the device, against which the expert stages' rates are read.  Every
// workgroup strides over the buffer with 16-byte non-temporal loads, eight in
// flight per lane; the loaded words are folded into a value that is stored
// only if it matches an impossible pattern, so the loads are kept.
// Not part of the DeaMoE library.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void read_probe_kernel(const u32x4 *__restrict__ p, size_t n16,
                                                         uint32_t *sink) {
  constexpr int U = 8;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(p + i);
    acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

}  // namespace

// Reads `bytes` (a multiple of 16) from the device buffer `buf` once on
// `stream` (a hipStream_t); `sink` is a device word the kernel may write.
// Returns 0, or a HIP error code.
extern "C" int deamoe_probe_read(const void *buf, size_t bytes, uint32_t *sink, int grid,
                                 void *stream) {
  if (!buf || !sink || bytes % 16 || grid <= 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(read_probe_kernel, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const u32x4 *>(buf), bytes / 16, sink);
  return (int)hipGetLastError();
}
