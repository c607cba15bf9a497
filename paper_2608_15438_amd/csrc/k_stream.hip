// Bandwidth self-check: one streaming pass over a device buffer with the same
// 16-byte vector loads the refinement issues, xor-folded so the loads are
// not removed.  Gives the achievable read rate on the running device.
#include "nr_internal.h"

namespace nr {

__global__ void __launch_bounds__(256) k_stream_read(const uint4 *p, int64_t n16, uint32_t *sink) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t acc = 0;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    uint4 a = p[i], b = p[i + stride], c = p[i + 2 * stride], d = p[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    uint4 a = p[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;  // practically never taken
}

hipError_t launch_stream_read(const void *buf, int64_t bytes, uint32_t *sink, int n_cu,
                              hipStream_t s) {
  hipLaunchKernelGGL(k_stream_read, dim3(n_cu * 8), dim3(256), 0, s, (const uint4 *)buf,
                     bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace nr
