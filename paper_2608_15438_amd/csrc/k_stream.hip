// Bandwidth self-check: one streaming pass over a device buffer, xor-folded
// so the loads are not removed.  Each wave reads 8 KB runs (lane l loads the
// 16-byte chunks l, l + 64, ..., l + 448 of the run: eight non-temporal loads
// in flight per lane), the waves taking the runs in turn, so at any time the
// chip reads one contiguous region.  Gives the achievable read rate on the
// running device.
#include "nr_internal.h"

namespace nr {

typedef unsigned int sr_u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) k_stream_read(const uint4 *p, int64_t n16, uint32_t *sink) {
  constexpr int RUN = 8 * WAVE;  // 16-byte chunks per run (8 KB)
  const int lane = threadIdx.x & (WAVE - 1);
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE;
  const int64_t nw = (int64_t)gridDim.x * (blockDim.x / WAVE);
  const int64_t nruns = n16 / RUN;
  const sr_u32x4 *q = reinterpret_cast<const sr_u32x4 *>(p);
  uint32_t acc = 0;
  for (int64_t r = wave; r < nruns; r += nw) {
    sr_u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(q + r * RUN + u * WAVE + lane);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (int64_t i = nruns * RUN + wave * WAVE + lane; i < n16; i += nw * WAVE) {
    const uint4 a = p[i];
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
