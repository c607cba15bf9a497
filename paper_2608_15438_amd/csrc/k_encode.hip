// Step 1: encoder forward pass (Sec. 3.2.1; architecture Sec. 4.5, App. A),
// one launch per linear layer.  Each layer is a dense contraction
//   out[m][n] = act( in_scale * sum_k in[m][k] * W[n][k] + bias[n] )
// on the fp32 matrix cores (v_mfma_f32_16x16x4f32).  A 256-thread block owns a
// 64 x 64 output tile, each wave a 32 x 32 quarter (2 x 2 MFMA blocks); K is
// staged through LDS 32 at a time in two buffers (the next tile is read into
// registers while the current one is multiplied; one barrier per tile), uint8
// inputs are widened while staging.
// Hidden layers fold eval-mode BatchNorm (per-channel scale and shift) and
// ReLU into the epilogue; the last layer writes the logits.
#include "nr_internal.h"

namespace nr {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int EB_M = 64, EB_N = 64, EB_K = 32;
constexpr int EB_LD = EB_M + 4;                      // LDS row stride (floats)
constexpr int EB_PER = EB_M * EB_K / 256;            // tile elements staged per thread

// element e of a K-tile: row e / EB_K, column e % EB_K (consecutive threads
// read consecutive columns of a row)
__device__ __forceinline__ float enc_load_in(const EncodeLayerArgs &a, int64_t m, int kg) {
  if (m >= a.M || kg >= a.K) return 0.f;
  return a.in_u8 ? (float)((const uint8_t *)a.in)[m * a.K + kg]
                 : ((const float *)a.in)[m * a.K + kg];
}

__global__ void __launch_bounds__(256) k_encode_layer(EncodeLayerArgs a) {
  // two K-tiles of A (activations) and W, each [EB_K][EB_LD]: the next tile
  // is loaded into registers while the current one feeds the matrix cores
  __shared__ float As[2][EB_K][EB_LD];
  __shared__ float Ws[2][EB_K][EB_LD];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * EB_M;
  const int n0 = blockIdx.y * EB_N;
  const int wm = (wave & 1) * 32, wn = (wave >> 1) * 32;
  const int K = a.K, N = a.N;
  v4f acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  float ra[EB_PER], rw[EB_PER];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int u = 0; u < EB_PER; ++u) {
      const int e = tid + 256 * u;
      const int r = e / EB_K, kk = e % EB_K;
      ra[u] = enc_load_in(a, m0 + r, k0 + kk);
      const int n = n0 + r, kg = k0 + kk;
      rw[u] = (n < N && kg < K) ? a.W[(int64_t)n * K + kg] : 0.f;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < EB_PER; ++u) {
      const int e = tid + 256 * u;
      const int r = e / EB_K, kk = e % EB_K;
      As[buf][kk][r] = ra[u];
      Ws[buf][kk][r] = rw[u];
    }
  };
  fetch(0);
  stash(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = 0; k0 < K; k0 += EB_K) {
    const bool more = k0 + EB_K < K;
    if (more) fetch(k0 + EB_K);
#pragma unroll
    for (int kk = 0; kk < EB_K; kk += 4) {
      const int kr = kk + (lane >> 4), c = lane & 15;
      float av[2], bv[2];
      av[0] = As[buf][kr][wm + c];
      av[1] = As[buf][kr][wm + 16 + c];
      bv[0] = Ws[buf][kr][wn + c];
      bv[1] = Ws[buf][kr][wn + 16 + c];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (more) stash(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  const int64_t M = a.M;
  // D layout of a 16x16 block: lane l, register r -> row 4*(l/16) + r, column l%16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn + 16 * j + (lane & 15);
      if (n >= N) continue;
      const float bias = a.bias ? a.bias[n] : 0.f;
      const float sc = a.bn_scale ? a.bn_scale[n] : 1.f;
      const float sh = a.bn_shift ? a.bn_shift[n] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm + 16 * i + 4 * (lane >> 4) + r;
        if (m >= M) continue;
        float v = acc[i][j][r] * a.in_scale + bias;
        if (a.relu) {
          v = v * sc + sh;
          v = v > 0.f ? v : 0.f;
        }
        a.out[m * N + n] = v;
      }
    }
}

hipError_t launch_encode_layer(const EncodeLayerArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  dim3 grid((unsigned)((a.M + EB_M - 1) / EB_M), (unsigned)((a.N + EB_N - 1) / EB_N));
  hipLaunchKernelGGL(k_encode_layer, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace nr
