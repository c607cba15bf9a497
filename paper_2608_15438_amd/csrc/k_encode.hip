// Step 1: encoder forward pass (Sec. 3.2.1; architecture Sec. 4.5, App. A),
// one launch per linear layer.  Each layer is a dense contraction
//   out[m][n] = act( in_scale * sum_k in[m][k] * W[n][k] + bias[n] )
// on the fp32 matrix cores (v_mfma_f32_16x16x4f32).  A 256-thread block owns a
// BM x BN output tile and each of its four waves a (BM/2) x (BN/2) quarter, as
// (BM/32) x (BN/32) blocks of 16 x 16.  K is staged through LDS BK at a time in
// two buffers (the next tile is read into registers while the current one is
// multiplied; one barrier per tile); uint8 inputs are widened while staging,
// and rows whose length is a multiple of 4 are read 4 elements per load.
// Every output is one MFMA chain over k in increasing order, 4 at a time,
// whatever the tile shape, so the logits do not depend on it.
// Hidden layers fold eval-mode BatchNorm (per-channel scale and shift) and
// ReLU into the epilogue; the last layer writes the logits.
#include "nr_internal.h"

namespace nr {

typedef float v4f __attribute__((ext_vector_type(4)));


// element (m, kg) of the input, zero outside [0, M) x [0, K)
__device__ __forceinline__ float enc_load_in(const EncodeLayerArgs &a, int64_t m, int kg) {
  if (m >= a.M || kg >= a.K) return 0.f;
  return a.in_u8 ? (float)((const uint8_t *)a.in)[m * a.K + kg]
                 : ((const float *)a.in)[m * a.K + kg];
}

// elements (m, kg .. kg+3) of the input (K a multiple of 4, so the four are
// all inside or all past the row)
__device__ __forceinline__ float4 enc_load_in4(const EncodeLayerArgs &a, int64_t m, int kg) {
  if (m >= a.M || kg >= a.K) return make_float4(0.f, 0.f, 0.f, 0.f);
  if (a.in_u8) {
    const uint32_t v = *reinterpret_cast<const uint32_t *>((const uint8_t *)a.in + m * a.K + kg);
    return make_float4((float)(v & 0xffu), (float)((v >> 8) & 0xffu), (float)((v >> 16) & 0xffu),
                       (float)(v >> 24));
  }
  return *reinterpret_cast<const float4 *>((const float *)a.in + m * a.K + kg);
}

__device__ __forceinline__ float4 enc_load_w4(const EncodeLayerArgs &a, int n, int kg) {
  if (n >= a.N || kg >= a.K) return make_float4(0.f, 0.f, 0.f, 0.f);
  return *reinterpret_cast<const float4 *>(a.W + (int64_t)n * a.K + kg);
}

template <int BM, int BN, int BK, bool VEC>
__global__ void __launch_bounds__(256) k_encode_layer(EncodeLayerArgs a) {
  constexpr int MI = BM / 32, NJ = BN / 32;  // 16 x 16 blocks per wave
  constexpr int VW = VEC ? 4 : 1;            // elements per load
  constexpr int LA = BM * BK / VW, LW = BN * BK / VW;  // loads per tile
  constexpr int PA = (LA + 255) / 256, PW = (LW + 255) / 256;  // per thread (at most)
  static_assert(BK % 4 == 0 && BM % 32 == 0 && BN % 32 == 0, "whole MFMA blocks");
  // two K-tiles of A (activations) and W, each [BK][B* + 4]
  __shared__ float As[2][BK][BM + 4];
  __shared__ float Ws[2][BK][BN + 4];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  // tile of this block: the column tiles of one row tile are consecutive
  // blocks on the same XCD (blocks go to XCDs in turn, block id mod 8), so
  // they share that XCD's L2 copy of the row tile's inputs
  const int64_t nb = (a.N + BN - 1) / BN;
  const int64_t t8 = (int64_t)(blockIdx.x >> 3);
  const int64_t u = (t8 / nb) * 8 + (blockIdx.x & 7);
  if (u * BM >= a.M) return;  // a slot past the last row tile
  const int64_t m0 = u * BM;
  const int n0 = (int)(t8 % nb) * BN;
  const int wm = (wave & 1) * (BM / 2), wn = (wave >> 1) * (BN / 2);
  const int K = a.K, N = a.N;
  v4f acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  // load e of a tile: row e / (BK / VW), elements VW * (e % (BK / VW)) onwards
  // (consecutive threads read consecutive elements of a row)
  float ra[PA][VW], rw[PW][VW];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int u = 0; u < PA; ++u) {
      const int e = tid + 256 * u;
      const int r = e / (BK / VW), kk = VW * (e % (BK / VW));
      if (LA % 256 != 0 && e >= LA) continue;
      if constexpr (VEC) {
        const float4 v = enc_load_in4(a, m0 + r, k0 + kk);
        ra[u][0] = v.x;
        ra[u][VW > 1 ? 1 : 0] = v.y;
        ra[u][VW > 2 ? 2 : 0] = v.z;
        ra[u][VW > 3 ? 3 : 0] = v.w;
      } else {
        ra[u][0] = enc_load_in(a, m0 + r, k0 + kk);
      }
    }
#pragma unroll
    for (int u = 0; u < PW; ++u) {
      const int e = tid + 256 * u;
      const int r = e / (BK / VW), kk = VW * (e % (BK / VW));
      if (LW % 256 != 0 && e >= LW) continue;
      if constexpr (VEC) {
        const float4 v = enc_load_w4(a, n0 + r, k0 + kk);
        rw[u][0] = v.x;
        rw[u][VW > 1 ? 1 : 0] = v.y;
        rw[u][VW > 2 ? 2 : 0] = v.z;
        rw[u][VW > 3 ? 3 : 0] = v.w;
      } else {
        const int n = n0 + r, kg = k0 + kk;
        rw[u][0] = (n < N && kg < K) ? a.W[(int64_t)n * K + kg] : 0.f;
      }
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < PA; ++u) {
      const int e = tid + 256 * u;
      const int r = e / (BK / VW), kk = VW * (e % (BK / VW));
      if (LA % 256 != 0 && e >= LA) continue;
#pragma unroll
      for (int v = 0; v < VW; ++v) As[buf][kk + v][r] = ra[u][v];
    }
#pragma unroll
    for (int u = 0; u < PW; ++u) {
      const int e = tid + 256 * u;
      const int r = e / (BK / VW), kk = VW * (e % (BK / VW));
      if (LW % 256 != 0 && e >= LW) continue;
#pragma unroll
      for (int v = 0; v < VW; ++v) Ws[buf][kk + v][r] = rw[u][v];
    }
  };
  fetch(0);
  stash(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = 0; k0 < K; k0 += BK) {
    const bool more = k0 + BK < K;
    if (more) fetch(k0 + BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      // A operand of a 16x16x4 block: lane l holds row l % 16, k l / 16
      const int kr = kk + (lane >> 4), c = lane & 15;
      float av[MI], bv[NJ];
#pragma unroll
      for (int i = 0; i < MI; ++i) av[i] = As[buf][kr][wm + 16 * i + c];
#pragma unroll
      for (int j = 0; j < NJ; ++j) bv[j] = Ws[buf][kr][wn + 16 * j + c];
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (more) stash(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  const int64_t M = a.M;
  // D layout of a 16x16 block: lane l, register r -> row 4*(l/16) + r, column l%16
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
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

template <int BM, int BN, int BK>
static hipError_t launch_tile(const EncodeLayerArgs &a, hipStream_t s) {
  // row tiles in groups of 8 (one per XCD), each with all its column tiles
  const int64_t nm = (a.M + BM - 1) / BM, nn = (a.N + BN - 1) / BN;
  const dim3 grid((unsigned)(((nm + 7) / 8) * 8 * nn));
  // four-element loads need rows (and so every row start) 4-element aligned
  const bool vec = a.K % 4 == 0 && (reinterpret_cast<uintptr_t>(a.in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(a.W) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL((k_encode_layer<BM, BN, BK, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_encode_layer<BM, BN, BK, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

// Tile shapes measured on MI355X (10,000 queries): 64 x 64 where that still
// gives the chip about four blocks per CU (the 1536 -> 512 layer: 196 us for
// the whole 1536-d encoder, 255 us with 64 x 64 x 32 tiles and one load per
// element), 32 x 64 for smaller layers (128 -> 256: the 1B encoder in 22 us
// against 29 us with 64 x 64), 32 x 32 for the code layer (at most 32 outputs)
hipError_t launch_encode_layer(const EncodeLayerArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.N <= 32) return launch_tile<32, 32, 16>(a, s);
  const int64_t tiles64 = ((a.M + 63) / 64) * ((a.N + 63) / 64);
  if (tiles64 >= 1024) return launch_tile<64, 64, 16>(a, s);
  return launch_tile<32, 64, 16>(a, s);
}

}  // namespace nr
