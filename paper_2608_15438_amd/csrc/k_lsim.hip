// Encoder training with the selective similarity loss L_sim (Sec. 3.2.2, the
// loss of Eq. "similarityconfig" with the dual-threshold mask of Eq. 8) for a
// mini-batch of B rows: inputs x [B x E] (scaled as the encoder sees them)
// and latents l [B x L], rho = sqrt(L / E),
//   S_emb(i, j) = ||x_i - x_j||,   S_lat(i, j) = ||l_i - l_j||,
//   m(i, j) = [i != j and (S_emb <= tau_emb or S_lat <= gamma rho tau_emb)],
//   L_sim = sum m (S_lat - gamma rho S_emb)^2 / sum m.
//
// k_pair_sqdist: all B x B squared input distances, |x_i|^2 + |x_j|^2 -
// 2 x_i . x_j with the dot products on the fp32 matrix cores
// (v_mfma_f32_16x16x4f32, one 64 x 64 tile per 256-thread block, E staged
// through LDS 16 at a time).  The rows are centred on the batch mean first
// (distances do not change), which keeps the norms, and so the cancellation
// in the expansion, small.
//
// k_lsim_grad: one pass over the pairs that yields the loss's numerator and
// mask count and the gradient with respect to the latents.  The mask is a
// constant of the step (as in the paper's formulation, the thresholds select
// pairs) and the distances are symmetric, so for row i
//   dL/dl_i = (1 / sum m) sum_j 4 m_ij d_ij (l_i - l_j) / S_lat(i, j),
// d_ij = S_lat(i, j) - gamma rho S_emb(i, j); the kernel writes the sum
// without the 1 / sum m factor.  Latent distances are taken directly from the
// coordinate differences (L <= 32).  One wave owns a row (a 4096-row batch
// spreads over 1024 blocks of four rows): its lanes take the columns in turn
// against 64-column tiles of latents staged in LDS, then the wave adds its
// lanes' partial gradients in a fixed butterfly order, so the gradient is the
// same bit for bit on every run.  Only the numerator's block sums meet in a
// double-precision atomic (its last bits may vary; the mask count is exact).
#include "nr_internal.h"

namespace nr {

typedef float v4f_l __attribute__((ext_vector_type(4)));

constexpr int LS_M = 64, LS_K = 16;

// column sums of x over blocks of LS_ROWS rows (partial[blk][c]), then the
// column means (the partials added in block order) and the squared norm of
// every centred row
constexpr int LS_ROWS = 256;

__global__ void k_col_partial(const float *x, int64_t B, int D, float *partial) {
  const int64_t r0 = (int64_t)blockIdx.x * LS_ROWS;
  const int64_t r1 = r0 + LS_ROWS < B ? r0 + LS_ROWS : B;
  for (int c = threadIdx.x; c < D; c += blockDim.x) {
    float s = 0.0f;
    for (int64_t i = r0; i < r1; ++i) s += x[i * D + c];
    partial[(int64_t)blockIdx.x * D + c] = s;
  }
}

__global__ void k_col_mean(const float *partial, int64_t nblk, int64_t B, int D, float *mean) {
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < D; c += gridDim.x * blockDim.x) {
    double s = 0.0;
    for (int64_t b = 0; b < nblk; ++b) s += partial[b * D + c];
    mean[c] = (float)(s / (double)B);
  }
}

__global__ void k_row_norms(const float *x, int64_t B, int D, const float *mean, float *norm) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < B;
       i += (int64_t)gridDim.x * blockDim.x) {
    float s = 0.0f;
    for (int c = 0; c < D; ++c) {
      const float v = x[i * D + c] - mean[c];
      s = fmaf(v, v, s);
    }
    norm[i] = s;
  }
}

__global__ void __launch_bounds__(256) k_pair_sqdist(const float *x, int64_t B, int D,
                                                      const float *mean, const float *norm,
                                                      float *out) {
  __shared__ float As[LS_K][LS_M + 4];
  __shared__ float Bs[LS_K][LS_M + 4];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  // tiles on and above the diagonal; each writes its mirror too, so the
  // matrix is symmetric bit for bit
  if (blockIdx.y < blockIdx.x) return;
  const int64_t i0 = (int64_t)blockIdx.x * LS_M, j0 = (int64_t)blockIdx.y * LS_M;
  const int wm = (wave & 1) * 32, wn = (wave >> 1) * 32;
  v4f_l acc[2][2];
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f_l{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < D; k0 += LS_K) {
    for (int e = tid; e < LS_M * LS_K; e += 256) {
      const int mm = e / LS_K, kk = e % LS_K, kg = k0 + kk;
      const int64_t ri = i0 + mm, rj = j0 + mm;
      As[kk][mm] = (ri < B && kg < D) ? x[ri * D + kg] - mean[kg] : 0.f;
      Bs[kk][mm] = (rj < B && kg < D) ? x[rj * D + kg] - mean[kg] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < LS_K; kk += 4) {
      const int kr = kk + (lane >> 4), c = lane & 15;
      float av[2], bv[2];
      av[0] = As[kr][wm + c];
      av[1] = As[kr][wm + 16 + c];
      bv[0] = Bs[kr][wn + c];
      bv[1] = Bs[kr][wn + 16 + c];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  // D layout of a 16x16 block: lane l, register r -> row 4*(l/16) + r, column l%16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t cj = j0 + wn + 16 * j + (lane & 15);
      if (cj >= B) continue;
      const float nj = norm[cj];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t ri = i0 + wm + 16 * i + 4 * (lane >> 4) + r;
        if (ri >= B) continue;
        float v = (norm[ri] + nj) - 2.0f * acc[i][j][r];
        v = v > 0.f ? v : 0.f;
        if (ri == cj) v = 0.f;
        out[ri * B + cj] = v;
        out[cj * B + ri] = v;
      }
    }
}

constexpr int LG_COLS = 64, LG_LMAX = 32, LG_WAVES = 4;

__global__ void __launch_bounds__(256) k_lsim_grad(const float *d2, const float *lat, int64_t B,
                                                    int L, float gr, float tau, double *num_cnt,
                                                    float *grad) {
  __shared__ float lj_s[LG_COLS][LG_LMAX + 1];
  __shared__ double red[2][LG_WAVES];
  const int tid = threadIdx.x;
  const int lane = tid & (WAVE - 1), w = tid / WAVE;
  const int64_t i = (int64_t)blockIdx.x * LG_WAVES + w;
  const bool row_ok = i < B;
  float li[LG_LMAX], g[LG_LMAX];
#pragma unroll
  for (int c = 0; c < LG_LMAX; ++c) {
    li[c] = (row_ok && c < L) ? lat[i * L + c] : 0.f;
    g[c] = 0.f;
  }
  const float lat_thr = gr * tau;
  double num = 0.0, cnt = 0.0;
  for (int64_t j0 = 0; j0 < B; j0 += LG_COLS) {
    __syncthreads();
    // the tile's latents: LG_COLS consecutive rows, read as one contiguous run
    for (int e = tid; e < LG_COLS * L; e += 256) {
      const int jj = e / L, c = e - jj * L;
      lj_s[jj][c] = j0 + jj < B ? lat[j0 * L + e] : 0.f;
    }
    __syncthreads();
    const int64_t j = j0 + lane;
    if (!row_ok || j >= B || j == i) continue;
    float sl2 = 0.f;
#pragma unroll
    for (int c = 0; c < LG_LMAX; ++c) {
      if (c < L) {
        const float t = li[c] - lj_s[lane][c];
        sl2 = fmaf(t, t, sl2);
      }
    }
    const float sl = sqrtf(sl2);
    const float se = sqrtf(d2[i * B + j]);
    const bool m = se <= tau || sl <= lat_thr;
    if (!m) continue;
    const float dd = sl - gr * se;
    num += (double)dd * (double)dd;
    cnt += 1.0;
    // the pairs (i, j) and (j, i) contribute alike
    const float coef = 4.0f * dd;
    if (coef != 0.f && sl > 0.f) {
      const float s = coef / sl;
#pragma unroll
      for (int c = 0; c < LG_LMAX; ++c)
        if (c < L) g[c] = fmaf(s, li[c] - lj_s[lane][c], g[c]);
    }
  }
  // the row's gradient: the lanes' partial sums added by a butterfly (the same
  // operations in the same order on every run; every lane ends with the total)
#pragma unroll
  for (int c = 0; c < LG_LMAX; ++c) {
    if (c < L) {
      float v = g[c];
      for (int m = 1; m < WAVE; m <<= 1) v += __shfl_xor(v, m);
      g[c] = v;
    }
  }
  if (row_ok && lane == 0)
    for (int c = 0; c < L; ++c) grad[i * L + c] = g[c];
  for (int m = 1; m < WAVE; m <<= 1) {
    num += __shfl_xor(num, m);
    cnt += __shfl_xor(cnt, m);
  }
  if (lane == 0) {
    red[0][w] = num;
    red[1][w] = cnt;
  }
  __syncthreads();
  if (tid == 0) {
    double tn = 0.0, tc = 0.0;
    for (int k = 0; k < LG_WAVES; ++k) {
      tn += red[0][k];
      tc += red[1][k];
    }
    atomicAdd(&num_cnt[0], tn);
    atomicAdd(&num_cnt[1], tc);
  }
}

size_t pair_sqdist_ws_floats(int64_t B, int D) {
  return (size_t)((B + LS_ROWS - 1) / LS_ROWS + 1) * (size_t)D + (size_t)B;
}

hipError_t launch_pair_sqdist(const float *x, int64_t B, int D, float *ws, float *out,
                              hipStream_t s) {
  if (B <= 0) return hipSuccess;
  const int64_t nblk = (B + LS_ROWS - 1) / LS_ROWS;
  float *partial = ws, *mean = ws + nblk * D, *norm = mean + D;
  hipLaunchKernelGGL(k_col_partial, dim3((unsigned)nblk), dim3(128), 0, s, x, B, D, partial);
  hipLaunchKernelGGL(k_col_mean, dim3((unsigned)((D + 127) / 128)), dim3(128), 0, s, partial, nblk,
                     B, D, mean);
  hipLaunchKernelGGL(k_row_norms, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, x, B, D,
                     mean, norm);
  const unsigned gb = (unsigned)((B + LS_M - 1) / LS_M);
  hipLaunchKernelGGL(k_pair_sqdist, dim3(gb, gb), dim3(256), 0, s, x, B, D, mean, norm, out);
  return hipGetLastError();
}

hipError_t launch_lsim_grad(const float *d2, const float *lat, int64_t B, int L, float gr,
                            float tau, double *num_cnt, float *grad, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipError_t e = launch_fill_i32((int32_t *)num_cnt, 4, 0, s);
  if (e != hipSuccess) return e;
  // one wave per row: every row's gradient is written once, by its wave
  const int64_t nb = (B + LG_WAVES - 1) / LG_WAVES;
  hipLaunchKernelGGL(k_lsim_grad, dim3((unsigned)nb), dim3(256), 0, s, d2, lat, B, L, gr, tau,
                     num_cnt, grad);
  return hipGetLastError();
}

}  // namespace nr
