// Calibration of the search knobs (Sec. 3.4 "Calibration"), one wavefront per
// calibration query with its top-K target rows:
//   * the bucket score of every target: the score Algorithm 1 gives the
//     target's bucket, with the enumeration's own arithmetic (deviations
//     delta_j = |l_j - tau_j|, dimensions ranked by (delta, dim), the fp32 sum
//     of the flipped deviations added in rank order), or +inf when the bucket
//     is out of the enumeration's reach (a flipped dimension outside the
//     l_sel least stable ones, or more than r_max flips) -- the input of the
//     bucket-score cutoff S_max ("Bucket-score cutoff");
//   * the gating-margin point ("Centroid gating margin"): x = the smallest
//     centroid distance over every centroid of the buckets that hold the
//     targets, y = the distance of the farthest target's cluster minus x, in
//     the search's squared latent distance (acc = fmaf(t, t, acc) over the
//     dimensions in order, as the centroid stage computes it).
// The quantile fits of S_max and M(x) over these arrays are host work.
#include "nr_internal.h"

namespace nr {

__global__ void k_inverse_perm(const int64_t *row_ids, int64_t n, uint32_t *row_of_id) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n; r += stride) {
    const int64_t id = row_ids[r];
    if (id >= 0 && id < n) row_of_id[id] = (uint32_t)r;
  }
}

hipError_t launch_inverse_perm(const int64_t *row_ids, int64_t n, uint32_t *row_of_id,
                               hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_inverse_perm, dim3((unsigned)blocks), dim3(256), 0, s, row_ids, n,
                     row_of_id);
  return hipGetLastError();
}

// last index i in [0, len) with a[i] <= key (a non-decreasing, a[0] <= key)
template <class T>
__device__ __forceinline__ int64_t last_le(const T *a, int64_t len, uint64_t key) {
  int64_t lo = 0, hi = len;  // a[lo] <= key < a[hi] (a[len] taken as +inf)
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) >> 1;
    if ((uint64_t)a[mid] <= key) lo = mid; else hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(64) k_calib(CalibArgs a) {
  __shared__ int s_rank[32];      // rank of dimension j
  __shared__ float s_dlt[32];     // deviation of the dimension of rank r
  const int lane = lane_id();
  const int64_t q = blockIdx.x;
  if (q >= a.nq) return;
  const int b = a.b;
  const float lg = lane < b ? a.logits[q * b + lane] : 0.0f;
  const float t = lane < b ? a.tau[lane] : 0.0f;
  const uint32_t code0 = (uint32_t)ballot(lane < b && lg >= t);
  const float dl = lane < b ? fabsf(lg - t) : INFINITY;
  int rank = 0;
  for (int i = 0; i < b; ++i) {
    const float di = __shfl(dl, i);
    rank += (di < dl) || (di == dl && i < lane);
  }
  if (lane < b) {
    s_rank[lane] = rank;
    s_dlt[rank] = dl;
  }
  __syncthreads();

  // lane i: target i (K <= 64)
  const int K = a.K;
  const int64_t id = lane < K ? a.targets[q * K + lane] : -1;
  const bool has = id >= 0 && id < a.n;
  int64_t clus = -1;
  uint32_t code = 0;
  float score = INFINITY;
  if (has) {
    const uint32_t row = a.row_of_id[id];
    clus = last_le(a.cl_off, a.n_clusters + 1, (uint64_t)row);
    // the bucket holding the cluster: the last code c with bc_off[c] <= clus
    // (its range [bc_off[c], bc_off[c + 1]) then holds clus)
    code = (uint32_t)last_le(a.bc_off, a.n_codes + 1, (uint64_t)clus);
    const uint32_t diff = code ^ code0;
    bool ok = __popc(diff) <= a.r_max;
    uint32_t rmask = 0;   // flipped dimensions by rank
    for (int j = 0; j < b; ++j)
      if ((diff >> j) & 1u) {
        const int r = s_rank[j];
        if (r >= a.l_sel) ok = false; else rmask |= 1u << r;
      }
    if (ok) {
      float s = 0.0f;
      for (int r = 0; r < a.l_sel; ++r)
        if ((rmask >> r) & 1u) s += s_dlt[r];
      score = s;
    }
    a.scores[q * K + lane] = score;
  } else if (lane < K) {
    a.scores[q * K + lane] = INFINITY;
  }

  // the search's latent distance of the query to centroid c.  The logits
  // come from the lanes holding them (readlane), so it runs on every lane:
  // callers pass a valid cluster in all lanes and mask the result
  auto cdist = [&](int64_t c) __attribute__((always_inline)) {
    const float *mu = a.centroids + c * b;
    float acc = 0.0f;
    for (int j = 0; j < b; ++j) {
      const float lj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lg), j));
      const float tj = lj - mu[j];
      acc = fmaf(tj, tj, acc);
    }
    return acc;
  };
  // y's distance: the targets' own clusters (with any target there is a
  // cluster 0, which lanes without one score and drop)
  const uint64_t any = ballot(has);
  float dt = -INFINITY;
  if (any) {
    const float dc = cdist(has ? clus : 0);
    if (has) dt = dc;
  }
  // x: every centroid of every distinct target bucket, one bucket at a time
  uint64_t todo = any;
  float xmin = INFINITY;
  while (todo) {
    const int src = __ffsll((unsigned long long)todo) - 1;
    const uint32_t cb = bcast_u32(code, src);
    // drop every target in this bucket from the to-do set
    todo &= ~ballot(has && code == cb);
    const uint32_t c0 = a.bc_off[cb], c1 = a.bc_off[(uint64_t)cb + 1];
    for (uint32_t cb0 = c0; cb0 < c1; cb0 += WAVE) {
      const uint32_t c = cb0 + lane;
      const float dc = cdist(c < c1 ? c : c0);
      if (c < c1) xmin = fminf(xmin, dc);
    }
  }
  const float x = wave_min_f32(xmin);
  float ymax = dt;
  for (int m = 32; m >= 1; m >>= 1) ymax = fmaxf(ymax, __shfl_xor(ymax, m));
  if (lane == 0) {
    a.xy[q * 2] = any ? x : INFINITY;
    a.xy[q * 2 + 1] = any ? ymax - x : 0.0f;
  }
}

hipError_t launch_calib(const CalibArgs &a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_calib, dim3((unsigned)a.nq), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace nr
