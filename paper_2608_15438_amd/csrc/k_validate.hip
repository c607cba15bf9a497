// Upload-time checks of the borrowed index arrays (index construction,
// Sec. 3.3): directory offsets non-decreasing and consistent with the
// cluster count, cluster offsets non-decreasing and ending at n, and row_ids
// a permutation of 0..n-1 (each id seen once, marked in a bitmap).
#include "nr_internal.h"

namespace nr {

enum { BAD_BC = 1, BAD_CL = 2, BAD_IDS = 4 };

__global__ void k_validate(const uint32_t *bc_off, int64_t n_codes, const uint64_t *cl_off,
                           int64_t n_clusters, const int64_t *row_ids, int64_t n,
                           uint32_t *bitmap, int32_t *flags) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t g0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int32_t bad = 0;
  if (g0 == 0) {
    if (bc_off[0] != 0 || (int64_t)bc_off[n_codes] != n_clusters) bad |= BAD_BC;
    if (cl_off[0] != 0 || (int64_t)cl_off[n_clusters] != n) bad |= BAD_CL;
  }
  for (int64_t i = g0; i < n_codes; i += stride)
    if (bc_off[i] > bc_off[i + 1]) bad |= BAD_BC;
  for (int64_t i = g0; i < n_clusters; i += stride)
    if (cl_off[i] > cl_off[i + 1]) bad |= BAD_CL;
  for (int64_t r = g0; r < n; r += stride) {
    const int64_t id = row_ids[r];
    if (id < 0 || id >= n) {
      bad |= BAD_IDS;
    } else {
      const uint32_t bit = 1u << (id & 31);
      const uint32_t old = atomicOr(&bitmap[id >> 5], bit);
      if (old & bit) bad |= BAD_IDS;
    }
  }
  if (bad) atomicOr(flags, bad);
}

hipError_t launch_validate(const uint32_t *bc_off, int64_t n_codes, const uint64_t *cl_off,
                           int64_t n_clusters, const int64_t *row_ids, int64_t n,
                           uint32_t *bitmap, int32_t *flags, hipStream_t s) {
  hipLaunchKernelGGL(k_validate, dim3(2048), dim3(256), 0, s, bc_off, n_codes, cl_off,
                     n_clusters, row_ids, n, bitmap, flags);
  return hipGetLastError();
}

}  // namespace nr
