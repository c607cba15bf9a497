// Seeded synthetic rows on the GPU: the same definition as synth/generators.py
// (Philox4x32-10, Salmon et al. SC'11; Irwin-Hall(12) noise from 16-bit
// draws), one thread per row, rows addressed by their id so that the payload
// can be generated directly in any (e.g. permuted) order.
// Compiled without FP contraction so every fp64 step is the NumPy one.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
constexpr uint32_t TAG_COMP = 1, TAG_NOISE = 2;
constexpr int64_t IH_CENTRE = 393210;

__device__ inline uint4 philox(uint4 c, uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)M0 * c.x, p1 = (uint64_t)M1 * c.z;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += W0;
    k1 += W1;
  }
  return c;
}

// sequential 16-bit draws of one row's noise stream
struct U16Stream {
  uint32_t lo, hi, seed, call = 0;
  uint32_t w[4];
  int pos = 8;  // halves consumed from the current call (8 per call)
  __device__ U16Stream(uint64_t row, uint32_t s) : lo((uint32_t)row), hi((uint32_t)(row >> 32)), seed(s) {}
  __device__ uint32_t next() {
    if (pos == 8) {
      uint4 o = philox(make_uint4(call, lo, hi, TAG_NOISE), seed, 0);
      w[0] = o.x; w[1] = o.y; w[2] = o.z; w[3] = o.w;
      ++call;
      pos = 0;
    }
    uint32_t word = w[pos >> 1];
    uint32_t v = (pos & 1) ? (word >> 16) : (word & 0xFFFFu);
    ++pos;
    return v;
  }
  __device__ double normal() {  // Irwin-Hall(12), centred, unit variance
    int64_t s = 0;
    for (int i = 0; i < 12; ++i) s += next();
    return (double)(s - IH_CENTRE) * (1.0 / 65536.0);
  }
};

__device__ inline int64_t component(uint64_t row, uint32_t seed, int64_t n_centers) {
  uint4 o = philox(make_uint4(0, (uint32_t)row, (uint32_t)(row >> 32), TAG_COMP), seed, 0);
  return (int64_t)(((uint64_t)o.x * (uint64_t)n_centers) >> 32);
}

__device__ inline uint64_t row_id(const int64_t *ids, int64_t first, int64_t i) {
  return ids ? (uint64_t)ids[i] : (uint64_t)(first + i);
}

__global__ void k_sift(uint32_t seed, const double *centers, int64_t n_centers, int d,
                       double sigma, const int64_t *ids, int64_t first, int64_t m, uint8_t *out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  uint64_t row = row_id(ids, first, i);
  const double *c = centers + component(row, seed, n_centers) * d;
  U16Stream st(row, seed);
  uint32_t *o = (uint32_t *)(out + i * d);
  for (int e0 = 0; e0 < d; e0 += 4) {
    uint32_t packed = 0;
    for (int j = 0; j < 4; ++j) {
      double z = st.normal() * sigma;
      double x = c[e0 + j] + z;
      x = rint(x);
      x = x < 0.0 ? 0.0 : (x > 255.0 ? 255.0 : x);
      packed |= (uint32_t)x << (8 * j);
    }
    o[e0 / 4] = packed;
  }
}

__global__ void k_deep(uint32_t seed, const double *centers, int64_t n_centers, int d,
                       const double *scale, const int64_t *ids, int64_t first, int64_t m,
                       float *out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  uint64_t row = row_id(ids, first, i);
  const double *c = centers + component(row, seed, n_centers) * d;
  double nrm2 = 0.0;
  {
    U16Stream st(row, seed);
    for (int e = 0; e < d; ++e) {
      double y = c[e] + st.normal() * scale[e];
      nrm2 = nrm2 + y * y;
    }
  }
  const double nrm = sqrt(nrm2);
  U16Stream st(row, seed);
  for (int e = 0; e < d; ++e) {
    double y = c[e] + st.normal() * scale[e];
    out[i * d + e] = (float)(y / nrm);
  }
}

__global__ void k_gauss(uint32_t seed, const double *centers, int64_t n_centers, int d,
                        double sigma, const int64_t *ids, int64_t first, int64_t m, float *out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  uint64_t row = row_id(ids, first, i);
  const double *c = centers + component(row, seed, n_centers) * d;
  U16Stream st(row, seed);
  for (int e = 0; e < d; ++e) out[i * d + e] = (float)(c[e] + st.normal() * sigma);
}

}  // namespace

extern "C" {

// kind: 0 = SIFT-like uint8, 1 = unit fp32 rows (Deep-like, GLD-like), 2 = Gaussian fp32.
// Rows are ids[i] (DEVICE int64) when ids is not NULL, else first + i.
// centers: DEVICE fp64 [n_centers x d]; out: DEVICE [m x d].  param is the
// noise std of kinds 0 and 2; scale (DEVICE fp64 [d]) the per-dimension noise
// std of kind 1.  Returns a hipError_t.
int synth_rows(int kind, uint32_t seed, const double *centers, int64_t n_centers, int d,
               double param, const double *scale, const int64_t *ids, int64_t first, int64_t m,
               void *out, hipStream_t stream) {
  if (m <= 0) return 0;
  if (d % 4 != 0 && kind == 0) return (int)hipErrorInvalidValue;
  if (kind == 1 && !scale) return (int)hipErrorInvalidValue;
  dim3 block(256), grid((unsigned)((m + 255) / 256));
  if (kind == 0)
    hipLaunchKernelGGL(k_sift, grid, block, 0, stream, seed, centers, n_centers, d, param, ids,
                       first, m, (uint8_t *)out);
  else if (kind == 1)
    hipLaunchKernelGGL(k_deep, grid, block, 0, stream, seed, centers, n_centers, d, scale, ids,
                       first, m, (float *)out);
  else
    hipLaunchKernelGGL(k_gauss, grid, block, 0, stream, seed, centers, n_centers, d, param, ids,
                       first, m, (float *)out);
  return (int)hipGetLastError();
}

}  // extern "C"
