// Step 2 (Algorithm 1, Sec. 3.4.1): binarisation (Eq. 10), deviation scores
// delta_j = |l_j - tau_j|, selection of the L_sel least stable dimensions and
// the ordered probe sequence, one wavefront per query.
//
// The sequence is the first P flip sets in ascending (score, rank mask) order,
// where the score is the fp32 sum of the flipped deltas added in rank order.
// It is built by a merge recursion over the selected ranks r = 0..L_sel-1:
//   L_r = firstP( L_{r-1}  merge  { m + {r} : m in L_{r-1}, |m| < R_max,
//                                    score(m) + delta_r <= S_max } ).
// Removing the highest rank of a flip set lowers its key, so every member of
// the global first-P has its parent in the previous first-P; the recursion is
// therefore exact, and adding delta_r last reproduces the rank-order sum.
// Keys are u64 (score bits << 32 | mask): scores are >= +0, so the float bit
// pattern orders like the value.  Lists live in LDS: L, the output of the
// merge, and the extension list E (which may need a sort when fp32 rounding
// maps different scores to one value); each merge is a merge-path merge in
// which every lane writes one contiguous slice of the output.
#include "nr_internal.h"

namespace nr {

static __host__ __device__ inline int pow2_ceil(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

__host__ __device__ size_t probe_lds_bytes_per_wave(int P) {
  return sizeof(uint64_t) * (size_t)(2 * P + pow2_ceil(P)) + 32 * (sizeof(int) + sizeof(float));
}

__global__ void k_probe(ProbeArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int wpb = blockDim.x >> 6;
  const int64_t q = (int64_t)blockIdx.x * wpb + wave;
  if (q >= a.nq) return;
  const int P = a.P, b = a.b, l_sel = a.l_sel;
  const int Pe = pow2_ceil(P);
  unsigned char *base = smem_raw + (size_t)wave * probe_lds_bytes_per_wave(P);
  uint64_t *L = reinterpret_cast<uint64_t *>(base);
  uint64_t *O = L + P;
  uint64_t *E = O + P;
  int *sel_dim = reinterpret_cast<int *>(E + Pe);
  float *sel_dlt = reinterpret_cast<float *>(sel_dim + 32);

  // a_j, b0 and delta_j, one dimension per lane
  float l = 0.f, t = 0.f;
  if (lane < b) {
    l = a.logits[q * b + lane];
    t = a.tau[lane];
  }
  const bool bit = lane < b && l >= t;
  const uint32_t code0 = (uint32_t)ballot(bit);
  const float dl = lane < b ? fabsf(l - t) : INFINITY;
  // rank of each dimension by (delta, dim): SmallestKIndices
  int rank = 0;
  for (int i = 0; i < b; ++i) {
    float di = __shfl(dl, i);
    rank += (di < dl) || (di == dl && i < lane);
  }
  if (lane < b && rank < l_sel) {
    sel_dim[rank] = lane;
    sel_dlt[rank] = dl;
  }
  __builtin_amdgcn_wave_barrier();

  if (lane == 0) L[0] = 0ull;  // the base address, score 0
  int n = 1;
  for (int r = 0; r < l_sel; ++r) {
    const float dr = sel_dlt[r];
    const uint32_t rbit = 1u << r;
    // extension list E
    int ne = 0;
    for (int i0 = 0; i0 < n; i0 += WAVE) {
      int i = i0 + lane;
      bool ok = false;
      uint64_t key = 0;
      if (i < n) {
        uint64_t k0 = L[i];
        uint32_t m = (uint32_t)k0;
        float c = __uint_as_float((uint32_t)(k0 >> 32));
        float c2 = c + dr;
        ok = __popc(m) < a.r_max && c2 <= a.s_max;
        key = ((uint64_t)__float_as_uint(c2) << 32) | (m | rbit);
      }
      uint64_t bm = ballot(ok);
      if (ok) E[ne + popc64(bm & lanemask_lt())] = key;
      ne += popc64(bm);
    }
    if (ne == 0) continue;
    __builtin_amdgcn_wave_barrier();
    // nothing of E can enter a full list whose last score is below E's first
    if (n == P) {
      float c_last = __uint_as_float((uint32_t)(L[n - 1] >> 32));
      float c_e = __uint_as_float((uint32_t)(E[0] >> 32));
      if (c_e > c_last) continue;
    }
    // E is ordered by score; equal scores may be out of mask order
    bool unsorted = false;
    for (int i0 = 0; i0 + 1 < ne; i0 += WAVE) {
      int i = i0 + lane;
      unsorted |= (i + 1 < ne) && E[i] > E[i + 1];
    }
    if (ballot(unsorted)) {
      int m2 = pow2_ceil(ne);
      for (int i = ne + lane; i < m2; i += WAVE) E[i] = ~0ull;
      __builtin_amdgcn_wave_barrier();
      for (int kk = 2; kk <= m2; kk <<= 1) {
        for (int j = kk >> 1; j > 0; j >>= 1) {
          for (int i0 = 0; i0 < m2; i0 += WAVE) {
            int i = i0 + lane;
            int ixj = i ^ j;
            if (i < m2 && ixj > i) {
              uint64_t x = E[i], y = E[ixj];
              bool asc = (i & kk) == 0;
              if ((x > y) == asc) { E[i] = y; E[ixj] = x; }
            }
          }
          __builtin_amdgcn_wave_barrier();
        }
      }
    }
    // merge path: lane l writes output slots [o0, o1) of the first P of
    // L merge E; keys are distinct (only E's masks hold bit r)
    {
      const int nout = n + ne < P ? n + ne : P;
      const int per = (nout + WAVE - 1) / WAVE;
      const int o0 = lane * per;
      const int o1 = o0 + per < nout ? o0 + per : nout;
      if (o0 < o1) {
        int lo = o0 - ne > 0 ? o0 - ne : 0;
        int hi = o0 < n ? o0 : n;
        while (lo < hi) {  // how many of the first o0 outputs come from L
          const int mid = (lo + hi) >> 1;
          if (L[mid] < E[o0 - mid - 1]) lo = mid + 1; else hi = mid;
        }
        int i = lo, j = o0 - lo;
        uint64_t x = i < n ? L[i] : ~0ull;
        uint64_t y = j < ne ? E[j] : ~0ull;
        for (int o = o0; o < o1; ++o) {
          if (x < y) {
            O[o] = x;
            ++i;
            x = i < n ? L[i] : ~0ull;
          } else {
            O[o] = y;
            ++j;
            y = j < ne ? E[j] : ~0ull;
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    n = n + ne < P ? n + ne : P;
    uint64_t *tmp = L; L = O; O = tmp;
  }

  // codes, scores and bins of the sequence
  for (int i0 = 0; i0 < n; i0 += WAVE) {
    int i = i0 + lane;
    if (i < n) {
      uint64_t key = L[i];
      uint32_t m = (uint32_t)key;
      float c = __uint_as_float((uint32_t)(key >> 32));
      uint32_t code = code0;
      while (m) {
        int rr = __ffs(m) - 1;
        m &= m - 1;
        code ^= 1u << sel_dim[rr];
      }
      int bin = i;
      if (a.finite) {
        int z = (int)floorf(c * a.bin_scale);
        bin = z < a.n_bins - 1 ? z : a.n_bins - 1;
      }
      a.codes[q * P + i] = code;
      a.costs[q * P + i] = c;
      a.bins[q * P + i] = bin;
    }
  }
  if (lane == 0) a.counts[q] = n;
}

hipError_t launch_probe(const ProbeArgs &a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  size_t per = probe_lds_bytes_per_wave(a.P);
  int wpb = 4;
  while (wpb > 1 && per * wpb > 64 * 1024) wpb >>= 1;
  int64_t blocks = (a.nq + wpb - 1) / wpb;
  size_t lds = per * wpb;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k_probe,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_probe, dim3((unsigned)blocks), dim3(64 * wpb), lds, s, a);
  return hipGetLastError();
}

}  // namespace nr
