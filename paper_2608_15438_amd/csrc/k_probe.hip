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
// pattern orders like the value.  The lists live in registers: element
// i = 64 j + lane of a list of PE = 64 K slots (PE the power of two >= P) is
// register j of that lane, unused slots hold all ones.  Each step keeps the
// PE smallest of L and E as min(L[i], E[PE-1-i]) -- a bitonic sequence --
// and sorts it with a bitonic merge (register pairs for distances >= 64,
// lane shuffles below).  E is compacted through LDS (one write and one read
// per step).  E keeps L's order except where fp32 rounding mapped different
// scores of L to one value and left equal scores out of mask order; such
// short runs are repaired by odd-even transposition rounds before the merge,
// and a list that is still unsorted after eight rounds is fully sorted.
#include "nr_internal.h"

namespace nr {

__device__ __forceinline__ uint64_t xor_u64(uint64_t v, int m) {
  const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
  const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t from_lane_u64(uint64_t v, int src) {
  const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src);
  const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a < b ? b : a; }

// sort a bitonic list ascending
template <int K>
__device__ __forceinline__ void bitonic_merge(uint64_t (&v)[K]) {
  const int lane = lane_id();
#pragma unroll
  for (int dj = K / 2; dj >= 1; dj >>= 1) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
      if ((j & dj) == 0) {
        const uint64_t x = v[j], y = v[j | dj];
        v[j] = umin64(x, y);
        v[j | dj] = umax64(x, y);
      }
    }
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const uint64_t o = xor_u64(v[j], d);
      v[j] = (lane & d) ? umax64(v[j], o) : umin64(v[j], o);
    }
  }
}

// sort any list ascending (bitonic sorting network)
template <int K>
__device__ __forceinline__ void bitonic_sort(uint64_t (&v)[K]) {
  const int lane = lane_id();
  constexpr int PE = 64 * K;
#pragma unroll
  for (int kk = 2; kk <= PE; kk <<= 1) {
#pragma unroll
    for (int d = kk >> 1; d >= 1; d >>= 1) {
      if (d >= 64) {
        const int dj = d >> 6;
#pragma unroll
        for (int j = 0; j < K; ++j) {
          if ((j & dj) == 0) {
            const bool asc = ((j * 64) & kk) == 0;
            const uint64_t x = v[j], y = v[j | dj];
            v[j] = asc ? umin64(x, y) : umax64(x, y);
            v[j | dj] = asc ? umax64(x, y) : umin64(x, y);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < K; ++j) {
          const int i = j * 64 + lane;
          const uint64_t o = xor_u64(v[j], d);
          const bool asc = (i & kk) == 0;
          const bool lower = (lane & d) == 0;
          v[j] = (lower == asc) ? umin64(v[j], o) : umax64(v[j], o);
        }
      }
    }
  }
}

template <int K>
__global__ void __launch_bounds__(256) k_probe(ProbeArgs a) {
  constexpr int PE = 64 * K;
  __shared__ uint64_t s_e[4][PE];
  const int lane = lane_id();
  uint64_t *es = s_e[threadIdx.x >> 6];
  const int64_t q = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (q >= a.nq) return;
  const int P = a.P, b = a.b, l_sel = a.l_sel;

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
    const float di = __shfl(dl, i);
    rank += (di < dl) || (di == dl && i < lane);
  }
  // lane r < l_sel: the dimension of rank r and its delta
  int sel_dim = 0;
  float sel_dlt = 0.f;
  for (int i = 0; i < b; ++i) {
    const int ri = __shfl(rank, i);
    const float di = __shfl(dl, i);
    if (lane == ri) {
      sel_dim = i;
      sel_dlt = di;
    }
  }

  uint64_t L[K];
#pragma unroll
  for (int j = 0; j < K; ++j) L[j] = ~0ull;
  if (lane == 0) L[0] = 0ull;  // the base address, score 0
  int n = 1;
  for (int r = 0; r < l_sel; ++r) {
    const float dr = __shfl(sel_dlt, r);
    const uint32_t rbit = 1u << r;
    // extension list E: every kept flip set plus rank r, compacted in L's
    // order through LDS (flip sets at r_max or past s_max drop out)
    uint64_t E[K];
    int ne = 0;
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const uint64_t k0 = L[j];
      const uint32_t m = (uint32_t)k0;
      const float c2 = __uint_as_float((uint32_t)(k0 >> 32)) + dr;
      const bool ok = k0 != ~0ull && __popc(m) < a.r_max && c2 <= a.s_max;
      const uint64_t bm = ballot(ok);
      if (ok) es[ne + popc64(bm & lanemask_lt())] = ((uint64_t)__float_as_uint(c2) << 32) | (m | rbit);
      ne += popc64(bm);
    }
    if (ne == 0) continue;
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const int i = j * 64 + lane;
      E[j] = i < ne ? es[i] : ~0ull;
    }
    __builtin_amdgcn_wave_barrier();
    // E follows L's order except inside runs of scores that rounding made
    // equal: odd-even transposition rounds repair such short runs; a list
    // still unsorted after 8 rounds gets the full sorting network.  Lane j of
    // bn / bp holds element 64 (j + 1) / 64 j - 1 (the neighbours across
    // register boundaries), taken before a round changes anything.
    for (int round = 0;; ++round) {
      uint64_t bn = ~0ull, bp = 0ull;
#pragma unroll
      for (int j = 0; j < K; ++j) {
        if (j + 1 < K) {
          const uint64_t v = bcast_u64(E[j + 1 < K ? j + 1 : j], 0);
          if (lane == j) bn = v;
        }
        if (j > 0) {
          const uint64_t v = bcast_u64(E[j > 0 ? j - 1 : j], 63);
          if (lane == j) bp = v;
        }
      }
      bool inv = false;
#pragma unroll
      for (int j = 0; j < K; ++j) {
        // every lane takes part in both exchanges before the select
        const uint64_t up = from_lane_u64(E[j], lane < 63 ? lane + 1 : lane);
        const uint64_t bj = bcast_u64(bn, j);
        const uint64_t nx = lane == 63 ? bj : up;
        inv |= E[j] > nx;
      }
      if (!ballot(inv)) break;
      if (round == 8) {
        bitonic_sort<K>(E);
        break;
      }
#pragma unroll
      for (int parity = 0; parity < 2; ++parity) {
        if (parity == 1) {  // the even round moved values: new boundary neighbours
          bn = ~0ull;
          bp = 0ull;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            if (j + 1 < K) {
              const uint64_t v = bcast_u64(E[j + 1 < K ? j + 1 : j], 0);
              if (lane == j) bn = v;
            }
            if (j > 0) {
              const uint64_t v = bcast_u64(E[j > 0 ? j - 1 : j], 63);
              if (lane == j) bp = v;
            }
          }
        }
#pragma unroll
        for (int j = 0; j < K; ++j) {
          // pairs (i, i + 1) with i of this parity; 64 is even, so the pair
          // of lane 63 and the next register's lane 0 has odd parity
          const uint64_t up = from_lane_u64(E[j], lane < 63 ? lane + 1 : lane);
          const uint64_t dn = from_lane_u64(E[j], lane > 0 ? lane - 1 : lane);
          const uint64_t bnj = bcast_u64(bn, j), bpj = bcast_u64(bp, j);
          const uint64_t nx = lane == 63 ? bnj : up;
          const uint64_t pv = lane == 0 ? bpj : dn;
          const bool first = (lane & 1) == parity;
          E[j] = first ? umin64(E[j], nx) : umax64(E[j], pv);
        }
      }
    }
    // the PE smallest of L and E, then sorted
#pragma unroll
    for (int j = 0; j < K; ++j) L[j] = umin64(L[j], from_lane_u64(E[K - 1 - j], 63 - lane));
    bitonic_merge<K>(L);
    n = n + ne < P ? n + ne : P;
#pragma unroll
    for (int j = 0; j < K; ++j)
      if (j * 64 + lane >= P) L[j] = ~0ull;
  }

  // codes, scores and bins of the sequence
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int i = j * 64 + lane;
    const uint64_t key = L[j];
    const uint32_t m = (uint32_t)key;
    uint32_t code = code0;
    for (int r = 0; r < l_sel; ++r) {
      const int dim = __shfl(sel_dim, r);
      if ((m >> r) & 1u) code ^= 1u << dim;
    }
    if (i < n) {
      const float c = __uint_as_float((uint32_t)(key >> 32));
      int bin = i;
      if (a.finite) {
        const int z = (int)floorf(c * a.bin_scale);
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
  const unsigned blocks = (unsigned)((a.nq + 3) / 4);
  const int P = a.P;
#define NR_PROBE_CASE(KK)                                                          \
  if (P <= 64 * KK) {                                                              \
    hipLaunchKernelGGL(k_probe<KK>, dim3(blocks), dim3(256), 0, s, a);             \
    return hipGetLastError();                                                      \
  }
  NR_PROBE_CASE(1)
  NR_PROBE_CASE(2)
  NR_PROBE_CASE(4)
  NR_PROBE_CASE(8)
  NR_PROBE_CASE(16)
#undef NR_PROBE_CASE
  return hipErrorInvalidValue;
}

}  // namespace nr
