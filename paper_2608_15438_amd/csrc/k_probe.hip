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
// pattern orders like the value.
//
// The lists live in LDS (one wave per query).  Each step compacts the
// extension list E in L's order; E keeps that order except where fp32
// rounding mapped different scores of L to one value and left equal scores
// out of mask order, which odd-even transposition rounds repair.  The merge
// is split by output position: lane t finds where output slot t * c falls
// in L and E by a binary search on the merge path (keys of L and E never
// tie: E's carry rank r, L's do not) and writes the next c outputs.
#include "nr_internal.h"

namespace nr {

__global__ void __launch_bounds__(64) k_probe(ProbeArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  const int lane = lane_id();
  const int64_t q = blockIdx.x;
  if (q >= a.nq) return;
  const int P = a.P, b = a.b, l_sel = a.l_sel;
  const int pc = (P + WAVE - 1) / WAVE * WAVE;
  uint64_t *L = reinterpret_cast<uint64_t *>(smem_raw);
  uint64_t *Ln = L + pc;
  uint64_t *E = Ln + pc;

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
    const float di = bcast_f32(dl, i);  // i is the same in every lane
    rank += (di < dl) || (di == dl && i < lane);
  }
  // lane r < l_sel: the dimension of rank r and its delta
  int sel_dim = 0;
  float sel_dlt = 0.f;
  for (int i = 0; i < b; ++i) {
    const int ri = (int)bcast_u32((uint32_t)rank, i);
    const float di = bcast_f32(dl, i);
    if (lane == ri) {
      sel_dim = i;
      sel_dlt = di;
    }
  }

  if (lane == 0) L[0] = 0ull;  // the base address, score 0
  int n = 1;
  __builtin_amdgcn_wave_barrier();
  for (int r = 0; r < l_sel; ++r) {
    const float dr = bcast_f32(sel_dlt, r);
    const uint32_t rbit = 1u << r;
    // E: every kept flip set plus rank r, in L's order (flip sets at R_max
    // or past S_max drop out)
    int ne = 0;
    for (int i0 = 0; i0 < n; i0 += WAVE) {
      const int i = i0 + lane;
      const uint64_t k0 = i < n ? L[i] : ~0ull;
      const uint32_t m = (uint32_t)k0;
      const float c2 = __uint_as_float((uint32_t)(k0 >> 32)) + dr;
      const bool ok = i < n && __popc(m) < a.r_max && c2 <= a.s_max;
      const uint64_t bm = ballot(ok);
      if (ok) E[ne + popc64(bm & lanemask_lt())] = ((uint64_t)__float_as_uint(c2) << 32) | (m | rbit);
      ne += popc64(bm);
    }
    if (ne == 0) continue;
    __builtin_amdgcn_wave_barrier();
    // odd-even transposition rounds until E is sorted (ties are rare and
    // their runs short; n rounds always suffice)
    for (;;) {
      bool inv = false;
      for (int i0 = 0; i0 + 1 < ne; i0 += WAVE) {
        const int i = i0 + lane;
        if (i + 1 < ne) inv |= E[i] > E[i + 1];
      }
      if (!ballot(inv)) break;
      for (int parity = 0; parity < 2; ++parity) {
        for (int p0 = 0; 2 * p0 + parity + 1 < ne; p0 += WAVE) {
          const int i = 2 * (p0 + lane) + parity;
          if (i + 1 < ne) {
            const uint64_t x = E[i], y = E[i + 1];
            if (x > y) {
              E[i] = y;
              E[i + 1] = x;
            }
          }
        }
        __builtin_amdgcn_wave_barrier();
      }
    }
    // Ln = first min(n + ne, P) of merge(L, E); lane t writes [t c, t c + c)
    const int nout = n + ne < P ? n + ne : P;
    const int c = (nout + WAVE - 1) / WAVE;
    const int d = lane * c;
    if (d < nout) {
      int lo = d - ne > 0 ? d - ne : 0;
      int hi = d < n ? d : n;
      while (lo < hi) {  // i = number of L's entries among the first d outputs
        const int mid = (lo + hi) >> 1;
        if (L[mid] < E[d - mid - 1]) lo = mid + 1; else hi = mid;
      }
      int i = lo, j = d - lo;
      uint64_t x = i < n ? L[i] : ~0ull;
      uint64_t y = j < ne ? E[j] : ~0ull;
      const int end = d + c < nout ? d + c : nout;
      for (int o = d; o < end; ++o) {
        if (x < y) {
          Ln[o] = x;
          ++i;
          x = i < n ? L[i] : ~0ull;
        } else {
          Ln[o] = y;
          ++j;
          y = j < ne ? E[j] : ~0ull;
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    uint64_t *tmp = L;
    L = Ln;
    Ln = tmp;
    n = nout;
  }

  // codes, scores and bins of the sequence, four per lane at a time (every
  // lane runs each round: the dimension of rank r is read from lane r); for
  // the search, each probe's bucket range from the directory (the four
  // lookups of a lane in flight together) and the query's route pass
  uint32_t msum = 0;  // clusters in the query's multi-cluster buckets
  for (int i0 = 0; i0 < n; i0 += 4 * WAVE) {
    uint64_t key[4];
    uint32_t code[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * WAVE + lane;
      key[u] = i < n ? L[i] : 0ull;
      code[u] = code0;
    }
    for (int r = 0; r < l_sel; ++r) {
      const uint32_t bit = 1u << bcast_u32((uint32_t)sel_dim, r);
#pragma unroll
      for (int u = 0; u < 4; ++u) code[u] ^= (((uint32_t)key[u] >> r) & 1u) ? bit : 0u;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * WAVE + lane;
      if (i < n) {
        const float c = __uint_as_float((uint32_t)(key[u] >> 32));
        int bin = i;
        if (a.finite) {
          const int z = (int)floorf(c * a.bin_scale);
          bin = z < a.n_bins - 1 ? z : a.n_bins - 1;
        }
        a.codes[q * P + i] = code[u];
        a.costs[q * P + i] = c;
        a.bins[q * P + i] = bin;
      }
    }
    if (a.lk) {
      uint2 r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * WAVE + lane;
        if (i < n) r[u] = make_uint2(a.bc_off[code[u]], a.bc_off[(uint64_t)code[u] + 1]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * WAVE + lane;
        if (i < n) {
          a.lk[q * P + i] = r[u];
          const uint32_t sz = r[u].y - r[u].x;
          msum += sz >= 2 ? sz : 0u;
        }
      }
    }
  }
  if (lane == 0) a.counts[q] = n;
  if (a.tier) {
    msum = wave_sum_u32(msum);
    if (lane == 0)
      a.tier[q] = msum <= (uint32_t)a.tier_h0
                      ? 0
                      : (a.tier_n > 2 && msum <= (uint32_t)a.tier_h1 ? 1 : a.tier_n - 1);
  }
}

hipError_t launch_probe(const ProbeArgs &a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  if (a.P < 1 || a.P > NR_MAX_PROBES) return hipErrorInvalidValue;
  const size_t pc = (size_t)(a.P + WAVE - 1) / WAVE * WAVE;
  const size_t lds = 3 * pc * sizeof(uint64_t);  // 96 KiB at P = 4096 (gfx950: 160 KiB per CU)
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)k_probe,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_probe, dim3((unsigned)a.nq), dim3(64), lds, s, a);
  return hipGetLastError();
}

}  // namespace nr
