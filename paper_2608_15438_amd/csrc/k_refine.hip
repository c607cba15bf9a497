// Step 5: exact refinement of C(q) in the original space (Sec. 3.4 intro,
// Sec. 3.5) -- the HBM-bound part of the search.
//
//  plan   (one wave per query)  row prefix over the query's clusters, total
//         rows R_q, tile size T_q = max(TILE_MIN_ROWS, ceil(R_q / 64)), then
//         a scan over queries numbers the (query, row range) tiles;
//  refine (persistent waves)    each wave takes tiles from an atomic counter
//         and walks the tile's virtual rows; 8 lanes cover one 128-byte row
//         segment with one 16-byte load each, so a wave instruction reads 8
//         full cache lines; U rows per lane group are in flight;
//         uint8:  |x - q|^2 = x.x - 2 x.q + q.q with packed u8 dot products,
//                 exact in int32;   fp32: fmaf((x-q), (x-q), acc);
//         the 8 partial sums are combined with xor shuffles; a sorted top-k
//         of (distance, original id) lives in lanes 0..k-1 and a candidate
//         reads its original id only when it can enter it.  Rows past 1 KB
//         are summed per 1 KB slab (reduced over the 8 lanes, added in slab
//         order) against the query row in LDS, and an fp32 row stops being
//         read once its sum passes the list's k-th key;
//  merge  (one wave per query)  the tiles' partial top-k lists are merged.
#include "nr_internal.h"

// launch shape of the refinement (tuned on MI355X)
#ifndef NR_REFINE_BLOCKS_PER_CU
#define NR_REFINE_BLOCKS_PER_CU 8
#endif
#ifndef NR_REFINE_U1
#define NR_REFINE_U1 8          // rows in flight per lane group for 128-byte rows
#endif
#ifndef NR_REFINE_NT
#define NR_REFINE_NT 1          // non-temporal payload loads (+3% on MI355X)
#endif

namespace nr {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_payload(const uint4 *p) {
#if NR_REFINE_NT
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
#else
  return *p;
#endif
}

// ------------------------------------------------------------------ plan
// cluster counts come from the caller in nr_refine: keep them in [0, cap]
__device__ __forceinline__ int clamp_count(int32_t n, int64_t cap) {
  return n < 0 ? 0 : (n > cap ? (int)cap : n);
}

__global__ void __launch_bounds__(256) k_plan_rows(PlanArgs a) {
  const int lane = lane_id();
  const int64_t q = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (q >= a.nq) return;
  if (a.qmask && !a.qmask[q]) {
    if (lane == 0) {
      a.rtot[q] = 0;
      a.tsize[q] = TILE_MIN_ROWS;
      a.ntile[q] = 0;
    }
    return;
  }
  const int n = clamp_count(a.nclus[q], a.cap);
  const uint32_t *cl = a.clus + q * a.cap;
  uint32_t *pre = a.rowpre + q * (a.cap + 1);
  uint64_t run = 0;
  const int own0 = a.own_cseed ? a.own_cseed[q] : 0;
  // own (seed) pass of the shared schedule: only the leading clusters, compacted
  uint32_t *co = a.clus_out ? a.clus_out + q * a.cap : nullptr;
  int nout = 0;
  if (lane == 0) pre[0] = 0;
  // the compacted seed pass needs only the leading clusters
  const int nw = co && a.own_cseed && own0 < n ? own0 : n;
  for (int i0 = 0; i0 < nw; i0 += WAVE) {
    const int i = i0 + lane;
    uint32_t c = 0;
    uint64_t sz = 0;
    if (i < nw) {
      c = cl[i];
      if (c < a.n_clusters) {
        sz = a.cl_off[(uint64_t)c + 1] - a.cl_off[c];
        // the seed pass leaves every later cluster to the scan
        if (a.own_cseed && i >= own0) sz = 0;
      }
    }
    const uint64_t incl = wave_incl_scan_u64(sz);
    if (co) {
      const uint64_t keep = ballot(sz > 0);
      const int pos = nout + popc64(keep & lanemask_lt());
      if (sz > 0) {
        co[pos] = c;
        pre[pos + 1] = (uint32_t)(run + incl);
      }
      nout += popc64(keep);
    } else if (i < n) {
      pre[i + 1] = (uint32_t)(run + incl);
    }
    run += bcast_u64(incl, WAVE - 1);
  }
  if (lane == 0) {
    // a list of more than 2^32 - 1 rows (only possible with repeated clusters
    // given to nr_refine) is refused: it returns no candidates
    const uint32_t tot = run > 0xffffffffull ? 0u : (uint32_t)run;
    const uint32_t tmin = a.tile_min ? a.tile_min : TILE_MIN_ROWS;
    uint32_t t = (tot + MAX_TILES_PER_QUERY - 1) / MAX_TILES_PER_QUERY;
    if (t < tmin) t = tmin;
    a.rtot[q] = tot;
    a.tsize[q] = t;
    a.ntile[q] = (int32_t)(((uint64_t)tot + t - 1) / t);
    if (a.rfull) a.rfull[q] = tot;
    if (co) a.nclus_out[q] = nout;
  }
}

// exclusive scan of ntile over all queries in one block; resets the counter
__global__ void __launch_bounds__(1024) k_plan_scan(PlanArgs a) {
  __shared__ int32_t part[1024];
  const int tid = threadIdx.x;
  const int64_t per = (a.nq + 1023) / 1024;
  const int64_t s0 = tid * per;
  int32_t sum = 0;
  for (int64_t i = s0; i < s0 + per && i < a.nq; ++i) sum += a.ntile[i];
  part[tid] = sum;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    int32_t v = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int32_t run = part[tid] - sum;
  for (int64_t i = s0; i < s0 + per && i < a.nq; ++i) {
    a.tile_off[i] = run;
    run += a.ntile[i];
  }
  if (tid == 1023) {
    a.tile_off[a.nq] = part[1023];
    *a.counter = 0;
  }
}

// one thread per (query, tile slot): tile -> query and first cluster
__global__ void __launch_bounds__(256) k_plan_tiles(PlanArgs a) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t q = g / MAX_TILES_PER_QUERY;
  const int t = (int)(g % MAX_TILES_PER_QUERY);
  if (q >= a.nq || t >= a.ntile[q]) return;
  const int32_t tix = a.tile_off[q] + t;
  const uint32_t v0 = (uint32_t)t * a.tsize[q];
  const uint32_t *pre = a.rowpre + q * (a.cap + 1);
  // last cluster i with pre[i] <= v0 (clusters of zero rows are skipped)
  int lo = 0, hi = clamp_count(a.clus_out ? a.nclus_out[q] : a.nclus[q], a.cap) - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= v0) lo = mid; else hi = mid - 1;
  }
  a.tile_q[tix] = (int32_t)q;
  a.tile_c0[tix] = lo;
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_plan_rows, dim3((unsigned)((a.nq + 3) / 4)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_plan_scan, dim3(1), dim3(1024), 0, s, a);
  int64_t th = a.nq * MAX_TILES_PER_QUERY;
  hipLaunchKernelGGL(k_plan_tiles, dim3((unsigned)((th + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ top-k in lanes
// Lanes 0..k-1 hold a list sorted by (key, id); `kth` is the last entry when full.
struct TopK {
  uint32_t key;
  int64_t id;
  int cnt;
  uint32_t kth_key;
  int64_t kth_id;
};

__device__ __forceinline__ void topk_init(TopK &t) {
  t.key = 0xffffffffu;
  t.id = -1;
  t.cnt = 0;
  t.kth_key = 0xffffffffu;
  t.kth_id = INT64_MAX;
}

// insert (ck, cid) if it ranks among the k best (wave-uniform arguments)
__device__ __forceinline__ void topk_insert(TopK &t, int k, uint32_t ck, int64_t cid) {
  const int lane = lane_id();
  if (t.cnt == k && (ck > t.kth_key || (ck == t.kth_key && cid >= t.kth_id))) return;
  const bool less = lane < t.cnt && (t.key < ck || (t.key == ck && t.id < cid));
  const int pos = popc64(ballot(less));
  const uint32_t up_key = (uint32_t)__shfl_up((int)t.key, 1);
  const int64_t up_id = (int64_t)shfl_up_u64((uint64_t)t.id, 1);
  if (lane == pos) { t.key = ck; t.id = cid; }
  else if (lane > pos && lane < k) { t.key = up_key; t.id = up_id; }
  t.cnt = t.cnt + 1 < k ? t.cnt + 1 : k;
  if (t.cnt == k) {
    t.kth_key = bcast_u32(t.key, k - 1);
    t.kth_id = (int64_t)bcast_u64((uint64_t)t.id, k - 1);
  }
}

// The refinement's running top-k: like TopK, but an entry's original id is
// read only when it decides something -- a candidate whose key equals a key in
// the list (ids order equal keys) -- or when the tile's list is written out,
// so the row loop does not wait for id loads.  Entries keep their payload row
// (phys) until then; `known` marks the lanes whose id has been read.
struct LazyTopK {
  uint32_t key;
  int64_t id;
  uint64_t phys;
  bool known;
  int cnt;
  uint32_t kth_key;
};

__device__ __forceinline__ void ltopk_init(LazyTopK &t) {
  t.key = 0xffffffffu;
  t.id = -1;
  t.phys = 0;
  t.known = true;
  t.cnt = 0;
  t.kth_key = 0xffffffffu;
}

// insert the payload row cp with key ck if (ck, its id) ranks among the k best
// (wave-uniform arguments); ids are ordered as in TopK
__device__ __forceinline__ void ltopk_insert(LazyTopK &t, int k, uint32_t ck, uint64_t cp,
                                             const int64_t *row_ids) {
  const int lane = lane_id();
  if (t.cnt == k && ck > t.kth_key) return;
  // ids matter only among equal keys: read the candidate's and those of the
  // listed entries with its key (one round of loads, rare)
  const bool eq = lane < t.cnt && t.key == ck;
  int64_t cid = -1;
  bool cknown = false;
  if (ballot(eq)) {
    cid = row_ids[cp];
    cknown = true;
    if (eq && !t.known) {
      t.id = row_ids[t.phys];
      t.known = true;
    }
    // a tie with the k-th entry: the candidate enters only below its id
    if (t.cnt == k && ck == t.kth_key &&
        cid >= (int64_t)bcast_u64((uint64_t)t.id, k - 1)) return;
  }
  const bool less = lane < t.cnt && (t.key < ck || (t.key == ck && t.id < cid));
  const int pos = popc64(ballot(less));
  const uint32_t up_key = (uint32_t)__shfl_up((int)t.key, 1);
  const int64_t up_id = (int64_t)shfl_up_u64((uint64_t)t.id, 1);
  const uint64_t up_phys = shfl_up_u64(t.phys, 1);
  const bool up_known = __shfl_up((int)t.known, 1) != 0;
  if (lane == pos) {
    t.key = ck;
    t.id = cid;
    t.phys = cp;
    t.known = cknown;
  } else if (lane > pos && lane < k) {
    t.key = up_key;
    t.id = up_id;
    t.phys = up_phys;
    t.known = up_known;
  }
  t.cnt = t.cnt + 1 < k ? t.cnt + 1 : k;
  if (t.cnt == k) t.kth_key = bcast_u32(t.key, k - 1);
}

// ------------------------------------------------------------------ refine
#ifndef NR_REFINE_WAVES1
#define NR_REFINE_WAVES1 1      // waves per SIMD the registers are sized for (128-byte rows; 1: free)
#endif

template <int IS_U8, int NSEG, int U>
__global__ void __launch_bounds__(256, NSEG <= 1 ? NR_REFINE_WAVES1 : 1) k_refine(RefineArgs a) {
  __shared__ uint32_t s_vs[4][STAGE_CLUSTERS + 1];
  __shared__ uint64_t s_ps[4][STAGE_CLUSTERS];
  // rows longer than 8 segments: the wave's copy of the query row (slot gl of
  // segment s at s * 8 + gl), read a chunk at a time
  constexpr int SC = 8;
  __shared__ uint4 s_qrow[4][NSEG > SC ? NSEG * 8 : 1];
  const int lane = lane_id();
  const int w = threadIdx.x >> 6;
  const int g = lane >> 3;      // lane group: one row at a time
  const int gl = lane & 7;      // 16-byte slot inside a 128-byte row segment
  uint32_t *vs = s_vs[w];
  uint64_t *ps = s_ps[w];
  const int total = a.tile_off[a.nq];
  const int rb = a.row_bytes;
  const int k = a.k;
  if (total == 0) return;  // nothing to do: skip the counter (an empty redo launch)
  unsigned long long nbytes = 0;  // row bytes this lane group read (its lane 0)

  for (;;) {
    int t = 0;
    if (lane == 0) t = atomicAdd(a.counter, 1);
    t = __builtin_amdgcn_readfirstlane(t);
    if (t >= total) break;
    const int64_t q = a.tile_q[t];
    const uint32_t T = a.tsize[q];
    const uint32_t R = a.rtot[q];
    const uint32_t v0 = (uint32_t)(t - a.tile_off[q]) * T;
    const uint32_t v1 = v0 + T < R ? v0 + T : R;
    const uint32_t *pre = a.rowpre + q * (a.cap + 1);
    const uint32_t *cl = a.clus + q * a.cap;
    const int n_cl = clamp_count(a.nclus[q], a.cap);
    int c = a.tile_c0[t];

    // this lane's slices of the query: in registers for rows of up to 8
    // segments, from the wave's LDS copy for longer ones
    uint4 qv[NSEG <= SC ? NSEG : 1];
    uint4 *qrow = s_qrow[w];
    const unsigned char *qb = (const unsigned char *)a.queries + q * (int64_t)rb;
    if constexpr (NSEG <= SC) {
#pragma unroll
      for (int s = 0; s < NSEG; ++s) {
        const int off = 128 * s + 16 * gl;
        qv[s] = off < rb ? *(const uint4 *)(qb + off) : make_uint4(0, 0, 0, 0);
      }
    } else {
      __builtin_amdgcn_wave_barrier();  // the previous tile is done with the copy
      for (int i = lane; i < NSEG * 8; i += WAVE)
        qrow[i] = 16 * i < rb ? *(const uint4 *)(qb + 16 * i) : make_uint4(0, 0, 0, 0);
      __builtin_amdgcn_wave_barrier();
    }
    int32_t qq = 0;
    if (IS_U8) {
#pragma unroll
      for (int s = 0; s < NSEG; ++s) {
        const uint4 qs4 = NSEG <= SC ? qv[NSEG <= SC ? s : 0] : qrow[s * 8 + gl];
        uint32_t acc = (uint32_t)qq;
        acc = __builtin_amdgcn_udot4(qs4.x, qs4.x, acc, false);
        acc = __builtin_amdgcn_udot4(qs4.y, qs4.y, acc, false);
        acc = __builtin_amdgcn_udot4(qs4.z, qs4.z, acc, false);
        acc = __builtin_amdgcn_udot4(qs4.w, qs4.w, acc, false);
        qq = (int32_t)acc;
      }
      qq += __shfl_xor(qq, 1);
      qq += __shfl_xor(qq, 2);
      qq += __shfl_xor(qq, 4);
    }
    LazyTopK tk;
    ltopk_init(tk);

    uint32_t v = v0;
    while (v < v1) {
      // stage clusters c .. c+ns-1: virtual and physical first rows
      const int ns = n_cl - c < STAGE_CLUSTERS ? n_cl - c : STAGE_CLUSTERS;
      for (int j = lane; j < ns; j += WAVE) {
        vs[j] = pre[c + j];
        const uint32_t cj = cl[c + j];
        ps[j] = cj < a.n_clusters ? a.cl_off[cj] : 0;
      }
      if (lane == 0) vs[ns] = pre[c + ns];
      __builtin_amdgcn_wave_barrier();
      const uint32_t vend = v1 < vs[ns] ? v1 : vs[ns];
      // per lane group (rows of a group only increase): the staged cluster
      // holding its rows, its first virtual row and physical row, and the
      // next cluster's first virtual row, kept in registers so that a row
      // costs an LDS read only where it crosses into the next cluster
      int cur = 0;
      uint32_t vcur = vs[0], vnext = vs[1];
      uint64_t pcur = ps[0];
      if constexpr (NSEG == 1) {
        // rows of one 128-byte segment: a two-stage pipeline, the rows of the
        // next step loading while those of this one are scored (two register
        // buffers, the loop unrolled by two).  A row's payload index is kept
        // only until its load is issued; an entrant's is found again from
        // the staged clusters.
        uint4 xa[U], xb[U];
        auto issue = [&](uint32_t vb, uint4(&x)[U]) __attribute__((always_inline)) {
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const uint32_t rv = vb + 8 * u + g;
            const bool ok = rv < vend;
            uint64_t phys = 0;
            if (ok) {
              if (vnext <= rv) {
                do {
                  ++cur;
                  vnext = vs[cur + 1];
                } while (vnext <= rv);
                vcur = vs[cur];
                pcur = ps[cur];
              }
              phys = pcur + (rv - vcur);
            }
            x[u] = (ok && 16 * gl < rb) ? load_payload(a.ra.seg(phys, 16 * gl))
                                        : make_uint4(0, 0, 0, 0);
          }
        };
        auto score = [&](uint32_t vb, const uint4(&x)[U]) __attribute__((always_inline)) {
          uint32_t key[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            if (IS_U8) {
              uint32_t xx = 0, xq = 0;
              xx = __builtin_amdgcn_udot4(x[u].x, x[u].x, xx, false);
              xx = __builtin_amdgcn_udot4(x[u].y, x[u].y, xx, false);
              xx = __builtin_amdgcn_udot4(x[u].z, x[u].z, xx, false);
              xx = __builtin_amdgcn_udot4(x[u].w, x[u].w, xx, false);
              xq = __builtin_amdgcn_udot4(x[u].x, qv[0].x, xq, false);
              xq = __builtin_amdgcn_udot4(x[u].y, qv[0].y, xq, false);
              xq = __builtin_amdgcn_udot4(x[u].z, qv[0].z, xq, false);
              xq = __builtin_amdgcn_udot4(x[u].w, qv[0].w, xq, false);
              int32_t part = (int32_t)xx - 2 * (int32_t)xq;
              part += __shfl_xor(part, 1);
              part += __shfl_xor(part, 2);
              part += __shfl_xor(part, 4);
              key[u] = (uint32_t)(part + qq);
            } else {
              float acc = 0.0f;
              const float t0 = __uint_as_float(x[u].x) - __uint_as_float(qv[0].x);
              const float t1 = __uint_as_float(x[u].y) - __uint_as_float(qv[0].y);
              const float t2 = __uint_as_float(x[u].z) - __uint_as_float(qv[0].z);
              const float t3 = __uint_as_float(x[u].w) - __uint_as_float(qv[0].w);
              acc = fmaf(t0, t0, acc);
              acc = fmaf(t1, t1, acc);
              acc = fmaf(t2, t2, acc);
              acc = fmaf(t3, t3, acc);
              acc += __shfl_xor(acc, 1);
              acc += __shfl_xor(acc, 2);
              acc += __shfl_xor(acc, 4);
              key[u] = __float_as_uint(acc);
            }
          }
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const bool ok = vb + 8 * u + g < vend;
            if (ok && gl == 0) nbytes += (uint32_t)rb;
            uint64_t m = ballot(ok && gl == 0 && key[u] <= tk.kth_key);
            while (m) {
              const int src = __ffsll((unsigned long long)m) - 1;
              m &= m - 1;
              const uint32_t ck = bcast_u32(key[u], src);
              if (tk.cnt == k && ck > tk.kth_key) continue;
              // the entrant's payload row: the last staged cluster starting
              // at or before its virtual row
              const uint32_t rv = vb + 8 * u + (uint32_t)(src >> 3);
              int lo = 0, hi = ns - 1;
              while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (vs[mid] <= rv) lo = mid; else hi = mid - 1;
              }
              ltopk_insert(tk, k, ck, ps[lo] + (rv - vs[lo]), a.row_ids);
            }
          }
        };
        uint32_t vb = v;
        issue(vb, xa);
        for (;;) {
          const uint32_t vn = vb + 8 * U;
          if (vn < vend) issue(vn, xb);
          score(vb, xa);
          if (vn >= vend) break;
          const uint32_t vn2 = vn + 8 * U;
          if (vn2 < vend) issue(vn2, xa);
          score(vn, xb);
          if (vn2 >= vend) break;
          vb = vn2;
        }
      } else
      for (uint32_t vb = v; vb < vend; vb += 8 * U) {
        uint64_t phys[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const uint32_t rv = vb + 8 * u + g;
          ok[u] = rv < vend;
          phys[u] = 0;
          if (ok[u]) {
            if (vnext <= rv) {
              do {
                ++cur;
                vnext = vs[cur + 1];
              } while (vnext <= rv);
              vcur = vs[cur];
              pcur = ps[cur];
            }
            phys[u] = pcur + (rv - vcur);
          }
        }
        uint32_t key[U];
        if constexpr (NSEG > SC) {
          // long rows: slabs of SC segments (1 KB).  Each slab is accumulated
          // in segment order per lane, reduced over the row's 8 lanes, and
          // added to the row's running sum in slab order: the arithmetic the
          // batch-shared scan uses for rows this long
          uint32_t xx[U], xq[U];
          float fs[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            xx[u] = 0;
            xq[u] = 0;
            fs[u] = 0.0f;
          }
          const int nsl = (rb + 128 * SC - 1) / (128 * SC);
          // fp32: the running sum only grows (non-negative terms rounded to
          // nearest), so a row whose sum is already past the list's k-th key
          // cannot enter it and reads no further slabs
          const uint32_t bound = tk.kth_key;
#pragma unroll 1
          for (int sl = 0; sl < nsl; ++sl) {
            const int s0 = sl * SC;
            if (!IS_U8 && sl > 0) {
              bool any = false;
#pragma unroll
              for (int u = 0; u < U; ++u) {
                ok[u] = ok[u] && __float_as_uint(fs[u]) <= bound;
                any |= ok[u];
              }
              if (!ballot(any)) break;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
              if (ok[u] && gl == 0) nbytes += (uint32_t)(rb - 128 * s0 < 128 * SC ? rb - 128 * s0 : 128 * SC);
            uint4 xc[U][SC];
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
              for (int s = 0; s < SC; ++s) {
                const int off = 128 * (s0 + s) + 16 * gl;
                xc[u][s] = (ok[u] && off < rb) ? load_payload(a.ra.seg(phys[u], off))
                                               : make_uint4(0, 0, 0, 0);
              }
            }
            uint4 qc[SC];
#pragma unroll
            for (int s = 0; s < SC; ++s) qc[s] = qrow[(s0 + s) * 8 + gl];
#pragma unroll
            for (int u = 0; u < U; ++u) {
              float fa = 0.0f;
#pragma unroll
              for (int s = 0; s < SC; ++s) {
                if (IS_U8) {
                  xx[u] = __builtin_amdgcn_udot4(xc[u][s].x, xc[u][s].x, xx[u], false);
                  xx[u] = __builtin_amdgcn_udot4(xc[u][s].y, xc[u][s].y, xx[u], false);
                  xx[u] = __builtin_amdgcn_udot4(xc[u][s].z, xc[u][s].z, xx[u], false);
                  xx[u] = __builtin_amdgcn_udot4(xc[u][s].w, xc[u][s].w, xx[u], false);
                  xq[u] = __builtin_amdgcn_udot4(xc[u][s].x, qc[s].x, xq[u], false);
                  xq[u] = __builtin_amdgcn_udot4(xc[u][s].y, qc[s].y, xq[u], false);
                  xq[u] = __builtin_amdgcn_udot4(xc[u][s].z, qc[s].z, xq[u], false);
                  xq[u] = __builtin_amdgcn_udot4(xc[u][s].w, qc[s].w, xq[u], false);
                } else {
                  const float t0 = __uint_as_float(xc[u][s].x) - __uint_as_float(qc[s].x);
                  const float t1 = __uint_as_float(xc[u][s].y) - __uint_as_float(qc[s].y);
                  const float t2 = __uint_as_float(xc[u][s].z) - __uint_as_float(qc[s].z);
                  const float t3 = __uint_as_float(xc[u][s].w) - __uint_as_float(qc[s].w);
                  fa = fmaf(t0, t0, fa);
                  fa = fmaf(t1, t1, fa);
                  fa = fmaf(t2, t2, fa);
                  fa = fmaf(t3, t3, fa);
                }
              }
              if (!IS_U8) {
                fa += __shfl_xor(fa, 1);
                fa += __shfl_xor(fa, 2);
                fa += __shfl_xor(fa, 4);
                fs[u] = sl == 0 ? fa : fs[u] + fa;
              }
            }
          }
#pragma unroll
          for (int u = 0; u < U; ++u) {
            if (IS_U8) {
              // integer sums: the slab order does not matter
              int32_t part = (int32_t)xx[u] - 2 * (int32_t)xq[u];
              part += __shfl_xor(part, 1);
              part += __shfl_xor(part, 2);
              part += __shfl_xor(part, 4);
              key[u] = (uint32_t)(part + qq);
            } else {
              key[u] = __float_as_uint(fs[u]);
            }
          }
        } else {
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (ok[u] && gl == 0) nbytes += (uint32_t)rb;
        uint4 xv[U][NSEG];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
          for (int s = 0; s < NSEG; ++s) {
            const int off = 128 * s + 16 * gl;
            xv[u][s] = (ok[u] && off < rb) ? load_payload(a.ra.seg(phys[u], off))
                                           : make_uint4(0, 0, 0, 0);
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (IS_U8) {
            uint32_t xx = 0, xq = 0;
#pragma unroll
            for (int s = 0; s < NSEG; ++s) {
              xx = __builtin_amdgcn_udot4(xv[u][s].x, xv[u][s].x, xx, false);
              xx = __builtin_amdgcn_udot4(xv[u][s].y, xv[u][s].y, xx, false);
              xx = __builtin_amdgcn_udot4(xv[u][s].z, xv[u][s].z, xx, false);
              xx = __builtin_amdgcn_udot4(xv[u][s].w, xv[u][s].w, xx, false);
              xq = __builtin_amdgcn_udot4(xv[u][s].x, qv[s].x, xq, false);
              xq = __builtin_amdgcn_udot4(xv[u][s].y, qv[s].y, xq, false);
              xq = __builtin_amdgcn_udot4(xv[u][s].z, qv[s].z, xq, false);
              xq = __builtin_amdgcn_udot4(xv[u][s].w, qv[s].w, xq, false);
            }
            int32_t part = (int32_t)xx - 2 * (int32_t)xq;
            part += __shfl_xor(part, 1);
            part += __shfl_xor(part, 2);
            part += __shfl_xor(part, 4);
            key[u] = (uint32_t)(part + qq);
          } else {
            float acc = 0.0f;
#pragma unroll
            for (int s = 0; s < NSEG; ++s) {
              float t0 = __uint_as_float(xv[u][s].x) - __uint_as_float(qv[s].x);
              float t1 = __uint_as_float(xv[u][s].y) - __uint_as_float(qv[s].y);
              float t2 = __uint_as_float(xv[u][s].z) - __uint_as_float(qv[s].z);
              float t3 = __uint_as_float(xv[u][s].w) - __uint_as_float(qv[s].w);
              acc = fmaf(t0, t0, acc);
              acc = fmaf(t1, t1, acc);
              acc = fmaf(t2, t2, acc);
              acc = fmaf(t3, t3, acc);
            }
            acc += __shfl_xor(acc, 1);
            acc += __shfl_xor(acc, 2);
            acc += __shfl_xor(acc, 4);
            key[u] = __float_as_uint(acc);
          }
        }
        }
        // rows that may enter the top-k, in row order
#pragma unroll
        for (int u = 0; u < U; ++u) {
          uint64_t m = ballot(ok[u] && gl == 0 && key[u] <= tk.kth_key);
          while (m) {
            const int src = __ffsll((unsigned long long)m) - 1;
            m &= m - 1;
            const uint32_t ck = bcast_u32(key[u], src);
            if (tk.cnt == k && ck > tk.kth_key) continue;
            ltopk_insert(tk, k, ck, bcast_u64(phys[u], src), a.row_ids);
          }
        }
      }
      v = vend;
      c += ns;
      __builtin_amdgcn_wave_barrier();
    }
    // partial result of this tile: the ids not read yet, all at once
    if (lane < tk.cnt && !tk.known) tk.id = a.row_ids[tk.phys];
    if (lane < k) {
      a.pkey[(int64_t)t * k + lane] = lane < tk.cnt ? tk.key : 0xffffffffu;
      a.pid[(int64_t)t * k + lane] = lane < tk.cnt ? tk.id : -1;
    }
  }
  if (a.rbytes && gl == 0 && nbytes) atomicAdd(a.rbytes, nbytes);
}

template <int IS_U8>
static hipError_t launch_refine_t(const RefineArgs &a, int nseg, int grid, hipStream_t s) {
#define NR_REFINE_CASE(NS, UU)                                                     \
  if (nseg <= NS) {                                                                \
    hipLaunchKernelGGL((k_refine<IS_U8, NS, UU>), dim3(grid), dim3(256), 0, s, a); \
    return hipGetLastError();                                                      \
  }
  NR_REFINE_CASE(1, NR_REFINE_U1)
  NR_REFINE_CASE(2, 4)
  NR_REFINE_CASE(3, 4)
  NR_REFINE_CASE(4, 2)
  NR_REFINE_CASE(8, 1)
  NR_REFINE_CASE(16, 2)
  NR_REFINE_CASE(48, 2)
#undef NR_REFINE_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_refine(const RefineArgs &a, int dtype, int n_cu, int blocks_per_cu,
                         hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  const int nseg = (a.row_bytes + 127) / 128;
  const int grid = n_cu * (blocks_per_cu > 0 ? blocks_per_cu : NR_REFINE_BLOCKS_PER_CU);
  return dtype == NR_U8 ? launch_refine_t<1>(a, nseg, grid, s) : launch_refine_t<0>(a, nseg, grid, s);
}

// ------------------------------------------------------------------ merge
__global__ void __launch_bounds__(256) k_merge(MergeArgs a) {
  const int lane = lane_id();
  const int64_t q = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (q >= a.nq) return;
  if (a.qmask && !a.qmask[q]) return;
  const int k = a.k;
  const int64_t e0 = (int64_t)a.tile_off[q] * k, e1 = (int64_t)a.tile_off[q + 1] * k;
  TopK tk;
  topk_init(tk);
  for (int64_t i0 = e0; i0 < e1; i0 += WAVE) {
    const int64_t i = i0 + lane;
    uint32_t key = 0xffffffffu;
    int64_t id = -1;
    if (i < e1) {
      key = a.pkey[i];
      id = a.pid[i];
    }
    uint64_t m = ballot(id >= 0 && key <= tk.kth_key);
    while (m) {
      const int src = __ffsll((unsigned long long)m) - 1;
      m &= m - 1;
      topk_insert(tk, k, bcast_u32(key, src), (int64_t)bcast_u64((uint64_t)id, src));
    }
  }
  if (lane < k) {
    const bool have = lane < tk.cnt;
    a.out_ids[q * k + lane] = have ? tk.id : -1;
    a.out_dists[q * k + lane] =
        have ? (a.is_u8 ? (float)tk.key : __uint_as_float(tk.key)) : INFINITY;
  }
  if (lane == 0 && a.qstats) {
    a.qstats[q * NR_QSTATS + NR_QS_ROWS] = (int32_t)a.rtot[q];
    a.qstats[q * NR_QSTATS + NR_QS_TILES] = a.tile_off[q + 1] - a.tile_off[q];
  }
}

hipError_t launch_merge(const MergeArgs &a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_merge, dim3((unsigned)((a.nq + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace nr
