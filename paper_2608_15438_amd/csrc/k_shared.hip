// Batch-shared exact refinement (step 5 of the search, Sec. 3.4 intro and
// Sec. 3.5): the same top-k over C(q) as the per-query schedule, computed so
// that a cluster listed by several queries of the batch is read from HBM once
// for all of them.
//
//  hist    per query (one wave, at the end of the route kernel once the
//          query's list is final): the leading clusters of its list that
//          cover at least seed_min rows stay with the query; every later
//          (cluster, query) pair is counted per cluster; |q|^2 and its head
//          part are kept for uint8 rows;
//  seed    the per-query kernels refine each query's leading clusters.  Their
//          top-k is exact over a subset of C(q), so its k-th entry bounds
//          the final k-th entry: a later row can only enter the result if it
//          ranks at or before it;
//  prep    (on a second stream, beside the seed pass) the clusters with
//          pairs (nonzero pair counts, found by one sequential pass over the
//          counts) form the scan list in cluster order with their pair and
//          work ranges (rows x groups of <= g queries); the pairs are then
//          scattered by cluster;
//  scan    persistent waves take tiles of SHARED_TILE work from an atomic
//          counter and gather consecutive units of the tile into batches
//          whose query rows sit in LDS.  Each row's head (its first
//          scan_head bytes) is read once for all queries of its unit and
//          drops the pairs whose head part alone exceeds the bound; the
//          remaining rows are read whole and scored exactly, and a pair at
//          or before its query's bound becomes a survivor (per-query slots,
//          then a shared pool).  fp32 rows past 1 KB are scored on their
//          first 1 KB slab only; the pairs it leaves open are finished by
//          the open-pair pass, slab by slab;
//  merge   seed top-k + survivors -> top-k.  A query whose survivors found
//          the pool full is flagged and recomputed by the per-query
//          schedule.
#include <cstring>

#include "nr_internal.h"

// launch shape of the shared scan (tuned on MI355X)
#ifndef NR_SHARED_BLOCKS_PER_CU
#define NR_SHARED_BLOCKS_PER_CU 8
#endif
#ifndef NR_SHARED_TILE
#define NR_SHARED_TILE 4096     // work (rows x query groups) per scan tile
#endif
#ifndef NR_SCAN_U1
#define NR_SCAN_U1 6            // head loads in flight per lane (16-byte heads)
#endif
#ifndef NR_SCAN_UB1
#define NR_SCAN_UB1 4           // whole rows in flight per lane group (128-byte rows)
#endif
#ifndef NR_SCAN_SLACK
#define NR_SCAN_SLACK 124       // listed rows beyond one pass before whole rows are read
#endif
#ifndef NR_SCAN_QMAX1
#define NR_SCAN_QMAX1 32        // query slots per batch (128-byte rows)
#endif
// waves per SIMD the register budget is sized for, rows of one 128-byte
// segment (five blocks of four waves per CU also need at most 32 KiB of LDS
// per block); longer rows keep what their registers allow
#ifndef NR_SCAN_WAVES1
#define NR_SCAN_WAVES1 5
#endif

namespace nr {

constexpr uint64_t SHARED_TILE = NR_SHARED_TILE;

typedef unsigned int su32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
  const su32x4 v = __builtin_nontemporal_load(reinterpret_cast<const su32x4 *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ int clamp_n(int32_t n, int64_t cap) {
  return n < 0 ? 0 : (n > cap ? (int)cap : n);
}

// Sum over the 8 lanes of an aligned lane group with DPP moves: pairs
// (l, l^1), then (l, l^2) inside quads, then the two quads of the group
// (row_half_mirror pairs lane i with lane 7-i; both quads hold uniform
// values by then).  Every lane of the group ends with the same value, added
// in the same order as an xor-1/2/4 shuffle reduction.
__device__ __forceinline__ int32_t group8_sum(int32_t v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm(1,0,3,2)
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm(2,3,0,1)
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  return v;
}

__device__ __forceinline__ float group8_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
  return v;
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}


// ------------------------------------------------------------------ hist
// The pair counts are taken at the end of the route kernel, per query, once
// its list is final (pair_hist_wave): hist[c] counts cluster c's pairs.  They
// start a search at zero: the prep clears the counts it read, so only a fresh
// workspace needs the full clear below (hist_words(n_clusters) words, whole
// 32-count words past the last cluster included).
hipError_t launch_shared_hist(const SharedArgs &a, bool fresh, hipStream_t s) {
  if (!fresh) return hipSuccess;
  return launch_fill_i32((int32_t *)a.hist, hist_words(a.n_clusters), 0, s);
}

PairHistArgs pair_hist_args(const SharedArgs &a) {
  PairHistArgs h;
  h.hist = a.hist;
  h.cl_off = a.cl_off;
  h.n_clusters = a.n_clusters;
  h.seed_min = a.seed_min;
  h.cseed = a.cseed;
  h.rfull = a.rfull;
  h.qnorm = a.qnorm;
  h.queries = (const unsigned char *)a.queries;
  h.row_bytes = a.row_bytes;
  h.scan_head = a.scan_head;
  h.is_u8 = a.is_u8;
  h.eager_rows = a.eager_rows;
  h.pair_rank = a.pair_rank;
  h.cap = a.cap;
  return h;
}

// ------------------------------------------------------------------ prep
// The scan list holds the clusters with pairs in cluster order, each with
// its pair range in pair_q and its range in the scan's work space (rows x
// groups of <= g queries).  It is built from the pair counts themselves:
// one coalesced pass over them (4 bytes per index cluster, read 32 counts =
// one 128-byte word per thread) plus work per listed cluster, with no
// per-pair atomics to mark the clusters:
//   count  thread t of block b owns LIST_WPT words of 32 counts; it sums
//          entries, pairs and work over its nonzero counts (block sums too);
//   scan   one block turns the block sums into exclusive offsets and the
//          totals (list length, pairs, work);
//   emit   each thread scans its block's thread sums, walks its nonzero
//          counts again and writes its entries, each cluster's pair start
//          (for the scatter), and clears those counts for the next search;
//   scatter one wave per query puts each pair at its cluster's start plus
//          the rank its counting atomic returned.

// bit b set: cluster 32 wi + b has pairs.  The counts array holds whole
// words (hist_words), so each word is read as eight 16-byte loads.
__device__ __forceinline__ uint32_t hist_word_bits(const SharedArgs &a, int64_t wi) {
  const uint4 *p = reinterpret_cast<const uint4 *>(a.hist + wi * 32);
  uint32_t bits = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint4 v = p[k];
    bits |= ((v.x != 0u ? 1u : 0u) | (v.y != 0u ? 2u : 0u) | (v.z != 0u ? 4u : 0u) |
             (v.w != 0u ? 8u : 0u)) << (4 * k);
  }
  return bits;
}

struct ListSums {
  uint32_t n, h;
  uint64_t w;
};

__device__ __forceinline__ ListSums list_thread_sums(const SharedArgs &a, int64_t w0,
                                                     int64_t nwords) {
  ListSums r{0u, 0u, 0ull};
  for (int j = 0; j < LIST_WPT; ++j) {
    const int64_t wi = w0 + j;
    if (wi >= nwords) break;
    uint32_t bits = hist_word_bits(a, wi);
    while (bits) {
      const uint64_t c = (uint64_t)wi * 32 + (uint64_t)(__ffs(bits) - 1);
      bits &= bits - 1;
      const uint32_t hc = a.hist[c];
      const uint64_t sz = a.cl_off[c + 1] - a.cl_off[c];
      r.n += 1;
      r.h += hc;
      r.w += (uint64_t)((hc + a.g - 1) / a.g) * sz;
    }
  }
  return r;
}

// block-wide exclusive scan of (n, h, w) over LIST_THREADS threads; returns
// the thread's exclusive prefix and writes the block total to *tot
__device__ __forceinline__ ListSums list_block_scan(ListSums v, ListSums *tot) {
  __shared__ uint32_t sn[LIST_THREADS / WAVE], sh[LIST_THREADS / WAVE];
  __shared__ uint64_t sw[LIST_THREADS / WAVE];
  const int lane = lane_id(), wv = threadIdx.x / WAVE;
  const uint32_t in = wave_incl_scan_u32(v.n), ih = wave_incl_scan_u32(v.h);
  const uint64_t iw = wave_incl_scan_u64(v.w);
  if (lane == WAVE - 1) {
    sn[wv] = in;
    sh[wv] = ih;
    sw[wv] = iw;
  }
  __syncthreads();
  uint32_t bn = 0, bh = 0;
  uint64_t bw = 0;
  ListSums t{0u, 0u, 0ull};
  for (int i = 0; i < LIST_THREADS / WAVE; ++i) {
    if (i == wv) {
      bn = t.n;
      bh = t.h;
      bw = t.w;
    }
    t.n += sn[i];
    t.h += sh[i];
    t.w += sw[i];
  }
  *tot = t;
  return ListSums{bn + in - v.n, bh + ih - v.h, bw + iw - v.w};
}

__global__ void __launch_bounds__(LIST_THREADS) k_list_count(SharedArgs a) {
  const int64_t nwords = list_words(a.n_clusters);
  const int64_t t = (int64_t)blockIdx.x * LIST_THREADS + threadIdx.x;
  const ListSums v = list_thread_sums(a, t * LIST_WPT, nwords);
  a.thr_n[t] = v.n;
  a.thr_h[t] = v.h;
  a.thr_w[t] = v.w;
  ListSums tot;
  (void)list_block_scan(v, &tot);
  if (threadIdx.x == 0) {
    a.blk_n[blockIdx.x] = tot.n;
    a.blk_h[blockIdx.x] = tot.h;
    a.blk_w[blockIdx.x] = tot.w;
  }
}

// one block: exclusive offsets of the blocks' sums, in place, and the totals
__global__ void __launch_bounds__(LIST_THREADS) k_list_scan(SharedArgs a, int64_t nblk) {
  const int64_t per = (nblk + LIST_THREADS - 1) / LIST_THREADS;
  const int64_t b0 = (int64_t)threadIdx.x * per;
  const int64_t b1 = b0 + per < nblk ? b0 + per : nblk;
  ListSums v{0u, 0u, 0ull};
  for (int64_t b = b0; b < b1; ++b) {
    v.n += a.blk_n[b];
    v.h += a.blk_h[b];
    v.w += a.blk_w[b];
  }
  ListSums tot;
  ListSums run = list_block_scan(v, &tot);
  for (int64_t b = b0; b < b1; ++b) {
    const ListSums x{a.blk_n[b], a.blk_h[b], a.blk_w[b]};
    a.blk_n[b] = run.n;
    a.blk_h[b] = run.h;
    a.blk_w[b] = run.w;
    run.n += x.n;
    run.h += x.h;
    run.w += x.w;
  }
  if (threadIdx.x == 0) {
    a.lmeta[0] = tot.n;       // list length
    a.lmeta[1] = tot.h;       // pairs
    a.lmeta[2] = tot.w;       // work
    a.swork_off[tot.n] = tot.w;
  }
}

// Each wave first gathers the clusters of its 64 words into a compact list in
// LDS (at most 64 x 32), then writes their entries with consecutive lanes on
// consecutive entries, so the list arrays are written in whole lines; the
// entries' pair and work offsets come from wave prefix sums, round by round.
__global__ void __launch_bounds__(LIST_THREADS) k_list_emit(SharedArgs a) {
  static_assert(LIST_WPT == 1, "one word of 32 counts per thread");
  __shared__ uint32_t s_cl[LIST_THREADS / WAVE][WAVE * 32];
  const int64_t nwords = list_words(a.n_clusters);
  const int64_t t = (int64_t)blockIdx.x * LIST_THREADS + threadIdx.x;
  const int lane = lane_id(), wv = threadIdx.x / WAVE;
  const ListSums v{a.thr_n[t], a.thr_h[t], a.thr_w[t]};
  ListSums tot;
  const ListSums ex = list_block_scan(v, &tot);
  // the wave's first entry and its pair and work offsets
  const uint32_t n0 = bcast_u32(ex.n, 0);
  const uint32_t nend = bcast_u32(ex.n + v.n, WAVE - 1);
  uint32_t *cl = s_cl[wv];
  if (t < nwords) {
    uint32_t bits = hist_word_bits(a, t);
    uint32_t o = ex.n - n0;
    while (bits) {
      cl[o++] = (uint32_t)t * 32u + (uint32_t)(__ffs(bits) - 1);
      bits &= bits - 1;
    }
  }
  __builtin_amdgcn_wave_barrier();
  const uint32_t ibase = a.blk_n[blockIdx.x] + n0;
  uint32_t hrun = a.blk_h[blockIdx.x] + bcast_u32(ex.h, 0);
  uint64_t wrun = a.blk_w[blockIdx.x] + bcast_u64(ex.w, 0);
  const uint32_t cnt = nend - n0;
  for (uint32_t e0 = 0; e0 < cnt; e0 += WAVE) {
    const uint32_t e = e0 + (uint32_t)lane;
    const bool ok = e < cnt;
    const uint64_t c = ok ? cl[e] : 0u;
    const uint32_t hc = ok ? a.hist[c] : 0u;
    const uint64_t base = ok ? a.cl_off[c] : 0u;
    const uint64_t sz = ok ? a.cl_off[c + 1] - base : 0u;
    const uint64_t work = (uint64_t)((hc + a.g - 1) / a.g) * sz;
    const uint32_t ih = wave_incl_scan_u32(hc);
    const uint64_t iw = wave_incl_scan_u64(work);
    if (ok) {
      const uint32_t i = ibase + e;
      const uint32_t hp = hrun + ih - hc;
      a.hist[c] = 0u;
      a.slist[i] = (uint32_t)c;
      a.lbase[i] = base;
      a.lsz[i] = (uint32_t)sz;
      a.lpair[i] = hp;
      a.lpm[i] = hc;
      a.swork_off[i] = wrun + iw - work;
      a.hpos[c] = hp;
    }
    hrun += bcast_u32(ih, WAVE - 1);
    wrun += bcast_u64(iw, WAVE - 1);
  }
}

// one wave per query: each of the query's pairs into its cluster's slots, at
// the rank its count returned
__global__ void __launch_bounds__(256) k_pair_scatter(SharedArgs a) {
  const int lane = lane_id();
  const int64_t q = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (q >= a.nq) return;
  const int n = clamp_n(a.nclus[q], a.cap);
  const uint32_t *cl = a.clus + q * a.cap;
  const uint32_t *rank = a.pair_rank + q * a.cap;
  for (int i = a.cseed[q] + lane; i < n; i += WAVE) {
    const uint32_t c = cl[i];
    if (c < a.n_clusters) {
      const uint64_t pos = (uint64_t)a.hpos[c] + rank[i];
      if (pos < (uint64_t)a.nq * (uint64_t)a.cap) a.pair_q[pos] = (uint32_t)q;
    }
  }
}

hipError_t launch_shared_prep(const SharedArgs &a, hipStream_t s) {
  hipError_t e = launch_fill_i32(a.scnt, a.nq, 0, s);
  if (e == hipSuccess) e = launch_fill_i32(a.flag, a.nq, 0, s);
  if (e == hipSuccess) e = launch_fill_i32((int32_t *)(a.wstats + 3), 6, 0, s);
  if (e == hipSuccess) e = launch_fill_i32((int32_t *)a.pool_cnt, 2, 0, s);
  if (e == hipSuccess) e = launch_fill_i32((int32_t *)a.open_cnt, 2, 0, s);
  if (e == hipSuccess) e = launch_fill_i32((int32_t *)a.counter, 2, 0, s);
  if (e != hipSuccess) return e;
  const int64_t nblk = list_blocks(a.n_clusters);
  hipLaunchKernelGGL(k_list_count, dim3((unsigned)nblk), dim3(LIST_THREADS), 0, s, a);
  hipLaunchKernelGGL(k_list_scan, dim3(1), dim3(LIST_THREADS), 0, s, a, nblk);
  hipLaunchKernelGGL(k_list_emit, dim3((unsigned)nblk), dim3(LIST_THREADS), 0, s, a);
  if (a.nq > 0)
    hipLaunchKernelGGL(k_pair_scatter, dim3((unsigned)((a.nq + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// one wave per query: rows of its whole list (diagnostics)
__global__ void __launch_bounds__(256) k_list_rows(const uint32_t *clus, const int32_t *nclus,
                                                   int64_t cap, int64_t nq, const uint64_t *cl_off,
                                                   int64_t n_clusters, uint32_t *rows) {
  const int lane = lane_id();
  const int64_t q = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (q >= nq) return;
  const int n = clamp_n(nclus[q], cap);
  uint64_t sum = 0;
  for (int i = lane; i < n; i += WAVE) {
    const uint32_t c = clus[q * cap + i];
    if (c < n_clusters) sum += cl_off[(uint64_t)c + 1] - cl_off[c];
  }
  for (int m = 32; m >= 1; m >>= 1) sum += shfl_xor_u64(sum, m);
  if (lane == 0) rows[q] = sum > 0xffffffffull ? 0u : (uint32_t)sum;
}

hipError_t launch_list_rows(const uint32_t *clus, const int32_t *nclus, int64_t cap, int64_t nq,
                            const uint64_t *cl_off, int64_t n_clusters, uint32_t *rows,
                            hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_list_rows, dim3((unsigned)((nq + 3) / 4)), dim3(256), 0, s, clus, nclus,
                     cap, nq, cl_off, n_clusters, rows);
  return hipGetLastError();
}

// ------------------------------------------------------------------ survivors
// one survivor of query q: its own slots first, then the shared pool; a
// survivor that finds the pool full is lost, so its query is flagged and
// recomputed by the per-query schedule
__device__ __forceinline__ void add_survivor(const SharedArgs &a, uint32_t q, uint32_t key,
                                             int64_t id) {
  const int pos = atomicAdd(&a.scnt[q], 1);
  if (pos < SURVIVOR_CAP) {
    a.skey[(int64_t)q * SURVIVOR_CAP + pos] = key;
    a.sid[(int64_t)q * SURVIVOR_CAP + pos] = id;
    return;
  }
  const unsigned long long pp = atomicAdd(a.pool_cnt, 1ull);
  if (pp < SURVIVOR_POOL) {
    a.pool_q[pp] = q;
    a.pool_key[pp] = key;
    a.pool_id[pp] = id;
  } else {
    a.flag[q] = 1;
  }
}

// ------------------------------------------------------------------ scan
// The work of scan-list entry i (cluster slist[i]) is swork[i] = rows x query
// groups; a unit (group gi, row chunk ch) starts at swork_off[i] + gi * rows +
// ch * R.  A tile is a SHARED_TILE-long range of that work space and takes the
// units that start inside it, so each unit belongs to exactly one tile.  A
// wave gathers up to SCAN_UMAX consecutive units of its tile (with up to 32
// query slots for 128-byte rows, fewer for longer ones) into a batch whose
// rows form one virtual row range; the batch's query rows sit in LDS:
//   phase A  HL lanes read the head of one virtual row (16 B each) and test it
//            against every query of its unit: the head's part of the squared
//            distance only grows with the rest of the row, so a row whose head
//            part already exceeds the query's bound cannot enter its top-k
//            (fp32 keeps a relative margin of 1e-4 for rounding); rows with any
//            query left go to an LDS list as (unit, row, query mask);
//   phase B  8 lanes per listed row (several rows in flight per lane group)
//            load the whole row and compute the exact distance for the listed
//            queries in the same arithmetic and order as k_refine; rows at or
//            before the query's bound become survivors.
// Rows longer than 8 x 128 bytes hold only one 1 KB slab of each query row in
// LDS at a time (slab partials are reduced over the 8 lanes and added in slab
// order, as k_refine does for such rows).  uint8 rows: phase B runs slab by
// slab over the listed rows, keeps every (row, query) pair's running sums in
// LDS, and tests the survivors after the last slab.  fp32 rows: phase B runs
// the first slab only; a pair whose sum is still at or before its bound goes
// to the open list, which k_scan_open finishes.
constexpr int SCAN_UMAX = 64;    // units per batch

template <int HL>
__device__ __forceinline__ int32_t head_sum(int32_t v) {
  if (HL >= 2) v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  if (HL >= 4) v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  if (HL >= 8) v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  return v;
}

template <int HL>
__device__ __forceinline__ float head_sum(float v) {
  if (HL >= 2) v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  if (HL >= 4) v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  if (HL >= 8) v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
  return v;
}

// exact key of one (row, query) pair from 8 lanes' 16-byte slices: the same
// arithmetic and reduction order as k_refine
template <int IS_U8, int NSEG>
__device__ __forceinline__ uint32_t pair_key(const uint4 *xv, const uint4 *qv, int32_t xx,
                                             int32_t qq) {
  if (IS_U8) {
    uint32_t xq = 0;
#pragma unroll
    for (int s = 0; s < NSEG; ++s) {
      xq = __builtin_amdgcn_udot4(xv[s].x, qv[s].x, xq, false);
      xq = __builtin_amdgcn_udot4(xv[s].y, qv[s].y, xq, false);
      xq = __builtin_amdgcn_udot4(xv[s].z, qv[s].z, xq, false);
      xq = __builtin_amdgcn_udot4(xv[s].w, qv[s].w, xq, false);
    }
    return (uint32_t)(group8_sum(xx - 2 * (int32_t)xq) + qq);
  }
  float acc = 0.0f;
#pragma unroll
  for (int s = 0; s < NSEG; ++s) {
    const float t0 = __uint_as_float(xv[s].x) - __uint_as_float(qv[s].x);
    const float t1 = __uint_as_float(xv[s].y) - __uint_as_float(qv[s].y);
    const float t2 = __uint_as_float(xv[s].z) - __uint_as_float(qv[s].z);
    const float t3 = __uint_as_float(xv[s].w) - __uint_as_float(qv[s].w);
    acc = fmaf(t0, t0, acc);
    acc = fmaf(t1, t1, acc);
    acc = fmaf(t2, t2, acc);
    acc = fmaf(t3, t3, acc);
  }
  return __float_as_uint(group8_sum(acc));
}

template <int IS_U8, int NSEG, int HL, int U>
__global__ void __launch_bounds__(256, NSEG <= 1 ? NR_SCAN_WAVES1 : (NSEG > 8 ? 2 : 1))
    k_scan(SharedArgs a) {
  constexpr bool LONG = NSEG > 8;            // query rows staged a 1 KB slab at a time
  constexpr int RPW = WAVE / HL;             // virtual rows per phase-A load
  constexpr int STEP = RPW * U;              // virtual rows per phase-A pass
  constexpr int SCAP = STEP + NR_SCAN_SLACK;  // listed rows before phase B runs
  constexpr int G = SHARED_G;
  constexpr int QCH = LONG ? 64 : NSEG * 8;  // 16-byte chunks of a (padded) query row or slab
  constexpr int QMAX = NSEG <= 1 ? NR_SCAN_QMAX1 : (NSEG <= 2 ? 16 : 8);  // query slots per batch
  constexpr int UB = NSEG <= 1 ? NR_SCAN_UB1 : (NSEG <= 4 || (LONG && IS_U8) ? 2 : 1);  // phase-B rows per lane group
  static_assert(QMAX <= WAVE, "one query slot per lane");
  static_assert(!LONG || QMAX == G, "a long-row slab holds one unit's queries per slot");
  constexpr int NSB = LONG ? 1 : NSEG;       // segments held per row by the short-row phase B
  __shared__ uint64_t s_ub[4][SCAN_UMAX];        // unit: first payload row
  __shared__ uint32_t s_uv[4][SCAN_UMAX + 1];    // unit: first virtual row
  __shared__ uint32_t s_uq[4][SCAN_UMAX];        // unit: first query slot | queries << 16
  __shared__ uint4 s_q[4][QMAX * QCH];           // the batch's query rows (zero padded)
  __shared__ int32_t s_th[4][QMAX];              // phase-A bound (int32 or fp32 bits)
  __shared__ uint32_t s_tk[4][QMAX];             // k-th key of the query's own pass
  __shared__ uint32_t s_qi[4][QMAX];             // query id
  __shared__ int32_t s_qq[4][QMAX];              // |q|^2 (uint8)
  __shared__ uint32_t s_sv[4][SCAP];             // listed rows: unit << 20 | row << 8 | mask
  __shared__ uint8_t s_umap[4][WAVE];            // batch formation: unit -> staged entry
  __shared__ uint32_t s_pslot[4][QMAX];          // batch formation: slot -> pair index
  __shared__ uint32_t s_run[4][LONG && IS_U8 ? SCAP * G : 1];  // long uint8 rows: running x.q per (listed row, query)
  constexpr int OPENL = 128;                     // long fp32 rows: open pairs held before they go out
  __shared__ uint32_t s_ol[4][LONG && !IS_U8 ? OPENL : 1];  // listed row << 8 | query slot
  __shared__ uint32_t s_ok[4][LONG && !IS_U8 ? OPENL : 1];  // its first slab's sum
  __shared__ int32_t s_runx[4][LONG && IS_U8 ? SCAP : 1];  // long uint8 rows: running |x|^2
  const int lane = lane_id();
  const int w = threadIdx.x >> 6;
  const int grp = lane >> 3;  // phase B: 8 lanes per row
  const int gl = lane & 7;
  const int hl = lane % HL;   // phase A: HL lanes per row
  uint64_t *ub = s_ub[w];
  uint32_t *uv = s_uv[w];
  uint32_t *uq = s_uq[w];
  uint4 *qs = s_q[w];
  int32_t *th = s_th[w];
  uint32_t *tk = s_tk[w];
  uint32_t *qi = s_qi[w];
  int32_t *qqs = s_qq[w];
  uint32_t *sv = s_sv[w];
  uint8_t *umap = s_umap[w];
  uint32_t *pslot = s_pslot[w];
  uint32_t *run = s_run[w];
  int32_t *runx = s_runx[w];
  uint32_t *ol = s_ol[w];
  uint32_t *olk = s_ok[w];
  const int64_t NS = (int64_t)a.lmeta[0];
  const uint64_t W = a.lmeta[2];
  const uint64_t ntiles = (W + SHARED_TILE - 1) / SHARED_TILE;
  const int rb = a.row_bytes;
  const int k = a.k;
  const unsigned char *queries = (const unsigned char *)a.queries;
  unsigned long long full_rows = 0, body_bytes = 0;
  uint32_t nbatch = 0, tested_batches = 0;  // direct batches: see below
  uint64_t tested_rows = 0, open_rows = 0;
  if (ntiles == 0) return;

  for (;;) {
    unsigned long long t = 0;
    if (lane == 0) t = atomicAdd(a.counter, 1ull);
    t = bcast_u64(t, 0);
    if (t >= ntiles) break;
    const uint64_t ws = (uint64_t)t * SHARED_TILE;
    const uint64_t we = ws + SHARED_TILE < W ? ws + SHARED_TILE : W;
    // the list entry holding ws: the last i with swork_off[i] <= ws (64-ary search)
    int64_t lo = 0, hi = NS;
    while (hi - lo > 1) {
      const int64_t step = (hi - lo + WAVE - 1) / WAVE;
      const int64_t pos = lo + (int64_t)lane * step;
      const bool pred = lane > 0 && pos < hi && a.swork_off[pos] <= ws;
      const uint64_t m = ballot(pred);
      const int last = m ? 63 - __clzll((long long)m) : 0;
      const int64_t nlo = lo + (int64_t)last * step;
      const int64_t nhi = nlo + step < hi ? nlo + step : hi;
      lo = nlo;
      hi = nhi;
    }
    // the first unit of entry i = lo that starts at or after ws: unit uo of
    // the entry, units numbered group-major (gi * nch + ch).  The entry
    // holding ws has work, so sz > 0; the guard keeps the division defined.
    int64_t i = lo;
    uint32_t uo = 0;
    {
      const uint64_t wo0 = a.swork_off[i];
      const uint64_t sz0 = a.lsz[i];
      const uint32_t m0 = a.lpm[i];
      if (sz0 > 0) {
        const uint64_t rel = ws - wo0;
        uint64_t gi0 = rel / sz0;
        uint64_t ch0 = (rel - gi0 * sz0 + SHARED_ROWS - 1) / SHARED_ROWS;
        const uint64_t nch0 = (sz0 + SHARED_ROWS - 1) / SHARED_ROWS;
        if (ch0 >= nch0) {
          ch0 = 0;
          ++gi0;
        }
        if (gi0 >= (m0 + G - 1) / G) {
          ++i;
        } else {
          uo = (uint32_t)(gi0 * nch0 + ch0);
        }
      } else {
        ++i;
      }
    }

    for (;;) {
      // ---- a batch: the units of this tile from (i, uo) on, one per lane,
      // while their query slots fit.  Lane j stages entry i + j; the units of
      // the staged entries are numbered by a prefix sum and lane u takes unit u
      if (i >= NS) break;
      int lnb = lane;
      // the lane id made opaque here, so the addresses derived from it in the
      // batch setup are recomputed per batch rather than kept live (and
      // spilled) across the whole kernel
      __asm__ volatile("" : "+v"(lnb));
      const int64_t e = i + lnb;
      uint64_t ewo = 0, ebase = 0;
      uint32_t esz = 0, ehp = 0, em = 0;
      if (e < NS) {
        ewo = a.swork_off[e];
        ebase = a.lbase[e];
        esz = a.lsz[e];
        ehp = a.lpair[e];
        em = a.lpm[e];
      }
      const uint32_t enc = (esz + SHARED_ROWS - 1) / SHARED_ROWS;
      const uint32_t eun = enc * ((em + G - 1) / G) - (lnb == 0 ? uo : 0u);
      const uint32_t eincl = wave_incl_scan_u32(eun);
      const uint32_t eexcl = eincl - eun;
      // unit -> staged entry, for the first 64 units
      for (uint32_t x = eexcl; x < eincl && x < (uint32_t)WAVE; ++x) umap[x] = (uint8_t)lnb;
      __builtin_amdgcn_wave_barrier();
      const uint32_t all_u = bcast_u32(eincl, WAVE - 1);
      const uint32_t avail = all_u < (uint32_t)WAVE ? all_u : (uint32_t)WAVE;
      if (avail == 0) {
        // 64 entries without units (or the end of the list)
        i += WAVE;
        uo = 0;
        continue;
      }
      const bool uok = (uint32_t)lnb < avail;
      const int ej = uok ? (int)umap[lnb] : 0;
      const uint64_t uwo = shfl_u64(ewo, ej);
      const uint64_t ubase = shfl_u64(ebase, ej);
      const uint32_t usz = (uint32_t)__shfl((int)esz, ej);
      const uint32_t uhp = (uint32_t)__shfl((int)ehp, ej);
      const uint32_t um = (uint32_t)__shfl((int)em, ej);
      const uint32_t unc = (uint32_t)__shfl((int)enc, ej);
      const uint32_t uidx = (uint32_t)lnb - (uint32_t)__shfl((int)eexcl, ej) + (ej == 0 ? uo : 0u);
      const uint32_t ugi = uok ? uidx / unc : 0u;
      const uint32_t uch = uidx - ugi * unc;
      const uint32_t ugm = uok ? (um - ugi * G < (uint32_t)G ? um - ugi * G : (uint32_t)G) : 0u;
      const uint32_t urows = uok ? (usz - uch * SHARED_ROWS < SHARED_ROWS ? usz - uch * SHARED_ROWS
                                                                            : SHARED_ROWS)
                                 : 0u;
      const uint64_t ustart = uwo + (uint64_t)ugi * usz + (uint64_t)uch * SHARED_ROWS;
      const uint32_t sincl = wave_incl_scan_u32(ugm);
      // the units taken: a prefix (unit starts and slot counts only grow)
      const uint64_t nofit = ballot(!(uok && ustart < we && sincl <= (uint32_t)QMAX));
      const int nu = nofit ? __ffsll((unsigned long long)nofit) - 1 : WAVE;
      if (nu == 0) break;  // the next unit starts past this tile
      const bool take = lnb < nu;
      const uint32_t vincl = wave_incl_scan_u32(take ? urows : 0u);
      const uint32_t vtot = bcast_u32(vincl, nu - 1);
      const int nqs = (int)bcast_u32(sincl, nu - 1);
      int gmax = 0;
      {
        uint32_t g = take ? ugm : 0u;
        for (int o = 32; o >= 1; o >>= 1) {
          const uint32_t h = (uint32_t)__shfl_xor((int)g, o);
          g = h > g ? h : g;
        }
        gmax = (int)g;
      }
      if (take) {
        ub[lnb] = ubase + (uint64_t)uch * SHARED_ROWS;
        uv[lnb] = vincl - urows;
        uq[lnb] = (sincl - ugm) | (ugm << 16);
        // slots of this unit: its pairs (the query of slot s is pair_q[pslot[s]])
        for (uint32_t t = 0; t < ugm; ++t) pslot[sincl - ugm + t] = uhp + ugi * G + t;
      }
      if (lnb == 0) uv[nu] = vtot;
      __builtin_amdgcn_wave_barrier();
      const uint32_t myq = lnb < nqs ? a.pair_q[pslot[lnb]] : 0u;
      // where the next batch starts: the entry holding unit nu (units of the
      // staged entries beyond the first 64 included), else past them
      {
        const uint64_t hold = ballot(e < NS && eexcl <= (uint32_t)nu && (uint32_t)nu < eincl);
        if (hold) {
          const int j = __ffsll((unsigned long long)hold) - 1;
          uo = (uint32_t)nu - bcast_u32(eexcl, j) + (j == 0 ? uo : 0u);
          i += j;
        } else {
          i += WAVE;
          uo = 0;
        }
      }
      // ---- the batch's queries: rows into LDS, bounds, |q|^2 (one slot per
      // lane).  myq is a valid query id in every lane (0 in lanes without a
      // slot), so all loads go out unconditionally and together; what lies
      // past the batch's slots or the row is replaced by zeros afterwards
      constexpr int QL = QMAX * QCH / WAVE;
      static_assert(QMAX * QCH % WAVE == 0, "whole loads of query chunks");
      uint4 qload[QL];
#pragma unroll
      for (int t = 0; t < QL; ++t) {
        const int c = t * WAVE + lnb;
        const int sl = c / QCH;
        const int off = (c - sl * QCH) * 16;
        const uint32_t qsl = (uint32_t)__shfl((int)myq, sl);
        qload[t] = *(const uint4 *)(queries + (uint64_t)qsl * rb + (off < rb ? off : 0));
      }
      const uint4 rec = a.qrec[myq];
#pragma unroll
      for (int t = 0; t < QL; ++t) {
        const int c = t * WAVE + lnb;
        const int sl = c / QCH;
        const int off = (c - sl * QCH) * 16;
        qs[c] = sl < nqs && off < rb ? qload[t] : make_uint4(0, 0, 0, 0);
      }
      if (lnb < nqs) {
        qi[lnb] = myq;
        tk[lnb] = rec.x;
        th[lnb] = (int32_t)rec.y;
        qqs[lnb] = (int32_t)rec.z;
      }
      __builtin_amdgcn_wave_barrier();

      // ---- phase B: whole rows of the listed (row, queries), UB rows per lane group
      auto phase_b_short = [&](int nsv) __attribute__((always_inline)) {
        for (int e0 = 0; e0 < nsv; e0 += 8 * UB) {
          uint32_t ent[UB];
          uint64_t row[UB];
          uint4 xv[UB][NSB];
#pragma unroll
          for (int b = 0; b < UB; ++b) {
            const int e = e0 + 8 * b + grp;
            ent[b] = e < nsv ? sv[e] : 0u;
            row[b] = ub[ent[b] >> 20] + ((ent[b] >> 8) & 0xfffu);
#pragma unroll
            for (int s = 0; s < NSB; ++s) {
              const int off = 128 * s + 16 * gl;
              xv[b][s] = ((ent[b] & 0xffu) && off < rb) ? load_stream(a.ra.seg(row[b], off))
                                                       : make_uint4(0, 0, 0, 0);
            }
          }
          // the query slots any of this round's rows lists (of gmax)
          uint32_t jset = 0;
          {
            uint32_t lm = 0;
#pragma unroll
            for (int b = 0; b < UB; ++b) lm |= ent[b] & 0xffu;
            for (int j = 0; j < gmax; ++j)
              if (ballot(((lm >> j) & 1u) != 0)) jset |= 1u << j;
          }
#pragma unroll
          for (int b = 0; b < UB; ++b) {
            const uint32_t mask = ent[b] & 0xffu;
            if (!ballot(mask != 0)) continue;
            int32_t xx = 0;
            if (IS_U8) {
              uint32_t acc = 0;
#pragma unroll
              for (int s = 0; s < NSB; ++s) {
                acc = __builtin_amdgcn_udot4(xv[b][s].x, xv[b][s].x, acc, false);
                acc = __builtin_amdgcn_udot4(xv[b][s].y, xv[b][s].y, acc, false);
                acc = __builtin_amdgcn_udot4(xv[b][s].z, xv[b][s].z, acc, false);
                acc = __builtin_amdgcn_udot4(xv[b][s].w, xv[b][s].w, acc, false);
              }
              xx = (int32_t)acc;
            }
            const int slot0 = (int)(uq[ent[b] >> 20] & 0xffffu);
            for (uint32_t js = jset; js; js &= js - 1) {
              const int j = __ffs(js) - 1;
              const bool bit = ((mask >> j) & 1u) != 0;
              if (!ballot(bit)) continue;
              const int slot = slot0 + (bit ? j : 0);
              uint4 qv[NSB];
#pragma unroll
              for (int s = 0; s < NSB; ++s) qv[s] = qs[slot * QCH + 8 * s + gl];
              const uint32_t key = pair_key<IS_U8, NSB>(xv[b], qv, xx, qqs[slot]);
              // at or before the bound: a survivor (ties included; the merge orders them)
              if (bit && gl == 0 && key <= tk[slot]) {
                add_survivor(a, qi[slot], key, a.row_ids[row[b]]);
              }
            }
          }
        }
        full_rows += (unsigned long long)nsv;
        body_bytes += (unsigned long long)nsv * (uint32_t)rb;
      };

      // ---- phase B for long rows, slab by slab.  Lane c of a slab load holds
      // 16-byte chunk c of slot t's slab (slot t's query id is qi[t])
      auto stage_slab = [&](int s0) __attribute__((always_inline)) {
        __builtin_amdgcn_wave_barrier();  // every read of the previous slab is done
        uint4 sl[QMAX];
#pragma unroll
        for (int t = 0; t < QMAX; ++t) {
          const int off = 128 * s0 + 16 * lane;
          sl[t] = t < nqs && off < rb
                      ? *(const uint4 *)(queries + (uint64_t)qi[t] * rb + off)
                      : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < QMAX; ++t) qs[t * QCH + lane] = sl[t];
        __builtin_amdgcn_wave_barrier();
      };
      auto phase_b_long = [&](int nsv) __attribute__((always_inline)) {
        const int nsl = (rb + 1023) / 1024;
        // uint8 rows are finished here, slab by slab; for fp32 rows only the
        // first slab is, and the pairs it leaves at or before their bound go
        // to the open list (their running sums are bounds: see below)
        const int nslk = IS_U8 ? nsl : 1;
        full_rows += (unsigned long long)nsv;
        // fp32: the open pairs, collected in LDS and sent out with one atomic
        // per OPENL of them; a pair that finds the open list full flags its
        // query for recomputation
        int nopen = 0;
        auto flush_open = [&]() __attribute__((always_inline)) {
          __builtin_amdgcn_wave_barrier();
          unsigned long long base = 0;
          if (lane == 0) base = atomicAdd(a.open_cnt, (unsigned long long)nopen);
          base = bcast_u64(base, 0);
          for (int i = lane; i < nopen; i += WAVE) {
            const uint32_t v = ol[i];
            const int slot = (int)(v & 0xffu);
            const uint32_t ent = sv[v >> 8];
            const uint64_t row = ub[ent >> 20] + ((ent >> 8) & 0xfffu);
            const unsigned long long p = base + (unsigned long long)i;
            if (p < OPEN_PAIRS) {
              a.open_q[p] = qi[slot];
              a.open_key[p] = olk[i];
              a.open_row[p] = row;
            } else {
              a.flag[qi[slot]] = 1;
            }
          }
          nopen = 0;
          __builtin_amdgcn_wave_barrier();
        };
        for (int sl = 0; sl < nslk && nsv > 0; ++sl) {
          const int s0 = 8 * sl;
          if (sl > 0) stage_slab(s0);
          body_bytes += (unsigned long long)nsv * (uint32_t)(rb - 1024 * sl < 1024 ? rb - 1024 * sl : 1024);
          for (int e0 = 0; e0 < nsv; e0 += 8 * UB) {
            uint32_t ent[UB];
            uint64_t row[UB];
            uint4 xv[UB][8];
#pragma unroll
            for (int b = 0; b < UB; ++b) {
              const int e = e0 + 8 * b + grp;
              ent[b] = e < nsv ? sv[e] : 0u;
              row[b] = ub[ent[b] >> 20] + ((ent[b] >> 8) & 0xfffu);
#pragma unroll
              for (int s = 0; s < 8; ++s) {
                const int off = 128 * (s0 + s) + 16 * gl;
                xv[b][s] = ((ent[b] & 0xffu) && off < rb) ? load_stream(a.ra.seg(row[b], off))
                                                         : make_uint4(0, 0, 0, 0);
              }
            }
#pragma unroll
            for (int b = 0; b < UB; ++b) {
              const uint32_t mask = ent[b] & 0xffu;
              if (!ballot(mask != 0)) continue;
              const int e = e0 + 8 * b + grp;
              if (IS_U8) {
                uint32_t acc = 0;
#pragma unroll
                for (int s = 0; s < 8; ++s) {
                  acc = __builtin_amdgcn_udot4(xv[b][s].x, xv[b][s].x, acc, false);
                  acc = __builtin_amdgcn_udot4(xv[b][s].y, xv[b][s].y, acc, false);
                  acc = __builtin_amdgcn_udot4(xv[b][s].z, xv[b][s].z, acc, false);
                  acc = __builtin_amdgcn_udot4(xv[b][s].w, xv[b][s].w, acc, false);
                }
                const int32_t p = group8_sum((int32_t)acc);
                if (mask && gl == 0) runx[e] = sl == 0 ? p : runx[e] + p;
              }
              const int slot0 = (int)(uq[ent[b] >> 20] & 0xffffu);
              for (int j = 0; j < gmax; ++j) {
                const bool bit = ((mask >> j) & 1u) != 0;
                if (!ballot(bit)) continue;
                const int slot = slot0 + (bit ? j : 0);
                uint4 qv[8];
#pragma unroll
                for (int s = 0; s < 8; ++s) qv[s] = qs[slot * QCH + 8 * s + gl];
                uint32_t pbits;
                if (IS_U8) {
                  uint32_t xq = 0;
#pragma unroll
                  for (int s = 0; s < 8; ++s) {
                    xq = __builtin_amdgcn_udot4(xv[b][s].x, qv[s].x, xq, false);
                    xq = __builtin_amdgcn_udot4(xv[b][s].y, qv[s].y, xq, false);
                    xq = __builtin_amdgcn_udot4(xv[b][s].z, qv[s].z, xq, false);
                    xq = __builtin_amdgcn_udot4(xv[b][s].w, qv[s].w, xq, false);
                  }
                  const int32_t p = group8_sum((int32_t)xq);
                  pbits = (uint32_t)(sl == 0 ? p : (int32_t)run[bit ? e * G + j : 0] + p);
                  if (bit && gl == 0) run[e * G + j] = pbits;
                } else {
                  float acc = 0.0f;
#pragma unroll
                  for (int s = 0; s < 8; ++s) {
                    const float t0 = __uint_as_float(xv[b][s].x) - __uint_as_float(qv[s].x);
                    const float t1 = __uint_as_float(xv[b][s].y) - __uint_as_float(qv[s].y);
                    const float t2 = __uint_as_float(xv[b][s].z) - __uint_as_float(qv[s].z);
                    const float t3 = __uint_as_float(xv[b][s].w) - __uint_as_float(qv[s].w);
                    acc = fmaf(t0, t0, acc);
                    acc = fmaf(t1, t1, acc);
                    acc = fmaf(t2, t2, acc);
                    acc = fmaf(t3, t3, acc);
                  }
                  // the first slab's sum.  Later slabs only add non-negative
                  // terms, rounded to nearest, so the running sum never
                  // decreases: a pair past its bound now stays past it
                  pbits = __float_as_uint(group8_sum(acc));
                  const bool op = bit && gl == 0 && pbits <= tk[slot];
                  const uint64_t om = ballot(op);
                  if (om) {
                    const int c = popc64(om);
                    if (nopen + c > OPENL) flush_open();
                    if (op) {
                      const int i = nopen + popc64(om & lanemask_lt());
                      ol[i] = ((uint32_t)e << 8) | (uint32_t)slot;
                      olk[i] = pbits;
                    }
                    nopen += c;
                  }
                }
              }
            }
          }
          __builtin_amdgcn_wave_barrier();
        }
        if (IS_U8) {
          // the finished pairs: at or before the bound, a survivor
          for (int e = lane; e < nsv; e += WAVE) {
            const uint32_t ent = sv[e];
            const uint32_t mask = ent & 0xffu;
            const int slot0 = (int)(uq[ent >> 20] & 0xffffu);
            const uint64_t row = ub[ent >> 20] + ((ent >> 8) & 0xfffu);
            for (int j = 0; j < G; ++j) {
              if (!((mask >> j) & 1u)) continue;
              const int slot = slot0 + j;
              const uint32_t key = (uint32_t)(runx[e] - 2 * (int32_t)run[e * G + j] + qqs[slot]);
              if (key <= tk[slot]) add_survivor(a, qi[slot], key, a.row_ids[row]);
            }
          }
          if (nsl > 1 && nsv > 0) stage_slab(0);  // slab 0 back for the heads of the next rows
        } else if (nopen > 0) {
          flush_open();
        }
      };

      auto phase_b = [&](int nsv) __attribute__((always_inline)) {
        if constexpr (LONG) phase_b_long(nsv); else phase_b_short(nsv);
      };

      // ---- direct batches: when the heads this wave has tested so far (at
      // least 16 batches, drawn from across the work) left more than two
      // thirds of the rows open, list every row with all its unit's queries
      // (the head test only ever drops rows, so skipping it changes no
      // result); every 8th batch still tests
      ++nbatch;
      const bool direct = (nbatch & 7) != 0 && tested_batches >= 16 && 3 * open_rows > 2 * tested_rows;
      if (direct) {
        int nsv = 0;
        int cur = 0;
        for (uint32_t v0 = 0; v0 < vtot; v0 += WAVE) {
          if (nsv > SCAP - WAVE) {
            phase_b(nsv);
            nsv = 0;
          }
          const uint32_t v = v0 + lane;
          const bool ok = v < vtot;
          if (ok)
            while (uv[cur + 1] <= v) ++cur;
          const uint64_t m = ballot(ok);
          if (ok) {
            const uint32_t gmu = uq[cur] >> 16;
            sv[nsv + popc64(m & lanemask_lt())] =
                ((uint32_t)cur << 20) | ((v - uv[cur]) << 8) | ((1u << gmu) - 1u);
          }
          nsv += popc64(m);
        }
        phase_b(nsv);
        __builtin_amdgcn_wave_barrier();
        continue;
      }

      // ---- phase A: heads of the batch's virtual rows
      int nsv = 0;
      uint32_t listed = 0;  // rows left open by their heads
      // per lane (its virtual rows only increase): the unit holding them, its
      // first virtual and payload rows and the next unit's first virtual
      // row, kept in registers so that a load costs an LDS read only where
      // it crosses into the next unit
      int cur = 0;
      uint32_t vcur = uv[0], vnext = uv[1];
      uint64_t bcur = ub[0];
      for (uint32_t v0 = 0; v0 < vtot; v0 += STEP) {
        if (nsv > SCAP - STEP) {
          phase_b(nsv);
          nsv = 0;
        }
        uint4 hv[U];
        // the unit of each load, 6 bits apiece (units < SCAN_UMAX = 64); the
        // virtual row and its bound check are recomputed where needed
        uint64_t cpack = 0;
#pragma unroll
        for (int uu = 0; uu < U; ++uu) {
          const uint32_t v = v0 + uu * RPW + lane / HL;
          const bool ok = v < vtot;
          if (ok && vnext <= v) {
            do {
              ++cur;
              vnext = uv[cur + 1];
            } while (vnext <= v);
            vcur = uv[cur];
            bcur = ub[cur];
          }
          cpack |= (uint64_t)cur << (6 * uu);
          const uint64_t row = bcur + (v - vcur);
          hv[uu] = ok ? load_stream(reinterpret_cast<const uint4 *>(a.scan_hb + row * a.scan_hs +
                                                                     16 * hl))
                      : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int uu = 0; uu < U; ++uu) {
          const uint32_t vu = v0 + uu * RPW + lane / HL;
          const bool oku = vu < vtot;
          const int cu = (int)((cpack >> (6 * uu)) & 63u);
          int32_t xx = 0;
          if (IS_U8) {
            uint32_t acc = 0;
            acc = __builtin_amdgcn_udot4(hv[uu].x, hv[uu].x, acc, false);
            acc = __builtin_amdgcn_udot4(hv[uu].y, hv[uu].y, acc, false);
            acc = __builtin_amdgcn_udot4(hv[uu].z, hv[uu].z, acc, false);
            acc = __builtin_amdgcn_udot4(hv[uu].w, hv[uu].w, acc, false);
            xx = (int32_t)acc;
          }
          const uint32_t uqv = uq[cu];
          const int slot0 = (int)(uqv & 0xffffu);
          const int gmu = (int)(uqv >> 16);
          uint32_t mask = 0;
          for (int j = 0; j < gmax; ++j) {
            const bool valid = oku && j < gmu;
            if (!ballot(valid)) break;  // no row of this load has a j-th query
            const int slot = slot0 + (valid ? j : 0);
            const uint4 q4 = qs[slot * QCH + hl];
            bool keep;
            if (IS_U8) {
              uint32_t xq = 0;
              xq = __builtin_amdgcn_udot4(hv[uu].x, q4.x, xq, false);
              xq = __builtin_amdgcn_udot4(hv[uu].y, q4.y, xq, false);
              xq = __builtin_amdgcn_udot4(hv[uu].z, q4.z, xq, false);
              xq = __builtin_amdgcn_udot4(hv[uu].w, q4.w, xq, false);
              keep = head_sum<HL>(xx - 2 * (int32_t)xq) <= th[slot];
            } else {
              const float t0 = __uint_as_float(hv[uu].x) - __uint_as_float(q4.x);
              const float t1 = __uint_as_float(hv[uu].y) - __uint_as_float(q4.y);
              const float t2 = __uint_as_float(hv[uu].z) - __uint_as_float(q4.z);
              const float t3 = __uint_as_float(hv[uu].w) - __uint_as_float(q4.w);
              float acc = 0.0f;
              acc = fmaf(t0, t0, acc);
              acc = fmaf(t1, t1, acc);
              acc = fmaf(t2, t2, acc);
              acc = fmaf(t3, t3, acc);
              keep = head_sum<HL>(acc) <= __uint_as_float((uint32_t)th[slot]);
            }
            mask |= (valid && keep ? 1u : 0u) << j;
          }
          const bool lead = hl == 0 && mask != 0;
          const uint64_t m = ballot(lead);
          if (lead)
            sv[nsv + popc64(m & lanemask_lt())] = ((uint32_t)cu << 20) | ((vu - uv[cu]) << 8) | mask;
          nsv += popc64(m);
          listed += popc64(m);
        }
      }
      phase_b(nsv);
      ++tested_batches;
      tested_rows += vtot;
      open_rows += listed;
      __builtin_amdgcn_wave_barrier();
    }
  }
  if (lane == 0 && full_rows) atomicAdd((unsigned long long *)&a.wstats[3], full_rows);
  if (lane == 0 && body_bytes) atomicAdd((unsigned long long *)&a.wstats[4], body_bytes);
}

// The scan's record of each query, one thread per query, once the seed merge
// has written the query's own top-k: its bound (the k-th key of the seed
// pass, or all ones while that list is short), the bound the head test
// compares with, and |q|^2 for uint8 rows.  uint8 keys are integers, so the
// head bound is the key minus |q head|^2 (a row's head part of the distance
// is |x_h|^2 - 2 x_h.q_h + |q_h|^2); fp32 rows keep a relative margin of 1e-4
// over the key for the rounding of the head's partial sum.
__global__ void __launch_bounds__(256) k_scan_qrec(SharedArgs a) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= a.nq) return;
  const int k = a.k;
  const int64_t own_id = a.own_ids[q * k + k - 1];
  const float own_d = a.own_dists[q * k + k - 1];
  const uint32_t bound =
      own_id < 0 ? 0xffffffffu : (a.is_u8 ? (uint32_t)own_d : __float_as_uint(own_d));
  uint4 r;
  r.x = bound;
  r.w = 0;
  if (a.is_u8) {
    const uint2 qn = a.qnorm[q];
    r.y = (uint32_t)(bound == 0xffffffffu ? INT32_MAX
                                          : (int32_t)((int64_t)bound - (int64_t)qn.y));
    r.z = qn.x;
  } else {
    r.y = bound == 0xffffffffu ? __float_as_uint(INFINITY)
                               : __float_as_uint(__uint_as_float(bound) * 1.0001f);
    r.z = 0;
  }
  a.qrec[q] = r;
}

template <int IS_U8, int NSEG>
static hipError_t launch_scan_h(const SharedArgs &a, int hl, int grid, hipStream_t s) {
  switch (hl) {
    case 1: hipLaunchKernelGGL((k_scan<IS_U8, NSEG, 1, NR_SCAN_U1>), dim3(grid), dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_scan<IS_U8, NSEG, 2, 4>), dim3(grid), dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_scan<IS_U8, NSEG, 4, 4>), dim3(grid), dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_scan<IS_U8, NSEG, 8, 2>), dim3(grid), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int IS_U8>
static hipError_t launch_scan_t(const SharedArgs &a, int nseg, int hl, int grid, hipStream_t s) {
  if (nseg <= 1) return launch_scan_h<IS_U8, 1>(a, hl, grid, s);
  if (nseg <= 2) return launch_scan_h<IS_U8, 2>(a, hl, grid, s);
  if (nseg <= 3) return launch_scan_h<IS_U8, 3>(a, hl, grid, s);
  if (nseg <= 4) return launch_scan_h<IS_U8, 4>(a, hl, grid, s);
  if (nseg <= 8) return launch_scan_h<IS_U8, 8>(a, hl, grid, s);
  if (nseg <= 48) return launch_scan_h<IS_U8, 48>(a, hl, grid, s);
  return hipErrorInvalidValue;
}

hipError_t launch_shared_refine(const SharedArgs &a, int dtype, int n_cu, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  const int nseg = (a.row_bytes + 127) / 128;
  const int hl = a.scan_head / 16;
  if (nseg > SHARED_MAX_NSEG || a.scan_head % 16 != 0 || a.scan_head > a.row_bytes)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_scan_qrec, dim3((unsigned)((a.nq + 255) / 256)), dim3(256), 0, s, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int grid = n_cu * NR_SHARED_BLOCKS_PER_CU;
  return dtype == NR_U8 ? launch_scan_t<1>(a, nseg, hl, grid, s)
                        : launch_scan_t<0>(a, nseg, hl, grid, s);
}

// ------------------------------------------------------------------ open pairs
// The pairs of fp32 rows past 1 KB that the scan's first slab left at or
// before their bound: 8 lanes per pair add the remaining 1 KB slabs in order
// to the stored running sum (each slab accumulated per lane in segment order
// and reduced over the 8 lanes, as everywhere else for such rows), stop once
// the sum is past the bound, and keep the pair as a survivor otherwise.
__global__ void __launch_bounds__(256) k_scan_open(SharedArgs a) {
  const int lane = lane_id();
  const int gl = lane & 7;
  const uint64_t n0 = *a.open_cnt;
  const uint64_t n = n0 < OPEN_PAIRS ? n0 : OPEN_PAIRS;
  const int rb = a.row_bytes;
  const int k = a.k;
  const int nsl = (rb + 1023) / 1024;
  const unsigned char *queries = (const unsigned char *)a.queries;
  unsigned long long body = 0;
  const uint64_t stride = (uint64_t)gridDim.x * (blockDim.x >> 3);
  for (uint64_t p = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 3; p < n; p += stride) {
    const uint32_t q = a.open_q[p];
    const uint64_t row = a.open_row[p];
    float run = __uint_as_float(a.open_key[p]);
    const int64_t own_id = a.own_ids[(int64_t)q * k + k - 1];
    const uint32_t bound = own_id < 0 ? 0xffffffffu : __float_as_uint(a.own_dists[(int64_t)q * k + k - 1]);
    const unsigned char *qb = queries + (uint64_t)q * rb;
    bool open = true;
    for (int sl = 1; sl < nsl && open; ++sl) {
      uint4 xv[8], qv[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int off = 1024 * sl + 128 * s + 16 * gl;
        xv[s] = off < rb ? load_stream(a.ra.seg(row, off)) : make_uint4(0, 0, 0, 0);
        qv[s] = off < rb ? *(const uint4 *)(qb + off) : make_uint4(0, 0, 0, 0);
      }
      float acc = 0.0f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const float t0 = __uint_as_float(xv[s].x) - __uint_as_float(qv[s].x);
        const float t1 = __uint_as_float(xv[s].y) - __uint_as_float(qv[s].y);
        const float t2 = __uint_as_float(xv[s].z) - __uint_as_float(qv[s].z);
        const float t3 = __uint_as_float(xv[s].w) - __uint_as_float(qv[s].w);
        acc = fmaf(t0, t0, acc);
        acc = fmaf(t1, t1, acc);
        acc = fmaf(t2, t2, acc);
        acc = fmaf(t3, t3, acc);
      }
      run = run + group8_sum(acc);
      body += (unsigned long long)(rb - 1024 * sl < 1024 ? rb - 1024 * sl : 1024);
      open = __float_as_uint(run) <= bound;
    }
    if (open && gl == 0) add_survivor(a, q, __float_as_uint(run), a.row_ids[row]);
  }
  if (gl == 0 && body) atomicAdd((unsigned long long *)&a.wstats[5], body);
}

hipError_t launch_scan_open(const SharedArgs &a, int dtype, int n_cu, hipStream_t s) {
  if (a.nq <= 0 || dtype == NR_U8 || a.row_bytes <= 1024) return hipSuccess;
  hipLaunchKernelGGL(k_scan_open, dim3(n_cu * 8), dim3(256), 0, s, a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ merge
// (key, id) of a top-k list held in lanes 0..k-1
struct SharedTopK {
  uint32_t key;
  int64_t id;
  int cnt;
  uint32_t kth_key;
  int64_t kth_id;
};

__device__ __forceinline__ void stk_insert(SharedTopK &t, int k, uint32_t ck, int64_t cid) {
  const int lane = lane_id();
  if (t.cnt == k && (ck > t.kth_key || (ck == t.kth_key && cid >= t.kth_id))) return;
  const bool less = lane < t.cnt && (t.key < ck || (t.key == ck && t.id < cid));
  const int pos = popc64(ballot(less));
  const uint32_t up_key = (uint32_t)__shfl_up((int)t.key, 1);
  const int64_t up_id = (int64_t)shfl_up_u64((uint64_t)t.id, 1);
  if (lane == pos) {
    t.key = ck;
    t.id = cid;
  } else if (lane > pos && lane < k) {
    t.key = up_key;
    t.id = up_id;
  }
  t.cnt = t.cnt + 1 < k ? t.cnt + 1 : k;
  if (t.cnt == k) {
    t.kth_key = bcast_u32(t.key, k - 1);
    t.kth_id = (int64_t)bcast_u64((uint64_t)t.id, k - 1);
  }
}

// pooled survivors per query: offsets (one block scans the per-query counts)
__global__ void __launch_bounds__(1024) k_pool_offsets(SharedArgs a) {
  __shared__ uint32_t part[1024];
  const int tid = threadIdx.x;
  const int64_t per = (a.nq + 1023) / 1024;
  const int64_t s0 = tid * per;
  uint32_t sum = 0;
  // a flagged query lost survivors and is recomputed: it takes no pool2 space,
  // so the offsets stay within the survivors actually pooled
  for (int64_t q = s0; q < s0 + per && q < a.nq; ++q) {
    const int c = a.flag[q] ? 0 : a.scnt[q];
    sum += c > SURVIVOR_CAP ? (uint32_t)(c - SURVIVOR_CAP) : 0u;
  }
  part[tid] = sum;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const uint32_t v = tid >= o ? part[tid - o] : 0u;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  uint32_t run = part[tid] - sum;
  for (int64_t q = s0; q < s0 + per && q < a.nq; ++q) {
    const int c = a.flag[q] ? 0 : a.scnt[q];
    a.poff[q] = run;
    a.pcur[q] = 0;
    run += c > SURVIVOR_CAP ? (uint32_t)(c - SURVIVOR_CAP) : 0u;
  }
  if (tid == 1023) a.poff[a.nq] = part[1023];
}

// pooled survivors grouped by query (order inside a query is arbitrary)
// (pooled entries of one query tend to be adjacent: the lanes of a wave that
// share a query take their positions with one atomic)
__global__ void k_pool_scatter(SharedArgs a) {
  const unsigned long long used = *a.pool_cnt;
  const uint64_t n = used < SURVIVOR_POOL ? used : SURVIVOR_POOL;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t first = (uint64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~63u);
  for (uint64_t e0 = first; e0 < n; e0 += stride) {
    const uint64_t e = e0 + lane_id();
    const bool in = e < n;
    const uint32_t q = in ? a.pool_q[e] : 0xffffffffu;
    const bool live = in && !a.flag[q];
    uint64_t todo = ballot(live);
    while (todo) {
      const uint32_t lq = bcast_u32(q, __ffsll((unsigned long long)todo) - 1);
      const uint64_t same = ballot(live && q == lq);
      todo &= ~same;
      uint32_t base = 0;
      if (live && q == lq && (same & lanemask_lt()) == 0)
        base = atomicAdd(&a.pcur[lq], (uint32_t)popc64(same));
      base = bcast_u32(base, __ffsll((unsigned long long)same) - 1);
      if (live && q == lq) {
        const uint32_t pos = a.poff[lq] + base + (uint32_t)popc64(same & lanemask_lt());
        a.pool2_key[pos] = a.pool_key[e];
        a.pool2_id[pos] = a.pool_id[e];
      }
    }
  }
}

__global__ void __launch_bounds__(256) k_shared_merge(SharedArgs a) {
  const int lane = lane_id();
  const int64_t q = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (q >= a.nq) return;
  if (lane == 0) {
    a.own_rows[q] = a.rtot[q];
    if (q == 0) a.wstats[1] = a.tile_off[a.nq];
  }
  const int k = a.k;
  if (a.flag[q]) return;  // a survivor was lost: recomputed by the per-query schedule
  const int cnt = a.scnt[q];
  const int own = cnt < SURVIVOR_CAP ? cnt : SURVIVOR_CAP;
  const uint32_t p0 = a.poff[q];
  SharedTopK tk;
  tk.key = 0xffffffffu;
  tk.id = -1;
  tk.cnt = 0;
  tk.kth_key = 0xffffffffu;
  tk.kth_id = INT64_MAX;
  // the seed top-k (sorted)
  {
    int64_t id = -1;
    uint32_t key = 0xffffffffu;
    if (lane < k) {
      id = a.own_ids[q * k + lane];
      const float d = a.own_dists[q * k + lane];
      key = a.is_u8 ? (uint32_t)d : __float_as_uint(d);
    }
    uint64_t m = ballot(lane < k && id >= 0);
    while (m) {
      const int src = __ffsll((unsigned long long)m) - 1;
      m &= m - 1;
      stk_insert(tk, k, bcast_u32(key, src), (int64_t)bcast_u64((uint64_t)id, src));
    }
  }
  // survivors: the query's own slots, then its pooled ones; four chunks of
  // 64 are loaded per round, ids only for keys that can still enter
  constexpr int RC = 4;
  for (int r0 = 0; r0 < cnt; r0 += RC * WAVE) {
    uint32_t key[RC];
#pragma unroll
    for (int u = 0; u < RC; ++u) {
      const int i = r0 + u * WAVE + lane;
      key[u] = 0xffffffffu;
      if (i < own) key[u] = a.skey[q * SURVIVOR_CAP + i];
      else if (i < cnt) key[u] = a.pool2_key[p0 + (uint32_t)(i - SURVIVOR_CAP)];
    }
#pragma unroll
    for (int u = 0; u < RC; ++u) {
      const int i = r0 + u * WAVE + lane;
      uint64_t m = ballot(i < cnt && key[u] <= tk.kth_key);
      if (!m) continue;
      int64_t id = -1;
      if ((m >> lane) & 1ull)
        id = i < own ? a.sid[q * SURVIVOR_CAP + i] : a.pool2_id[p0 + (uint32_t)(i - SURVIVOR_CAP)];
      while (m) {
        const int src = __ffsll((unsigned long long)m) - 1;
        m &= m - 1;
        stk_insert(tk, k, bcast_u32(key[u], src), (int64_t)bcast_u64((uint64_t)id, src));
      }
    }
  }
  if (lane < k) {
    const bool have = lane < tk.cnt;
    a.out_ids[q * k + lane] = have ? tk.id : -1;
    a.out_dists[q * k + lane] =
        have ? (a.is_u8 ? (float)tk.key : __uint_as_float(tk.key)) : INFINITY;
  }
  if (lane == 0 && a.qstats) a.qstats[q * NR_QSTATS + NR_QS_ROWS] = (int32_t)a.rfull[q];
}

hipError_t launch_shared_merge(const SharedArgs &a, hipStream_t s) {
  if (a.nq <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_pool_offsets, dim3(1), dim3(1024), 0, s, a);
  hipLaunchKernelGGL(k_pool_scatter, dim3(1024), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_shared_merge, dim3((unsigned)((a.nq + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ diagnostics
// rows of the shared clusters (each read once by the scan) -> out[0] and
// rows scored by the scan summed over pairs -> out[2], over the scan list
__global__ void k_unique_rows(const uint32_t *slist, const uint32_t *lpm, const uint64_t *lmeta,
                              const uint64_t *cl_off, int64_t *out) {
  __shared__ unsigned long long part[2][256];
  unsigned long long acc = 0, accp = 0;
  const int64_t ns = (int64_t)lmeta[0];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < ns; i += stride) {
    const uint32_t c = slist[i];
    const uint64_t sz = cl_off[(uint64_t)c + 1] - cl_off[c];
    acc += sz;
    accp += (uint64_t)lpm[i] * sz;
  }
  part[0][threadIdx.x] = acc;
  part[1][threadIdx.x] = accp;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      part[0][threadIdx.x] += part[0][threadIdx.x + o];
      part[1][threadIdx.x] += part[1][threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    atomicAdd((unsigned long long *)out, part[0][0]);
    atomicAdd((unsigned long long *)(out + 2), part[1][0]);
  }
}

hipError_t launch_unique_rows(const uint32_t *slist, const uint32_t *lpm, const uint64_t *lmeta,
                              const uint64_t *cl_off, int64_t *out, hipStream_t s) {
  hipLaunchKernelGGL(k_unique_rows, dim3(1024), dim3(256), 0, s, slist, lpm, lmeta, cl_off, out);
  return hipGetLastError();
}

}  // namespace nr
