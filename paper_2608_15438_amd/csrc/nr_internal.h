// Internal declarations of the gfx950 search library: kernel argument
// structs, launch wrappers and wave64 helpers.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "neuroute.h"

namespace nr {

constexpr int WAVE = 64;
#ifndef NR_MAX_TILES_PER_QUERY
#define NR_MAX_TILES_PER_QUERY 64
#endif
constexpr int MAX_TILES_PER_QUERY = NR_MAX_TILES_PER_QUERY;  // refinement tiles per query
#ifndef NR_TILE_MIN_ROWS
#define NR_TILE_MIN_ROWS 512
#endif
constexpr int TILE_MIN_ROWS = NR_TILE_MIN_ROWS;  // smallest refinement tile
constexpr int STAGE_CLUSTERS = 128;       // clusters staged in LDS per refinement wave
constexpr int64_t QUERY_CHUNK = 16384;    // queries per internal launch sequence
#ifndef NR_OWN_TILE_MIN_ROWS
#define NR_OWN_TILE_MIN_ROWS 2048
#endif
constexpr uint32_t OWN_TILE_MIN_ROWS = NR_OWN_TILE_MIN_ROWS;  // smallest tile of the own pass
#ifndef NR_SEED_ROWS
#define NR_SEED_ROWS 4096
#endif
constexpr uint32_t SEED_ROWS = NR_SEED_ROWS;      // rows of a query's first clusters refined on their own
constexpr uint32_t SEED_ROWS_LONG = 1024;          // the same for rows past 1 KB, which the scan
                                                   // mostly settles after their first 1 KB
#ifndef NR_SURVIVOR_CAP
#define NR_SURVIVOR_CAP 2048
#endif
constexpr int SURVIVOR_CAP = NR_SURVIVOR_CAP;  // survivors a query keeps in its own slots
#ifndef NR_SURVIVOR_POOL
#define NR_SURVIVOR_POOL (1u << 22)
#endif
constexpr uint32_t SURVIVOR_POOL = NR_SURVIVOR_POOL;  // survivors past SURVIVOR_CAP, all queries
#ifndef NR_OPEN_PAIRS
#define NR_OPEN_PAIRS (1u << 22)
#endif
constexpr uint32_t OPEN_PAIRS = NR_OPEN_PAIRS;  // fp32 rows past 1 KB: pairs open after slab 0
constexpr int SHARED_G = 8;               // queries scored per shared work unit (at most)
constexpr int SHARED_MAX_NSEG = 48;       // rows of at most 48 x 128 bytes use the shared scan
constexpr uint32_t SHARED_ROWS = 2048;    // rows per shared work unit (at most)
constexpr int MAX_KC = 16384;             // top-K_c heap held in LDS
// the shared schedule's scan-list build: LIST_WPT words of 32 pair counts per
// thread; the counts array is hist_words long (whole words, and at least
// n_clusters + 1 counts)
constexpr int LIST_WPT = 1;
constexpr int LIST_THREADS = 256;
__host__ __device__ inline int64_t list_words(int64_t n_clusters) { return (n_clusters + 31) / 32; }
__host__ __device__ inline int64_t hist_words(int64_t n_clusters) {
  return (list_words(n_clusters) + 1) * 32;
}
__host__ __device__ inline int64_t list_blocks(int64_t n_clusters) {
  const int64_t per = (int64_t)LIST_WPT * LIST_THREADS;
  const int64_t b = (list_words(n_clusters) + per - 1) / per;
  return b > 0 ? b : 1;
}

// ---------------------------------------------------------------- kernels
// Addressing of the permuted payload: bytes [0, h) of row r at hb + r * hs,
// bytes [h, row_bytes) at tb + r * ts.  Row-major: hb = tb - h = rows,
// hs = ts = row_bytes.  Split layout: a head plane then a tail plane.
struct RowAddr {
  const unsigned char *hb;
  const unsigned char *tb;
  uint64_t hs, ts;
  int h;
  __device__ __forceinline__ const uint4 *seg(uint64_t r, int off) const {
    return off < h ? reinterpret_cast<const uint4 *>(hb + r * hs + off)
                   : reinterpret_cast<const uint4 *>(tb + r * ts + (off - h));
  }
};

struct EncodeLayerArgs {
  const void *in;        // [M x K]: uint8 or fp32 (layer 0) / fp32 activations
  int in_u8;
  float *out;            // [M x N] fp32
  const float *W;        // [N x K] row-major
  const float *bias;     // [N]
  const float *bn_scale; // [N] or null
  const float *bn_shift; // [N] or null
  float in_scale;
  int relu;
  int64_t M;
  int N, K;
};

struct ProbeArgs {
  const float *logits;   // [nq x b]
  const float *tau;      // [b]
  int64_t nq;
  int b, l_sel, r_max, P, n_bins, finite;
  float s_max, bin_scale;
  uint32_t *codes;       // [nq x P]
  float *costs;
  int32_t *bins;
  int32_t *counts;       // [nq]
  // optional, for the search: each probe's bucket looked up in the directory
  // (lk[q x P + i] = [bc_off[code], bc_off[code + 1])) and each query's route
  // pass (see route_tiers; tier[q] = the first pass whose heap holds the
  // summed sizes of its multi-cluster buckets)
  const uint32_t *bc_off;
  uint2 *lk;             // [nq x P] (NULL: no lookup)
  int32_t *tier;         // [nq] (NULL: no tiers)
  int tier_n, tier_h0, tier_h1;
};

// calibration (k_calib.hip): bucket scores of the targets and margin points
struct CalibArgs {
  const float *logits;          // [nq x b]
  const float *tau;             // [b]
  int64_t nq, n;
  int b, l_sel, r_max, K;
  const int64_t *targets;       // [nq x K] original ids, < 0: none
  const uint32_t *row_of_id;    // [n] permuted row of each original id
  const uint64_t *cl_off;       // [n_clusters + 1]
  int64_t n_clusters, n_codes;  // n_codes = 2^b
  const uint32_t *bc_off;       // [n_codes + 1]
  const float *centroids;       // [n_clusters x b]
  float *scores;                // [nq x K]
  float *xy;                    // [nq x 2]
};

// per-query pair counting of the shared schedule (see pair_hist_wave)
struct PairHistArgs {
  uint32_t *hist;               // [n_clusters + 1] pairs per cluster past the leading clusters
  const uint64_t *cl_off;
  int64_t n_clusters;
  uint32_t seed_min;            // rows the leading clusters cover at least
  int32_t *cseed;               // [nq] leading clusters
  uint32_t *rfull;              // [nq] rows of the leading clusters (whole list: eager_rows)
  uint2 *qnorm;                 // [nq] uint8 rows: |q|^2 and its head part
  const unsigned char *queries;
  int row_bytes, scan_head, is_u8, eager_rows;
  uint32_t *pair_rank;          // [nq x cap] each counted pair's rank among its cluster's pairs
  int64_t cap;
};

struct RouteArgs {
  const float *logits;
  int64_t nq;
  int b, P;
  const int32_t *bins;
  const int32_t *counts;
  uint2 *lk;             // [nq x P] cluster range of each probe's bucket (written by k_probe)
  int pst;               // probes per query whose ranges are staged in LDS (set per pass)
  int hcap, pass;        // heap slots in LDS and pass number (set by launch_route)
  int tiered;            // redo[q] holds the pass that routes query q
  int32_t *redo;         // [nq] the pass of each query (written by k_probe when tiered)
  const float *centroids;
  int k_c, b_batch, b_min, t_low, u_heap, u_front;
  float alpha_front;
  int gate_on, early_stop_on, lowq_or, finite;
  int m_knots;
  float m_x[NR_MAX_KNOTS], m_y[NR_MAX_KNOTS], m_slope[NR_MAX_KNOTS];
  uint32_t *clus;        // [nq x cap]
  int32_t *nclus;        // [nq]
  int64_t cap;
  int32_t *qstats;       // [nq x NR_QSTATS] or null
  PairHistArgs ph;       // with ph_on: each query's pairs are counted once its list is final
  int ph_on;
};

struct PlanArgs {
  int64_t nq;
  const uint32_t *clus;
  const int32_t *nclus;
  int64_t cap;
  const uint64_t *cl_off;
  int64_t n_clusters;    // cluster ids >= n_clusters count as empty
  uint32_t *rowpre;      // [nq x (cap + 1)]
  uint32_t *rtot;        // [nq]
  uint32_t *tsize;       // [nq]
  int32_t *ntile;        // [nq]
  int32_t *tile_off;     // [nq + 1]
  int32_t *tile_q;       // [nq x MAX_TILES_PER_QUERY]
  int32_t *tile_c0;
  int32_t *counter;      // work counter of the refinement kernel
  uint32_t *rfull;       // [nq] rows of the whole list, may be null
  const int32_t *qmask;  // [nq] only queries with qmask[q] != 0 get tiles, may be null
  const int32_t *own_cseed;  // [nq] may be null; else only list positions i < own_cseed[q] count
  uint32_t *clus_out;        // with own_cseed: [nq x cap] the clusters that count, compacted
  int32_t *nclus_out;        // [nq]
  uint32_t tile_min;         // smallest tile (rows); 0: TILE_MIN_ROWS
};

struct RefineArgs {
  RowAddr ra;            // permuted payload
  const int64_t *row_ids;
  const uint64_t *cl_off;
  int64_t n_clusters;
  const void *queries;   // [nq x d]
  int64_t nq;
  int d, row_bytes, k;
  const uint32_t *clus;
  const int32_t *nclus;
  int64_t cap;
  const uint32_t *rowpre;
  const uint32_t *rtot;
  const uint32_t *tsize;
  const int32_t *tile_off;
  const int32_t *tile_q;
  const int32_t *tile_c0;
  int32_t *counter;
  uint32_t *pkey;        // [nq x MAX_TILES_PER_QUERY x k]
  int64_t *pid;
  unsigned long long *rbytes;  // row bytes the kernel read (added to)
};

struct MergeArgs {
  int64_t nq;
  int k, is_u8;
  const int32_t *tile_off;
  const uint32_t *pkey;
  const int64_t *pid;
  const uint32_t *rtot;
  int64_t *out_ids;
  float *out_dists;
  int32_t *qstats;
  const int32_t *qmask;  // only queries with qmask[q] != 0 are written, may be null
};

// batch-shared refinement: a candidate row listed by several queries of the
// batch is read once and scored for all of them
struct SharedArgs {
  int64_t nq;
  int k, is_u8, row_bytes;
  int g;                      // queries per work unit (SHARED_G)
  uint32_t seed_min;          // rows the leading clusters of a list cover at least
  int64_t n_clusters;
  RowAddr ra;                 // permuted payload
  int scan_head;              // bytes of each row the scan's filter reads (its head)
  const unsigned char *scan_hb;  // head of row r at scan_hb + r * scan_hs
  uint64_t scan_hs;
  const int64_t *row_ids;
  const uint64_t *cl_off;
  const void *queries;
  const uint32_t *clus;
  const int32_t *nclus;
  int64_t cap;
  int32_t *cseed;             // [nq] leading clusters, scored by the query's own (seed) pass
  uint32_t *rfull;            // [nq] rows of the whole list
  const uint32_t *rtot;       // [nq] rows of the own pass
  const int32_t *tile_off;    // [nq + 1] tiles of the own pass
  const int64_t *own_ids;     // [nq x k] top-k of the own pass (sorted)
  const float *own_dists;
  uint32_t *own_rows;         // [nq] copy of rtot kept for diagnostics
  uint32_t *hist;             // [n_clusters + 1] pairs per cluster past the leading clusters
  uint32_t *pair_rank;        // [nq x cap] rank of each counted pair among its cluster's pairs
  uint32_t *hpos;             // [n_clusters] start of cluster c's pairs in pair_q (clusters
                              // with pairs only)
  uint32_t *slist;            // [n_clusters] the scan list: clusters with pairs, in order
  uint32_t *lpair, *lpm;      // [list] start in pair_q and number of pairs of entry i
  uint64_t *lbase;            // [list] first payload row of entry i's cluster
  uint32_t *lsz;              // [list] rows of entry i's cluster
  uint64_t *swork_off;        // [list + 1] start of entry i in the work space
  uint64_t *lmeta;            // [4] list length, pairs, work
  uint32_t *thr_n, *thr_h;    // [list_blocks x LIST_THREADS] per-thread sums of the prep
  uint64_t *thr_w;
  uint32_t *blk_n, *blk_h;    // [list_blocks] per-block sums, then their offsets
  uint64_t *blk_w;
  int eager_rows;             // 1: rfull gets the rows of the whole list (else the leading ones)
  uint32_t *pair_q;           // [pairs] query of each scanned pair, grouped by cluster
  uint2 *qnorm;               // [nq] uint8 rows: (|q|^2, |q head|^2 over scan_head bytes)
  uint4 *qrec;                // [nq] the scan's record of a query, written after the seed
                              // merge: (bound key, head threshold, |q|^2, 0)
  int32_t *scnt;              // [nq] survivors appended
  uint32_t *skey;             // [nq x SURVIVOR_CAP]
  int64_t *sid;
  int32_t *flag;              // [nq] 1: survivors lost (pool full), recompute per query
  unsigned long long *pool_cnt;  // survivors appended to the pool
  uint32_t *pool_q, *pool_key;   // [SURVIVOR_POOL] query and key of pooled survivors
  int64_t *pool_id;
  uint32_t *poff;             // [nq + 1] per-query start of its pooled survivors in pool2
  uint32_t *pcur;             // [nq] scatter cursors
  uint32_t *pool2_key;        // [SURVIVOR_POOL] pooled survivors grouped by query
  int64_t *pool2_id;
  unsigned long long *open_cnt;  // fp32 rows past 1 KB: (query, row) pairs still at or
  uint32_t *open_q, *open_key;   // before the bound after the first 1 KB slab, their
  uint64_t *open_row;            // running sum and payload row [OPEN_PAIRS]
  unsigned long long *counter;  // work-unit counter
  int64_t *wstats;            // [7] scanned rows, seed tiles, scanned pair rows, rows read
                              // past their heads, bytes the scan read from them, row
                              // bytes of the open-pair pass, row bytes of k_refine
  int64_t *out_ids;
  float *out_dists;
  int32_t *qstats;
};


hipError_t launch_encode_layer(const EncodeLayerArgs &a, hipStream_t s);
hipError_t launch_probe(const ProbeArgs &a, hipStream_t s);
constexpr int ROUTE_LIGHT_HEAP = 512;  // heap slots of the route's first pass
constexpr int ROUTE_MID_HEAP = 2048;   // and of its second when K_c is larger still
// the heap sizes of the route's passes for K_c: one pass of K_c keys up to
// ROUTE_LIGHT_HEAP, else ROUTE_LIGHT_HEAP, ROUTE_MID_HEAP (when K_c is larger
// still) and K_c; returns the number of passes
inline int route_tiers(int k_c, int tiers[3]) {
  if (k_c <= ROUTE_LIGHT_HEAP) {
    tiers[0] = k_c;
    return 1;
  }
  int nt = 0;
  tiers[nt++] = ROUTE_LIGHT_HEAP;
  if (k_c > ROUTE_MID_HEAP) tiers[nt++] = ROUTE_MID_HEAP;
  tiers[nt++] = k_c;
  return nt;
}
size_t route_lds_bytes(int k_c, int pst);
// aux, fork, join (may be null): a second stream and two events, on which the
// passes with larger heaps run beside the first
hipError_t launch_route(const RouteArgs &a, hipStream_t s, hipStream_t aux = nullptr,
                        hipEvent_t fork = nullptr, hipEvent_t join = nullptr);
hipError_t launch_plan(const PlanArgs &a, hipStream_t s);
// blocks_per_cu: 0 for the tuned default; fewer leave room on every CU for
// work on another stream (the scan's preparation beside the seed pass)
hipError_t launch_refine(const RefineArgs &a, int dtype, int n_cu, int blocks_per_cu,
                         hipStream_t s);
hipError_t launch_merge(const MergeArgs &a, hipStream_t s);
// fresh: the workspace is new, so clear the pair counts
hipError_t launch_shared_hist(const SharedArgs &a, bool fresh, hipStream_t s);
PairHistArgs pair_hist_args(const SharedArgs &a);
hipError_t launch_shared_prep(const SharedArgs &a, hipStream_t s);
hipError_t launch_shared_refine(const SharedArgs &a, int dtype, int n_cu, hipStream_t s);
// the open pairs' remaining slabs (fp32 rows past 1 KB; a no-op otherwise)
hipError_t launch_scan_open(const SharedArgs &a, int dtype, int n_cu, hipStream_t s);
hipError_t launch_shared_merge(const SharedArgs &a, hipStream_t s);
hipError_t launch_unique_rows(const uint32_t *slist, const uint32_t *lpm, const uint64_t *lmeta,
                              const uint64_t *cl_off, int64_t *out, hipStream_t s);
hipError_t launch_list_rows(const uint32_t *clus, const int32_t *nclus, int64_t cap, int64_t nq,
                            const uint64_t *cl_off, int64_t n_clusters, uint32_t *rows,
                            hipStream_t s);
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);

hipError_t launch_inverse_perm(const int64_t *row_ids, int64_t n, uint32_t *row_of_id,
                               hipStream_t s);
hipError_t launch_calib(const CalibArgs &a, hipStream_t s);
// index construction (k_build.hip)
struct BuildArgs {
  int64_t n;
  int b;
  const float *lg;            // [n x b] latents by original id
  const uint32_t *codes;      // [n]
  const uint32_t *sizes;      // [2^b]
  int rule;
  uint32_t t;
  uint32_t *kb, *multi, *mpos, *mlist;   // [2^b] (+1 for the scans)
  unsigned long long *stats;  // [3] sum kb, multi buckets, max kb
  uint64_t *blk;              // scan scratch [build_scan_blocks(max items)]
  uint64_t *kbpre, *boff;     // [2^b + 1]
  uint32_t *cursor, *nkept, *ncl;        // [2^b] (+1)
  uint32_t *ids, *ids_tmp, *label;       // [n]
  uint64_t *skey, *skey_tmp;  // [n]
  double *d2;                 // [n]
  int64_t n_multi;
  const double *U;            // [n_multi x kmax]
  int kmax;
  uint32_t seed;
  int lloyd, spc;
  double *cent;               // [max_clusters x b]
  uint32_t *ccnt;             // [max_clusters]
  uint32_t *bc_off;           // [2^b + 1] out
  int64_t *row_ids;           // [n] out
  uint64_t *csize;            // [max_clusters]
  float *centroids;           // [max_clusters x b] out
};
size_t build_scan_blocks(int64_t n);
hipError_t launch_build_tau(const float *lg, int64_t ns, int b, float *tau, hipStream_t s);
hipError_t launch_build_codes(const float *lg, int64_t m, int b, const float *tau, uint32_t *codes,
                              uint32_t *sizes, hipStream_t s);
hipError_t launch_build_nonempty(const uint32_t *sizes, int64_t nb, unsigned long long *out,
                                 hipStream_t s);
hipError_t run_build_plan(const BuildArgs &a, hipStream_t s);
hipError_t run_build_index(const BuildArgs &a, hipStream_t s);
hipError_t launch_build_cl_off(const uint64_t *csize, int64_t n_clusters, uint64_t *cl_off,
                               uint64_t *blk, hipStream_t s);

// L_sim training (k_lsim.hip)
size_t pair_sqdist_ws_floats(int64_t B, int D);
hipError_t launch_pair_sqdist(const float *x, int64_t B, int D, float *ws, float *out,
                              hipStream_t s);
hipError_t launch_lsim_grad(const float *d2, const float *lat, int64_t B, int L, float gr,
                            float tau, double *num_cnt, float *grad, hipStream_t s);

hipError_t launch_stream_read(const void *buf, int64_t bytes, uint32_t *sink, int n_cu,
                              hipStream_t s);

// index validation at upload; flags[0] |= error bits
hipError_t launch_validate(const uint32_t *bc_off, int64_t n_codes, const uint64_t *cl_off,
                           int64_t n_clusters, const int64_t *row_ids, int64_t n,
                           uint32_t *bitmap, int32_t *flags, hipStream_t s);

// ---------------------------------------------------------------- wave64 helpers
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint32_t bcast_u32(uint32_t v, int src) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, src);
}
__device__ __forceinline__ float bcast_f32(float v, int src) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
}
__device__ __forceinline__ uint64_t bcast_u64(uint64_t v, int src) {
  uint32_t lo = bcast_u32((uint32_t)v, src), hi = bcast_u32((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
  uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src);
  uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int m) {
  uint32_t lo = (uint32_t)__shfl_up((int)(uint32_t)v, m);
  uint32_t hi = (uint32_t)__shfl_up((int)(uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ uint64_t lanemask_lt() {
  int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}
__device__ __forceinline__ float wave_min_f32(float v) {
  for (int m = 32; m >= 1; m >>= 1) v = fminf(v, __shfl_xor(v, m));
  return v;
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
  for (int m = 32; m >= 1; m >>= 1) v += (uint32_t)__shfl_xor((int)v, m);
  return v;
}
// inclusive scan over the wave (u32)
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
  int l = lane_id();
  for (int o = 1; o < WAVE; o <<= 1) {
    uint32_t t = (uint32_t)__shfl_up((int)v, o);
    if (l >= o) v += t;
  }
  return v;
}
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
  int l = lane_id();
  for (int o = 1; o < WAVE; o <<= 1) {
    uint64_t t = shfl_up_u64(v, o);
    if (l >= o) v += t;
  }
  return v;
}
// ascending bitonic sort of one u64 key per lane, where every lane from n on
// holds ~0: only the first power of two >= n lanes need the network
__device__ __forceinline__ uint64_t wave_sort_u64(uint64_t key, int n = WAVE) {
  int l = lane_id();
  int top = 2;
  while (top < n && top < WAVE) top <<= 1;
  for (int k = 2; k <= top; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      uint64_t other = shfl_xor_u64(key, j);
      bool up = (l & k) == 0;
      bool lower = (l & j) == 0;
      uint64_t mn = key < other ? key : other, mx = key < other ? other : key;
      key = (lower == up) ? mn : mx;
    }
  }
  return key;
}
// number of entries of sorted a[0..n) strictly below key
__device__ __forceinline__ int lower_bound_u64(const uint64_t *a, int n, uint64_t key) {
  int lo = 0, hi = n;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a[mid] < key) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// One wave, query q with list cl[0..n): the leading clusters covering at
// least seed_min rows stay with the query (cseed[q]); every later (cluster,
// query) pair is counted in hist (its rank among the cluster's pairs goes to
// pair_rank); rfull[q] gets the rows of the leading
// clusters (of the whole list with eager_rows); for uint8 rows qnorm[q] gets
// |q|^2 and the part of it over the scan's head.
__device__ inline void pair_hist_wave(const PairHistArgs &h, int64_t q, const uint32_t *cl, int n) {
  const int lane = lane_id();
  // rows of the leading clusters, and of the whole list when eager_rows is
  // set (otherwise the sizes of the later clusters are not needed here)
  const bool all = h.eager_rows != 0;
  uint64_t run = 0;
  int cs = -1;
  // the seed: sizes of the leading clusters until they cover seed_min rows
  for (int i0 = 0; i0 < n && (cs < 0 || all); i0 += WAVE) {
    const int i = i0 + lane;
    uint64_t sz = 0;
    if (i < n) {
      const uint32_t c = cl[i];
      if (c < h.n_clusters) sz = h.cl_off[(uint64_t)c + 1] - h.cl_off[c];
    }
    const uint64_t incl = wave_incl_scan_u64(sz);
    int upto = WAVE - 1;
    if (cs < 0) {
      const uint64_t hit = ballot(i < n && run + incl >= h.seed_min);
      if (hit) {
        cs = i0 + __ffsll((unsigned long long)hit);  // first position past the seed
        if (!all) upto = cs - 1 - i0;
      }
    }
    run += bcast_u64(incl, upto);
  }
  // the pairs past the seed, four per lane at a time: their cluster ids are
  // all loaded, then all counted, so each group costs two memory round trips
  if (cs >= 0) {
    for (int i0 = cs; i0 < n; i0 += 4 * WAVE) {
      uint32_t c[4], r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * WAVE + lane;
        c[u] = i < n ? cl[i] : 0xffffffffu;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) r[u] = c[u] < h.n_clusters ? atomicAdd(&h.hist[c[u]], 1u) : 0u;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (c[u] < h.n_clusters) h.pair_rank[q * h.cap + i0 + u * WAVE + lane] = r[u];
    }
  }
  if (lane == 0) {
    h.cseed[q] = cs < 0 ? n : cs;
    h.rfull[q] = run > 0xffffffffull ? 0u : (uint32_t)run;
  }
  // uint8 rows: |q|^2 and the part of it over the scan's head (at most 128
  // bytes, so within lanes 0..7's first chunks), lane c taking the 16-byte
  // chunks c, c + 64, ...; integer sums, so the order of the additions does
  // not matter
  if (h.is_u8) {
    uint32_t p = 0, ph = 0;
    for (int c = lane; 16 * c < h.row_bytes; c += WAVE) {
      const uint4 v = *reinterpret_cast<const uint4 *>(h.queries +
                                                       (uint64_t)q * h.row_bytes + 16 * c);
      uint32_t t = 0;
      t = __builtin_amdgcn_udot4(v.x, v.x, t, false);
      t = __builtin_amdgcn_udot4(v.y, v.y, t, false);
      t = __builtin_amdgcn_udot4(v.z, v.z, t, false);
      t = __builtin_amdgcn_udot4(v.w, v.w, t, false);
      p += t;
      if (16 * c < h.scan_head) ph += t;
    }
    const uint32_t full = wave_sum_u32(p);
    const uint32_t head = wave_sum_u32(ph);
    if (lane == 0) h.qnorm[q] = make_uint2(full, head);
  }
}

}  // namespace nr
