// Index construction on the GPU (Sec. 3.3 "Bucket allocation" and
// "In-bucket clustering"; binarisation thresholds, Sec. 3.2.3), from the
// latents the encoder kernel gives the base rows:
//   tau      per latent dimension, the lower median of a sample of rows
//            (radix select on order-preserving keys, one block per dimension);
//   codes    bit j of a row's code = [l_j >= tau_j] (Eq. 10) and the bucket
//            sizes (atomic counts);
//   buckets  exclusive scan of the sizes, an atomic scatter of the row ids into
//            bucket order, then every bucket's ids sorted ascending;
//   k-means  one block per bucket with K_B >= 2 clusters: k-means++ on a
//            sample, then Lloyd passes over the whole bucket, in fp64 and in a
//            fixed order of summation (below);
//   layout   clusters kept per bucket -> bc_off (scan), every bucket's rows in
//            (cluster, id) order -> row_ids, cluster sizes -> cl_off (scan),
//            centroids = fp64 means of the member latents (in id order),
//            rounded to fp32.
// The k-means follows the reading of "a limited number of k-means
// iterations" that the reference builder takes: the sample is the first
// min(|B|, spc K_B) members ordered by (mix32(id, seed), id); the first centre
// is its first member; each further centre is drawn with probability
// proportional to the integer weight floor(D^2 2^20) (capped at 2^30), by the
// bucket's pre-drawn uniform U: the first sample member whose running weight
// exceeds floor(U * total); squared distances add the dimensions in order;
// centroid sums add the members in id order.  Integer weights make the draws
// independent of summation order, so the result is the reference builder's.
#include "nr_internal.h"

namespace nr {

constexpr int BT = 256;               // threads per block of the build kernels
constexpr int SCAN_PER_THREAD = 16;   // items per thread of the scans
constexpr int64_t SCAN_BLOCK = (int64_t)BT * SCAN_PER_THREAD;
constexpr int SORT_LDS = 4096;        // keys sorted in LDS by one block

// ------------------------------------------------------------------ helpers
__device__ __forceinline__ uint32_t mix32_dev(uint64_t x, uint32_t seed) {
  uint64_t h = (x ^ (uint64_t)seed) & 0xFFFFFFFFull;
  h = (((h >> 16) ^ h) * 0x45D9F3Bull) & 0xFFFFFFFFull;
  h = (((h >> 16) ^ h) * 0x45D9F3Bull) & 0xFFFFFFFFull;
  return (uint32_t)((h >> 16) ^ h);
}

// fp64 squared distance of an fp32 latent row to an fp64 point, dimensions
// added in order (no contraction: the build compiles with -ffp-contract=off)
__device__ __forceinline__ double sqd_row(const float *x, const double *c, int b) {
  double acc = 0.0;
  for (int j = 0; j < b; ++j) {
    const double t = (double)x[j] - c[j];
    acc = acc + t * t;
  }
  return acc;
}

__device__ __forceinline__ int64_t d2_weight(double d2) {
  double w = floor(d2 * 1048576.0);           // 2^20
  if (w > 1073741824.0) w = 1073741824.0;     // 2^30
  return (int64_t)w;
}

// block-wide exclusive scan of one value per thread (any integral T);
// *total gets the block's sum.  Uses `sh` (BT / WAVE entries).
template <class T>
__device__ __forceinline__ T block_excl_scan(T v, T *sh, T *total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  T incl = v;
  for (int o = 1; o < WAVE; o <<= 1) {
    const T t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  __syncthreads();
  if (lane == WAVE - 1) sh[w] = incl;
  __syncthreads();
  T before = 0, all = 0;
  for (int i = 0; i < BT / WAVE; ++i) {
    if (i < w) before += sh[i];
    all += sh[i];
  }
  *total = all;
  return before + incl - v;
}

// ------------------------------------------------------------------ scans
// out[i] = sum of in[0..i), out[n] = total, for n up to ~2^40 items.
template <class In>
__global__ void __launch_bounds__(BT) k_scan_sums(const In *in, int64_t n, uint64_t *blk) {
  __shared__ uint64_t sh[BT / WAVE];
  const int64_t base = (int64_t)blockIdx.x * SCAN_BLOCK + (int64_t)threadIdx.x * SCAN_PER_THREAD;
  uint64_t s = 0;
  for (int u = 0; u < SCAN_PER_THREAD; ++u)
    if (base + u < n) s += (uint64_t)in[base + u];
  uint64_t tot;
  (void)block_excl_scan<uint64_t>(s, sh, &tot);
  if (threadIdx.x == 0) blk[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(BT) k_scan_top(uint64_t *blk, int64_t nblk) {
  __shared__ uint64_t sh[BT / WAVE];
  const int64_t per = (nblk + BT - 1) / BT;
  const int64_t b0 = (int64_t)threadIdx.x * per;
  const int64_t b1 = b0 + per < nblk ? b0 + per : nblk;
  uint64_t s = 0;
  for (int64_t b = b0; b < b1; ++b) s += blk[b];
  uint64_t tot;
  uint64_t run = block_excl_scan<uint64_t>(s, sh, &tot);
  for (int64_t b = b0; b < b1; ++b) {
    const uint64_t x = blk[b];
    blk[b] = run;
    run += x;
  }
  if (threadIdx.x == 0) blk[nblk] = tot;
}

template <class In, class Out>
__global__ void __launch_bounds__(BT) k_scan_apply(const In *in, int64_t n, const uint64_t *blk,
                                                   int64_t nblk, Out *out) {
  __shared__ uint64_t sh[BT / WAVE];
  const int64_t base = (int64_t)blockIdx.x * SCAN_BLOCK + (int64_t)threadIdx.x * SCAN_PER_THREAD;
  uint64_t s = 0;
  for (int u = 0; u < SCAN_PER_THREAD; ++u)
    if (base + u < n) s += (uint64_t)in[base + u];
  uint64_t tot;
  uint64_t run = blk[blockIdx.x] + block_excl_scan<uint64_t>(s, sh, &tot);
  for (int u = 0; u < SCAN_PER_THREAD; ++u)
    if (base + u < n) {
      out[base + u] = (Out)run;
      run += (uint64_t)in[base + u];
    }
  if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = (Out)blk[nblk];
}

// blk: [ceil(n / SCAN_BLOCK) + 1] scratch
template <class In, class Out>
hipError_t launch_scan(const In *in, int64_t n, Out *out, uint64_t *blk, hipStream_t s) {
  const int64_t nblk = n > 0 ? (n + SCAN_BLOCK - 1) / SCAN_BLOCK : 1;
  hipLaunchKernelGGL((k_scan_sums<In>), dim3((unsigned)nblk), dim3(BT), 0, s, in, n, blk);
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(BT), 0, s, blk, nblk);
  hipLaunchKernelGGL((k_scan_apply<In, Out>), dim3((unsigned)nblk), dim3(BT), 0, s, in, n, blk,
                     nblk, out);
  return hipGetLastError();
}

size_t build_scan_blocks(int64_t n) { return (size_t)((n + SCAN_BLOCK - 1) / SCAN_BLOCK) + 2; }

// ------------------------------------------------------------------ tau
// order-preserving u32 key of a float (-0 and +0 map apart, as their order
// in a total order; no NaN reaches here)
__device__ __forceinline__ uint32_t fkey(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float fkey_inv(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// one block per dimension: the (ns - 1) / 2-th smallest value of column j
__global__ void __launch_bounds__(BT) k_build_tau(const float *lg, int64_t ns, int b, float *tau) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_prefix, s_rank;
  const int j = blockIdx.x;
  uint32_t prefix = 0;
  uint32_t rank = (uint32_t)((ns - 1) / 2);   // rank among the keys matching the prefix
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hmask = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
    for (int i = threadIdx.x; i < 256; i += BT) hist[i] = 0;
    __syncthreads();
    for (int64_t i = threadIdx.x; i < ns; i += BT) {
      const uint32_t k = fkey(lg[i * b + j]);
      if ((k & hmask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t r = rank, d = 0;
      while (d < 255 && hist[d] <= r) {
        r -= hist[d];
        ++d;
      }
      s_prefix = prefix | (d << shift);
      s_rank = r;
    }
    __syncthreads();
    prefix = s_prefix;
    rank = s_rank;
    __syncthreads();
  }
  if (threadIdx.x == 0) tau[j] = fkey_inv(prefix);
}

// ------------------------------------------------------------------ codes
__global__ void k_build_codes(const float *lg, int64_t m, int b, const float *tau,
                              uint32_t *codes, uint32_t *sizes) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
    uint32_t c = 0;
    for (int j = 0; j < b; ++j) c |= (lg[i * b + j] >= tau[j] ? 1u : 0u) << j;
    codes[i] = c;
    atomicAdd(&sizes[c], 1u);
  }
}

// clusters per bucket: rule NR_CLUSTER_CAPACITY: ceil(size / t); FIXED:
// min(size, t); NONE: min(size, 1)
__global__ void k_build_kb(const uint32_t *sizes, int64_t nb, int rule, uint32_t t, uint32_t *kb,
                           uint32_t *multi) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nb; c += stride) {
    const uint32_t s = sizes[c];
    uint32_t k;
    if (rule == NR_CLUSTER_CAPACITY) k = (s + t - 1) / t;
    else if (rule == NR_CLUSTER_FIXED) k = s < t ? s : t;
    else k = s < 1u ? s : 1u;
    kb[c] = k;
    multi[c] = k >= 2 ? 1u : 0u;
  }
}

__global__ void k_build_multi_list(const uint32_t *multi, const uint32_t *mpos, int64_t nb,
                                   uint32_t *mlist) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nb; c += stride)
    if (multi[c]) mlist[mpos[c]] = (uint32_t)c;
}

// ------------------------------------------------------------------ buckets
__global__ void k_build_scatter(const uint32_t *codes, int64_t n, const uint64_t *boff,
                                uint32_t *cursor, uint32_t *ids) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint32_t c = codes[i];
    const uint64_t pos = boff[c] + atomicAdd(&cursor[c], 1u);
    if (pos < boff[c + 1]) ids[pos] = (uint32_t)i;   // sizes and codes agree
  }
}

// Ascending sort of keys[0, n) by one block: bitonic in LDS for n <= SORT_LDS,
// else a stable LSD radix sort over 4-bit digits through tmp[0, n).
template <class K>
__device__ void block_sort(K *keys, int64_t n, K *tmp, int key_bits) {
  __shared__ K lds[SORT_LDS];
  __shared__ uint32_t cnt[16][BT];
  __shared__ uint32_t shs[BT / WAVE];
  if (n <= 1) return;
  if (n <= SORT_LDS) {
    int p2 = 1;
    while (p2 < n) p2 <<= 1;
    for (int i = threadIdx.x; i < p2; i += BT) lds[i] = i < n ? keys[i] : (K)~(K)0;
    __syncthreads();
    for (int k = 2; k <= p2; k <<= 1)
      for (int jj = k >> 1; jj > 0; jj >>= 1) {
        for (int i = threadIdx.x; i < p2; i += BT) {
          const int l = i ^ jj;
          if (l > i) {
            const K a = lds[i], c = lds[l];
            const bool up = (i & k) == 0;
            if ((a > c) == up) {
              lds[i] = c;
              lds[l] = a;
            }
          }
        }
        __syncthreads();
      }
    for (int i = threadIdx.x; i < n; i += BT) keys[i] = lds[i];
    __syncthreads();
    return;
  }
  const int64_t per = (n + BT - 1) / BT;
  const int64_t i0 = (int64_t)threadIdx.x * per;
  const int64_t i1 = i0 + per < n ? i0 + per : n;
  K *src = keys, *dst = tmp;
  for (int shift = 0; shift < key_bits; shift += 4) {
    for (int d = 0; d < 16; ++d) cnt[d][threadIdx.x] = 0;
    for (int64_t i = i0; i < i1; ++i) cnt[(src[i] >> shift) & 15][threadIdx.x] += 1;
    __syncthreads();
    // exclusive offsets in (digit, thread) order: thread t owns digit t / 16's
    // columns 16 (t % 16) .. 16 (t % 16) + 15
    const int dg = threadIdx.x / 16, c0 = (threadIdx.x % 16) * 16;
    uint32_t loc = 0;
    for (int c = 0; c < 16; ++c) loc += cnt[dg][c0 + c];
    uint32_t tot;
    uint32_t run = block_excl_scan<uint32_t>(loc, shs, &tot);
    __syncthreads();
    for (int c = 0; c < 16; ++c) {
      const uint32_t x = cnt[dg][c0 + c];
      cnt[dg][c0 + c] = run;
      run += x;
    }
    __syncthreads();
    for (int64_t i = i0; i < i1; ++i) {
      const K k = src[i];
      const int d = (int)((k >> shift) & 15);
      dst[cnt[d][threadIdx.x]++] = k;
    }
    __syncthreads();
    K *t = src;
    src = dst;
    dst = t;
  }
  if (src != keys)
    for (int64_t i = threadIdx.x; i < n; i += BT) keys[i] = src[i];
  __syncthreads();
}

// one block per bucket: its ids ascending
__global__ void __launch_bounds__(BT) k_build_sort_ids(uint32_t *ids, const uint64_t *boff,
                                                        uint32_t *tmp) {
  const int64_t c = blockIdx.x;
  const uint64_t s0 = boff[c], s1 = boff[c + 1];
  block_sort<uint32_t>(ids + s0, (int64_t)(s1 - s0), tmp + s0, 32);
}

// ------------------------------------------------------------------ k-means
struct KmArgs {
  const float *lg;          // [n x b] latents by original id
  int b;
  const uint64_t *boff;     // [nb + 1] bucket row offsets
  const uint32_t *ids;      // [n] ids in bucket order, ascending inside a bucket
  const uint32_t *kb;       // [nb]
  const uint64_t *kbpre;    // [nb + 1] exclusive scan of kb: cluster slots of a bucket
  const uint32_t *mlist;    // [n_multi] buckets with kb >= 2, ascending
  const double *U;          // [n_multi x kmax]
  int kmax;
  uint32_t seed;
  int lloyd, spc;
  uint64_t *skey;           // [n] scratch: sample keys, in bucket order
  uint64_t *skey_tmp;       // [n] sort scratch
  double *d2;               // [n] scratch
  uint32_t *label;          // [n] label of each member (bucket order), renumbered at the end
  double *cent;             // [max_clusters x b] centres, by slot
  uint32_t *ccnt;           // [max_clusters] members per slot
  uint32_t *nkept;          // [nb] clusters kept per bucket (written for multi buckets)
};

__global__ void __launch_bounds__(BT) k_build_kmeans(KmArgs a) {
  __shared__ int64_t sh64[BT / WAVE];
  __shared__ uint32_t shu[BT / WAVE];
  __shared__ int64_t s_pick;
  const int mi = blockIdx.x;
  const uint32_t code = a.mlist[mi];
  const uint64_t s0 = a.boff[code];
  const int64_t m = (int64_t)(a.boff[code + 1] - s0);
  const int K = (int)a.kb[code];
  const int b = a.b;
  const uint32_t *mid = a.ids + s0;
  double *C = a.cent + a.kbpre[code] * b;
  uint32_t *cnt = a.ccnt + a.kbpre[code];
  uint32_t *lab = a.label + s0;
  double *D2 = a.d2 + s0;
  // the sample: members by (mix32(id), id), the first S of them
  uint64_t *sk = a.skey + s0;
  for (int64_t i = threadIdx.x; i < m; i += BT)
    sk[i] = ((uint64_t)mix32_dev(mid[i], a.seed) << 32) | mid[i];
  __syncthreads();
  block_sort<uint64_t>(sk, m, a.skey_tmp + s0, 64);
  int64_t S = m;
  if ((int64_t)a.spc * K < S) S = (int64_t)a.spc * K;
  if (S > (int64_t)(1 << 21)) S = (int64_t)1 << 21;
  // k-means++: the first centre is the first sampled member
  {
    const float *x0 = a.lg + (uint64_t)(uint32_t)sk[0] * b;
    for (int j = threadIdx.x; j < b; j += BT) C[j] = (double)x0[j];
  }
  __syncthreads();
  for (int64_t s = threadIdx.x; s < S; s += BT)
    D2[s] = sqd_row(a.lg + (uint64_t)(uint32_t)sk[s] * b, C, b);
  __syncthreads();
  const int64_t per = (S + BT - 1) / BT;
  const int64_t c0 = (int64_t)threadIdx.x * per;
  const int64_t c1 = c0 + per < S ? c0 + per : S;
  for (int r = 1; r < K; ++r) {
    int64_t wsum = 0;
    for (int64_t s = c0; s < c1; ++s) wsum += d2_weight(D2[s]);
    int64_t tot;
    int64_t run = block_excl_scan<int64_t>(wsum, sh64, &tot);
    if (threadIdx.x == 0) s_pick = S;
    __syncthreads();
    int64_t pick = 0;
    if (tot > 0) {
      const int64_t target = (int64_t)floor(a.U[(int64_t)mi * a.kmax + r] * (double)tot);
      int64_t mine = S;
      for (int64_t s = c0; s < c1; ++s) {
        run += d2_weight(D2[s]);
        if (run > target) {
          mine = s;
          break;
        }
      }
      if (mine < S) atomicMin((unsigned long long *)&s_pick, (unsigned long long)mine);
      __syncthreads();
      pick = s_pick < S ? s_pick : S - 1;
    }
    const float *xp = a.lg + (uint64_t)(uint32_t)sk[pick] * b;
    for (int j = threadIdx.x; j < b; j += BT) C[(int64_t)r * b + j] = (double)xp[j];
    __syncthreads();
    for (int64_t s = threadIdx.x; s < S; s += BT) {
      const double d = sqd_row(a.lg + (uint64_t)(uint32_t)sk[s] * b, C + (int64_t)r * b, b);
      if (d < D2[s]) D2[s] = d;
    }
    __syncthreads();
  }
  // Lloyd passes over every member (in id order)
  for (int it = 0; it < a.lloyd; ++it) {
    for (int64_t i = threadIdx.x; i < m; i += BT) {
      const float *x = a.lg + (uint64_t)mid[i] * b;
      double best = sqd_row(x, C, b);
      int bk = 0;
      for (int k = 1; k < K; ++k) {
        const double d = sqd_row(x, C + (int64_t)k * b, b);
        if (d < best) {
          best = d;
          bk = k;
        }
      }
      lab[i] = (uint32_t)bk;
    }
    __syncthreads();
    // each (k, j) sums its members in id order
    for (int kj = threadIdx.x; kj < K * b; kj += BT) {
      const int k = kj / b, j = kj % b;
      double sum = 0.0;
      uint32_t n_k = 0;
      for (int64_t i = 0; i < m; ++i)
        if (lab[i] == (uint32_t)k) {
          sum = sum + (double)a.lg[(uint64_t)mid[i] * b + j];
          ++n_k;
        }
      if (n_k > 0) C[(int64_t)k * b + j] = sum / (double)n_k;
      if (j == 0) cnt[k] = n_k;
    }
    __syncthreads();
  }
  // kept clusters (non-empty), renumbered in order
  if (threadIdx.x == 0) {
    uint32_t nk = 0;
    for (int k = 0; k < K; ++k) nk += cnt[k] > 0 ? 1u : 0u;
    a.nkept[code] = nk;
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < m; i += BT) {
    const uint32_t k = lab[i];
    uint32_t nr = 0;
    for (uint32_t k2 = 0; k2 < k; ++k2) nr += cnt[k2] > 0 ? 1u : 0u;
    lab[i] = nr;
  }
  (void)shu;
}

// clusters of each bucket: 0 (empty), 1 (K_B = 1) or the kept count
__global__ void k_build_ncl(const uint32_t *sizes, const uint32_t *kb, const uint32_t *nkept,
                            int64_t nb, uint32_t *ncl) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nb; c += stride)
    ncl[c] = sizes[c] == 0 ? 0u : (kb[c] >= 2 ? nkept[c] : 1u);
}

struct FinArgs {
  const float *lg;
  int b;
  const uint64_t *boff;
  const uint32_t *ids, *kb, *label, *ccnt;
  const uint64_t *kbpre;
  const double *cent;
  const uint32_t *bc_off;
  int64_t *row_ids;        // [n] out
  uint64_t *csize;         // [n_clusters] out: rows per cluster
  float *centroids;        // [n_clusters x b] out
};

// one block per bucket: rows in (cluster, id) order, cluster sizes, centroids
__global__ void __launch_bounds__(BT) k_build_finish(FinArgs a) {
  __shared__ uint32_t shu[BT / WAVE];
  const int64_t c = blockIdx.x;
  const uint64_t s0 = a.boff[c];
  const int64_t m = (int64_t)(a.boff[c + 1] - s0);
  if (m == 0) return;
  const int b = a.b;
  const uint32_t *mid = a.ids + s0;
  const uint32_t g0 = a.bc_off[c];
  if (a.kb[c] < 2) {  // one cluster: rows in id order, fp64 mean in id order
    for (int64_t i = threadIdx.x; i < m; i += BT) a.row_ids[s0 + i] = mid[i];
    for (int j = threadIdx.x; j < b; j += BT) {
      double sum = 0.0;
      for (int64_t i = 0; i < m; ++i) sum = sum + (double)a.lg[(uint64_t)mid[i] * b + j];
      a.centroids[(uint64_t)g0 * b + j] = (float)(sum / (double)m);
    }
    if (threadIdx.x == 0) a.csize[g0] = (uint64_t)m;
    return;
  }
  const uint32_t nk = a.bc_off[c + 1] - g0;
  const uint32_t *lab = a.label + s0;
  const uint32_t K = a.kb[c];
  const uint64_t slot0 = a.kbpre[c];
  // kept slots in order -> clusters g0 .. g0 + nk - 1
  uint64_t pos = s0;
  uint32_t kk = 0;
  for (uint32_t k = 0; k < K; ++k) {
    const uint32_t n_k = a.ccnt[slot0 + k];
    if (n_k == 0) continue;
    const uint32_t g = g0 + kk;
    for (int j = threadIdx.x; j < b; j += BT)
      a.centroids[(uint64_t)g * b + j] = (float)a.cent[(slot0 + k) * b + j];
    if (threadIdx.x == 0) a.csize[g] = n_k;
    // members with label kk, in id order: a block scan per round of BT members
    for (int64_t r0 = 0; r0 < m; r0 += BT) {
      const int64_t i = r0 + threadIdx.x;
      const uint32_t f = (i < m && lab[i] == kk) ? 1u : 0u;
      uint32_t tot;
      const uint32_t ex = block_excl_scan<uint32_t>(f, shu, &tot);
      if (f) a.row_ids[pos + ex] = mid[i];
      pos += tot;
      __syncthreads();
    }
    ++kk;
  }
  (void)nk;
}

// ------------------------------------------------------------------ launches
hipError_t launch_build_tau(const float *lg, int64_t ns, int b, float *tau, hipStream_t s) {
  hipLaunchKernelGGL(k_build_tau, dim3((unsigned)b), dim3(BT), 0, s, lg, ns, b, tau);
  return hipGetLastError();
}

hipError_t launch_build_codes(const float *lg, int64_t m, int b, const float *tau, uint32_t *codes,
                              uint32_t *sizes, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  int64_t blocks = (m + BT - 1) / BT;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_build_codes, dim3((unsigned)blocks), dim3(BT), 0, s, lg, m, b, tau, codes,
                     sizes);
  return hipGetLastError();
}

static dim3 grid_for(int64_t items) {
  int64_t g = (items + BT - 1) / BT;
  return dim3((unsigned)(g > 65536 ? 65536 : (g < 1 ? 1 : g)));
}

__global__ void k_build_nonempty(const uint32_t *sizes, int64_t nb, unsigned long long *out) {
  __shared__ unsigned long long sh[BT / WAVE];
  unsigned long long c = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nb; i += stride)
    c += sizes[i] > 0 ? 1ull : 0ull;
  unsigned long long tot;
  (void)block_excl_scan<unsigned long long>(c, sh, &tot);
  if (threadIdx.x == 0) atomicAdd(out, tot);
}

// stats[0] = sum kb, stats[1] = buckets with kb >= 2, stats[2] = max kb
__global__ void k_build_kb_stats(const uint32_t *kb, int64_t nb, unsigned long long *stats) {
  __shared__ unsigned long long sh[BT / WAVE];
  unsigned long long sum = 0, nm = 0, mx = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nb; i += stride) {
    const uint32_t k = kb[i];
    sum += k;
    nm += k >= 2 ? 1ull : 0ull;
    mx = k > mx ? k : mx;
  }
  unsigned long long t;
  (void)block_excl_scan<unsigned long long>(sum, sh, &t);
  if (threadIdx.x == 0) atomicAdd(&stats[0], t);
  (void)block_excl_scan<unsigned long long>(nm, sh, &t);
  if (threadIdx.x == 0) atomicAdd(&stats[1], t);
  atomicMax(&stats[2], mx);
}

hipError_t launch_build_nonempty(const uint32_t *sizes, int64_t nb, unsigned long long *out,
                                 hipStream_t s) {
  hipLaunchKernelGGL(k_build_nonempty, grid_for(nb), dim3(BT), 0, s, sizes, nb, out);
  return hipGetLastError();
}

hipError_t run_build_plan(const BuildArgs &A, hipStream_t s) {
  const int64_t nb = (int64_t)1 << A.b;
  hipError_t e;
  hipLaunchKernelGGL(k_build_kb, grid_for(nb), dim3(BT), 0, s, A.sizes, nb, A.rule, A.t, A.kb,
                     A.multi);
  hipLaunchKernelGGL(k_build_kb_stats, grid_for(nb), dim3(BT), 0, s, A.kb, nb, A.stats);
  if ((e = launch_scan(A.multi, nb, A.mpos, A.blk, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_build_multi_list, grid_for(nb), dim3(BT), 0, s, A.multi, A.mpos, nb,
                     A.mlist);
  return hipGetLastError();
}

hipError_t run_build_index(const BuildArgs &A, hipStream_t s) {
  const int64_t nb = (int64_t)1 << A.b;
  const int64_t n = A.n;
  hipError_t e;
  if ((e = launch_scan(A.kb, nb, A.kbpre, A.blk, s)) != hipSuccess) return e;
  // bucket order of the row ids
  if ((e = launch_scan(A.sizes, nb, A.boff, A.blk, s)) != hipSuccess) return e;
  if ((e = launch_fill_i32((int32_t *)A.cursor, nb, 0, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_build_scatter, grid_for(n), dim3(BT), 0, s, A.codes, n, A.boff, A.cursor,
                     A.ids);
  hipLaunchKernelGGL(k_build_sort_ids, dim3((unsigned)nb), dim3(BT), 0, s, A.ids, A.boff,
                     A.ids_tmp);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // k-means of the multi-cluster buckets
  if ((e = launch_fill_i32((int32_t *)A.nkept, nb, 0, s)) != hipSuccess) return e;
  if (A.n_multi > 0) {
    KmArgs k{};
    k.lg = A.lg;
    k.b = A.b;
    k.boff = A.boff;
    k.ids = A.ids;
    k.kb = A.kb;
    k.kbpre = A.kbpre;
    k.mlist = A.mlist;
    k.U = A.U;
    k.kmax = A.kmax;
    k.seed = A.seed;
    k.lloyd = A.lloyd;
    k.spc = A.spc;
    k.skey = A.skey;
    k.skey_tmp = A.skey_tmp;
    k.d2 = A.d2;
    k.label = A.label;
    k.cent = A.cent;
    k.ccnt = A.ccnt;
    k.nkept = A.nkept;
    hipLaunchKernelGGL(k_build_kmeans, dim3((unsigned)A.n_multi), dim3(BT), 0, s, k);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // directory, rows, cluster sizes, centroids
  hipLaunchKernelGGL(k_build_ncl, grid_for(nb), dim3(BT), 0, s, A.sizes, A.kb, A.nkept, nb, A.ncl);
  if ((e = launch_scan(A.ncl, nb, A.bc_off, A.blk, s)) != hipSuccess) return e;
  FinArgs f{};
  f.lg = A.lg;
  f.b = A.b;
  f.boff = A.boff;
  f.ids = A.ids;
  f.kb = A.kb;
  f.label = A.label;
  f.ccnt = A.ccnt;
  f.kbpre = A.kbpre;
  f.cent = A.cent;
  f.bc_off = A.bc_off;
  f.row_ids = A.row_ids;
  f.csize = A.csize;
  f.centroids = A.centroids;
  hipLaunchKernelGGL(k_build_finish, dim3((unsigned)nb), dim3(BT), 0, s, f);
  return hipGetLastError();
}

hipError_t launch_build_cl_off(const uint64_t *csize, int64_t n_clusters, uint64_t *cl_off,
                               uint64_t *blk, hipStream_t s) {
  return launch_scan(csize, n_clusters, cl_off, blk, s);
}

}  // namespace nr
