// Step 4: the centroid stage of Algorithm 2 (Sec. 3.4.2), one wavefront per
// query, on the bucket ranges the probe kernel looked up in the CSR directory.
//
// Bins are visited in increasing order; every visited bin increments b_proc.
// A probed bucket with one cluster goes straight to C_dir; the clusters of
// multi-cluster buckets form C_z (probe order, then cluster id) and are scored
// in batches of <= B_batch, one centroid per lane:
//   d_c = squared L2 in logit space, acc = fmaf(t, t, acc) over dims in order;
//   d_min tracks the best distance, theta = d_min + M(d_min) gates the heap;
//   H <- the K_c smallest (d, cluster) of (H u batch) with d <= theta;
//   u_heap / u_front count batch entries kept in H (and within the front
//   d_min + alpha_front * M(d_min)); t_low counts consecutive low batches;
//   stop once |H| = K_c, b_proc >= B_min and t_low >= T_low.
// C(q) = C_dir (visiting order) followed by H in (d, cluster) order.
//
// While the kept keys cannot reach K_c, H is an unsorted pool, sorted and
// pruned once (see route_query).  After that H is a sorted array of u64 keys
// (d bits << 32 | cluster) in LDS, for larger heaps fronted by a sorted
// 64-key staging buffer.  A batch is sorted across the wave, then merged by
// ranks: batch element i lands at slot i + |{h < key_i}|, and the other slots
// of the moving tail take the old keys in order; the tail is rewritten from
// the top down, 64 slots at a time, so no key is overwritten before it is
// read.  A batch that cannot push H past K_c merges into the buffer, which
// moves into H when it fills, before a batch that needs the K_c-smallest cut,
// and at the end.  The per-query pass stages the ranges of its first pst
// probes in LDS with one round of loads and walks them 64 at a time.
#include "nr_internal.h"

namespace nr {

constexpr int ROUTE_DIRECT_HEAP = 256;  // below this many keys H takes batches directly

struct RouteLds {
  uint32_t wc0[WAVE], wc1[WAVE];  // probe window: cluster ranges
  int32_t wbin[WAVE];
  uint32_t wpre[WAVE];            // exclusive prefix of multi-cluster sizes
  uint32_t pend[WAVE];            // pending batch (cluster ids)
  uint64_t bkey[WAVE];            // sorted batch keys
  float wd[WAVE];                 // distances of the window's first multi-bucket clusters
  int32_t mk[WAVE];               // merge: batch element (+1) landing in each slot of a chunk
  float lq[32];                   // the query's logits (read by every lane at once)
};

// M(x): piecewise linear through the knots, constant outside them.  Knot j
// sits in lane j (kx, ky, ks); the segment is the last i whose next knot is
// not above x, found with one ballot
__device__ __forceinline__ float margin_dev(int m, float kx, float ky, float ks, float x) {
  const int lane = lane_id();
  if (m <= 0) return 0.0f;
  const float x0 = bcast_f32(kx, 0), y0 = bcast_f32(ky, 0);
  if (m == 1 || x <= x0) return y0;
  if (x >= bcast_f32(kx, m - 1)) return bcast_f32(ky, m - 1);
  const uint64_t above = ballot(lane >= 1 && lane <= m - 2 && !(kx <= x));
  const int i = (above ? __ffsll((unsigned long long)above) - 1 : m - 1) - 1;
  const float yi = bcast_f32(ky, i), yn = bcast_f32(ky, i + 1);
  float v = fmaf(x - bcast_f32(kx, i), bcast_f32(ks, i), yi);
  v = v < yi ? yi : v;
  v = v > yn ? yn : v;
  return v;
}

// minimum over the wave with DPP moves inside each row of 16 lanes (pairs,
// quads, half rows, rows) and the four row minima read from lanes 0, 16, 32
// and 48; exact, like any order of fminf over finite values and +inf
__device__ __forceinline__ float route_min_f32(float v) {
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0xB1, 0xF, 0xF, false)));
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x4E, 0xF, 0xF, false)));
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x141, 0xF, 0xF, false)));
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x140, 0xF, 0xF, false)));
  return fminf(fminf(bcast_f32(v, 0), bcast_f32(v, 16)), fminf(bcast_f32(v, 32), bcast_f32(v, 48)));
}

// the keys of lanes 0..n-1 in ascending order (lanes from n on keep theirs):
// each lane counts the keys ranked before its own (by value, then lane) from
// scalar broadcasts and places its key at that rank through tmp[0, n) in LDS;
// for small n this is far shorter than a shuffle network
__device__ __forceinline__ uint64_t rank_sort_u64(uint64_t key, int n, uint64_t *tmp) {
  const int l = lane_id();
  const int klo = (int)(uint32_t)key, khi = (int)(uint32_t)(key >> 32);
  int r = 0;
  for (int j = 0; j < n; ++j) {
    const uint64_t kj = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(khi, j) << 32) |
                        (uint32_t)__builtin_amdgcn_readlane(klo, j);
    r += (kj < key || (kj == key && j < l)) ? 1 : 0;
  }
  __builtin_amdgcn_wave_barrier();
  if (l < n) tmp[r] = key;
  __builtin_amdgcn_wave_barrier();
  return l < n ? tmp[l] : key;
}

// entries of sorted a[0..n) below key, the same key in every lane: each round
// samples 64 evenly spaced entries and keeps the gap the key falls in
__device__ __forceinline__ int wave_lower_bound_u64(const uint64_t *a, int n, uint64_t key) {
  const int lane = lane_id();
  int lo = 0, hi = n;
  while (lo < hi) {
    const int chunk = (hi - lo + WAVE - 1) / WAVE;
    const int p = lo + lane * chunk;
    const int c = popc64(ballot(p < hi && a[p] < key));
    if (c == 0) break;
    const int top = lo + c * chunk;
    hi = top < hi ? top : hi;
    lo = lo + (c - 1) * chunk + 1;
  }
  return lo;
}

// Algorithm 2 for query q, one wave.  BUF: the staging buffer in front of H
// (passes whose heap may grow past the light first pass's size; small heaps
// merge straight into H)
template <bool BUF>
__device__ __forceinline__ void route_query(const RouteArgs &a, const int64_t q) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  RouteLds &S = *reinterpret_cast<RouteLds *>(smem_raw);
  uint64_t *H = reinterpret_cast<uint64_t *>(smem_raw + sizeof(RouteLds));
  uint64_t *HB = H + a.hcap;  // the heap's staging buffer (sorted; BUF only)
  uint32_t *st_c0 = reinterpret_cast<uint32_t *>(HB + (BUF ? WAVE : 0));
  uint32_t *st_c1 = st_c0 + a.pst;
  int32_t *st_bin = reinterpret_cast<int32_t *>(st_c1 + a.pst);
  const int lane = lane_id();
  __builtin_amdgcn_wave_barrier();  // the LDS of the block's previous query is done with
  S.mk[lane] = 0;
  const int b = a.b, P = a.P, k_c = a.k_c;
  const int hcap = a.hcap;  // heap slots in LDS (k_c, or fewer in a first pass)
  bool abort_q = false;     // the heap would outgrow hcap (guard: the pass of each
                            // query has room for every cluster it can score)
  const float kx = lane < a.m_knots ? a.m_x[lane] : 0.0f;
  const float ky = lane < a.m_knots ? a.m_y[lane] : 0.0f;
  const float ks = lane < a.m_knots ? a.m_slope[lane] : 0.0f;
  const float lg = lane < b ? a.logits[q * b + lane] : 0.0f;
  if (lane < 32) S.lq[lane] = lg;
  const int cnt = a.counts[q];
  const int32_t *bins = a.bins + q * P;
  uint32_t *out = a.clus + q * a.cap;

  int h = 0, ndir = 0, npend = 0;
  // H = H[0, hh) (sorted, in LDS) united with the staging buffer HB[0, hbn)
  // (sorted): batches that cannot make H overflow K_c merge into the small
  // buffer, which is merged into H only when it fills, at a truncation, and at
  // the end, so H itself moves rarely
  int hh = 0, hbn = 0;
  // Until the kept keys could reach K_c, no key is ever cut and the stop
  // cannot fire (it needs |H| = K_c), so a batch only appends its gated keys
  // to H unsorted: H[0, npool).  theta never rises from batch to batch (M is
  // non-decreasing and d_min never rises), so pruning the pool once by the
  // latest theta leaves what pruning after every batch would; the pool is
  // sorted and pruned when a batch could reach K_c, and at the end.
  bool fastm = true;
  int npool = 0;
  uint64_t cut_last = ~0ull;
  float d_min = INFINITY;
  int b_proc = 0, t_low = 0, n_scored = 0, n_batches = 0;
  bool stop = false;
  const int z_last = cnt > 0 ? bins[cnt - 1] : -1;

  auto full_and_quiet = [&]() {
    return a.early_stop_on && h == k_c && b_proc >= a.b_min && t_low >= a.t_low;
  };

  // distance of one centroid to the query's logits, dimensions in order.
  // The logits come from LDS (S.lq, the same 16 bytes for every lane per
  // load); callers run it on all lanes and mask the result afterwards.
  // Centroid rows of whole 16-byte groups (b a multiple of 4, centroids
  // 16-byte aligned) load 4 coordinates per instruction.
  const bool cvec = (b & 3) == 0 && (reinterpret_cast<uintptr_t>(a.centroids) & 15) == 0;
  auto centroid_dist = [&](uint32_t cid) __attribute__((always_inline)) {
    const float *mu = a.centroids + (int64_t)cid * b;
    // the whole centroid row is loaded at once (b <= 31; unused slots hold
    // coordinate 0 or stay unread), then accumulated in dimension order
    float m[32];
    if (cvec) {
      const float4 *mu4 = reinterpret_cast<const float4 *>(mu);
#pragma unroll
      for (int j4 = 0; j4 < 8; ++j4) {
        const float4 v = 4 * j4 < b ? mu4[j4] : make_float4(0.f, 0.f, 0.f, 0.f);
        m[4 * j4] = v.x;
        m[4 * j4 + 1] = v.y;
        m[4 * j4 + 2] = v.z;
        m[4 * j4 + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 32; ++j) m[j] = mu[j < b ? j : 0];
    }
    // the logits from LDS, the same 16 bytes for every lane
    const float4 *lq4 = reinterpret_cast<const float4 *>(S.lq);
    float acc = 0.0f;
#pragma unroll
    for (int j4 = 0; j4 < 8; ++j4) {
      if (4 * j4 < b) {
        const float4 l4 = lq4[j4];
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (4 * j4 + u < b) {
            const float t = lv[u] - m[4 * j4 + u];
            acc = fmaf(t, t, acc);
          }
        }
      }
    }
    return acc;
  };
  int p = 0;                 // next probe of the sequence
  int wb = 0;                // window: probes [wb, wb + WAVE), slot = lane
  bool have_window = false;
  // S.wd holds the distances of the window's multi-bucket clusters numbered
  // [pbase, pbase + npre) (numbers in window slot order; wtotal in all)
  int npre = 0, pbase = 0;
  uint32_t wtotal = 0;
  auto precompute = [&](int from) __attribute__((always_inline)) {
    const int lim = cnt - wb < WAVE ? cnt - wb : WAVE;
    const int n = (int)wtotal - from < WAVE ? (int)wtotal - from : WAVE;
    uint32_t cid = 0;  // lanes past n score cluster 0 and drop it
    if (lane < n) {
      const uint32_t num = (uint32_t)(from + lane);
      // the slot owning number num: the last slot whose prefix is <= num
      int lo = 0, hi = lim - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (S.wpre[mid] <= num) lo = mid; else hi = mid - 1;
      }
      cid = S.wc0[lo] + (num - S.wpre[lo]);
    }
    const float dc = centroid_dist(cid);
    const float dw = lane < n ? dc : 0.0f;
    __builtin_amdgcn_wave_barrier();
    S.wd[lane] = dw;
    __builtin_amdgcn_wave_barrier();
    pbase = from;
    npre = n;
  };

  // merge the nk keys held sorted in lanes 0..nk-1 into the sorted A[0, an),
  // keeping the first acap slots; returns each lane's key's slot.  From the
  // top down, 64 destination slots at a time: the keys' slots are marked in
  // LDS, and every other slot d takes A[d - (keys below d)]; reads of a chunk
  // come before its writes, and every source lies at or below its slot
  auto merge_keys = [&](uint64_t *A, int an, int acap, uint64_t key, int nk)
      __attribute__((always_inline)) {
    S.bkey[lane] = key;
    __builtin_amdgcn_wave_barrier();
    int pos = WAVE + lane;
    if (lane < nk) pos = lane + lower_bound_u64(A, an, key);
    if (nk > 0) {
      const int d_lo = (int)bcast_u32((uint32_t)pos, 0);  // the first key's slot
      const int d_hi = an + nk < acap ? an + nk : acap;
      for (int c1 = d_hi; c1 > d_lo;) {
        const int c0 = c1 - WAVE > d_lo ? c1 - WAVE : d_lo;
        if (lane < nk && pos >= c0 && pos < c1) S.mk[pos - c0] = lane + 1;
        const int below = popc64(ballot(lane < nk && pos < c0));
        __builtin_amdgcn_wave_barrier();
        const int d = c0 + lane;
        const bool act = d < c1;
        const int m = act ? S.mk[lane] : 0;
        const uint64_t mm = ballot(m > 0);
        uint64_t v = 0;
        if (act) v = m > 0 ? S.bkey[m - 1] : A[d - below - popc64(mm & lanemask_lt())];
        __builtin_amdgcn_wave_barrier();
        if (act) {
          A[d] = v;
          S.mk[lane] = 0;
        }
        __builtin_amdgcn_wave_barrier();
        c1 = c0;
      }
    }
    return pos;
  };
  // the buffer's first nb keys into H[0, nh) (their union fits K_c)
  auto flush = [&](int nh, int nb) __attribute__((always_inline)) {
    hh = nh;
    if (nb > 0) {
      const uint64_t bk = lane < nb ? HB[lane] : ~0ull;
      merge_keys(H, hh, k_c, bk, nb);
      hh += nb;
    }
    hbn = 0;
  };

  // the pool sorted into H[0, hh) and pruned to keys below cutv, 64 keys at
  // a time: a chunk is read into registers, sorted across the wave and merged
  // into the sorted prefix, which never reaches past the chunk just read
  auto normalize = [&](uint64_t cutv) __attribute__((always_inline)) {
    __builtin_amdgcn_wave_barrier();
    int sp = 0;
    for (int c0 = 0; c0 < npool; c0 += WAVE) {
      const int n = npool - c0 < WAVE ? npool - c0 : WAVE;
      uint64_t key = lane < n ? H[c0 + lane] : ~0ull;
      const bool keep = key < cutv;
      const int nk = popc64(ballot(keep));
      key = keep ? key : ~0ull;
      __builtin_amdgcn_wave_barrier();
      if (nk == 0) continue;
      key = wave_sort_u64(key, n);
      merge_keys(H, sp, k_c, key, nk);
      sp += nk;
    }
    hh = sp;
    hbn = 0;
    h = sp;
    npool = 0;
    fastm = false;
  };

  // score the pending batch and fold it into H; with pre >= 0 the batch is
  // window clusters pre, pre + 1, ... (cluster ids cbase, cbase + 1, ...)
  // whose distances may already be in S.wd, else the clusters in S.pend
  auto run_batch = [&](int pre, uint32_t cbase) __attribute__((always_inline)) {
    const int nb = npend;
    n_batches += 1;
    n_scored += nb;
    float d = INFINITY;
    uint32_t cid = 0;
    // a window batch whose distances are not all in S.wd first scores the
    // next 64 of the window's clusters at once
    if (pre >= 0 && (pre < pbase || pre + nb > pbase + npre)) precompute(pre);
    if (lane < nb) cid = pre >= 0 ? cbase + (uint32_t)lane : S.pend[lane];
    if (pre >= 0) {
      if (lane < nb) d = S.wd[pre - pbase + lane];
    } else {
      const float dc = centroid_dist(cid);  // all lanes (cluster 0 past nb)
      if (lane < nb) d = dc;
    }
    float dm = route_min_f32(d);
    d_min = dm < d_min ? dm : d_min;
    const float M = margin_dev(a.m_knots, kx, ky, ks, d_min);
    const float theta = a.gate_on ? d_min + M : INFINITY;
    const float am = a.alpha_front * M;
    const float theta_f = d_min + am;
    const bool valid = lane < nb && d <= theta;
    const uint64_t cut = ((uint64_t)__float_as_uint(theta) + 1ull) << 32;
    if (fastm) {
      const uint64_t vm = ballot(valid);
      const int nvf = popc64(vm);
      if (npool + nvf < k_c && npool + nvf <= hcap) {
        // every gated key is kept: u_heap = their count
        if (valid) H[npool + popc64(vm & lanemask_lt())] = ((uint64_t)__float_as_uint(d) << 32) | cid;
        npool += nvf;
        h = npool;
        cut_last = cut;
        const int u_front = popc64(ballot(valid && d <= theta_f));
        const bool low = a.lowq_or ? (nvf < a.u_heap || u_front < a.u_front)
                                   : (nvf < a.u_heap && u_front < a.u_front);
        t_low = low ? t_low + 1 : 0;
        npend = 0;
        return;
      }
      normalize(cut);
    }
    uint64_t key = valid ? (((uint64_t)__float_as_uint(d) << 32) | cid) : ~0ull;
    key = nb <= 32 ? rank_sort_u64(key, nb, S.bkey) : wave_sort_u64(key, nb);
    const int nv = popc64(ballot(valid));
    // prune H and the buffer to d <= theta (prefixes, as both are sorted)
    const int hvh = wave_lower_bound_u64(H, hh, cut);
    const int hvb = BUF ? wave_lower_bound_u64(HB, hbn, cut) : 0;
    const int hv = hvh + hvb;
    if ((hv + nv < k_c ? hv + nv : k_c) > hcap) {
      abort_q = true;
      stop = true;
      npend = 0;
      return;
    }
    int pos = WAVE + lane;
    if (hv + nv > k_c) {
      // the K_c smallest must be chosen: the buffer goes into H first
      flush(hvh, hvb);
      pos = merge_keys(H, hh, k_c, key, nv);
      hh = hh + nv < k_c ? hh + nv : k_c;
    } else {
      // every valid key is kept: straight into a small H, else into the
      // buffer (emptied into H when full)
      hh = hvh;
      hbn = hvb;
      if (!BUF || (hbn == 0 && hh < ROUTE_DIRECT_HEAP)) {
        pos = merge_keys(H, hh, k_c, key, nv);
        hh += nv;
      } else {
        if (hbn + nv > WAVE) flush(hh, hbn);
        if (nv > 0) pos = merge_keys(HB, hbn, WAVE, key, nv);
        hbn += nv;
      }
    }
    h = hh + hbn;
    const bool kept = lane < nv && pos < k_c;
    const float dk = __uint_as_float((uint32_t)(key >> 32));
    const int u_heap = popc64(ballot(kept));
    const int u_front = popc64(ballot(kept && dk <= theta_f));
    const bool low = a.lowq_or ? (u_heap < a.u_heap || u_front < a.u_front)
                               : (u_heap < a.u_heap && u_front < a.u_front);
    t_low = low ? t_low + 1 : 0;
    npend = 0;
    if (full_and_quiet()) stop = true;
  };

  // the window after the current one is fetched ahead: it usually starts
  // where the current one ends
  // the query's first nst probe ranges are staged in LDS at once; windows
  // copy from there (and read the global ranges only past nst)
  const uint2 *lk = a.lk + q * P;
  const int nst = cnt < a.pst ? cnt : a.pst;
  // the first round's loads cover slots below pst (all inside the query's P
  // slots), so they need not wait for cnt; only slots below nst are kept
  for (int base = 0; base < a.pst && (base == 0 || base < nst); base += 8 * WAVE) {
    uint2 v[8];
    int bv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = base + u * WAVE + lane;
      const int ii = i < a.pst ? i : 0;
      v[u] = lk[ii];
      bv[u] = bins[ii];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = base + u * WAVE + lane;
      if (i < nst) {
        st_c0[i] = v[u].x;
        st_c1[i] = v[u].y;
        st_bin[i] = bv[u];
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
  auto load_window = [&]() {
    wb = p;
    have_window = true;
    const int i = wb + lane;
    uint32_t c0 = 0, c1 = 0;
    int bn = 0x7fffffff;
    if (i < nst) {
      c0 = st_c0[i];
      c1 = st_c1[i];
      bn = st_bin[i];
    } else if (i < cnt) {
      const uint2 cc = lk[i];
      c0 = cc.x;
      c1 = cc.y;
      bn = bins[i];
    }
    S.wc0[lane] = c0;
    S.wc1[lane] = c1;
    S.wbin[lane] = bn;
    __builtin_amdgcn_wave_barrier();
  };

  if (!a.finite) {
    // S_max = +inf: every probe is its own bin.  Runs of bins without a
    // multi-cluster bucket change neither H nor t_low, so they are taken a
    // window at a time; the stop test after each of them can only fire
    // where b_proc reaches B_min, which is found in closed form.
    while (p < cnt && !stop) {
      if (!have_window || p >= wb + WAVE) {
        load_window();
        // the window's multi-bucket clusters, numbered in slot order: the
        // first 64 are scored here at once, so their batches need no loads
        const int limw = cnt - wb < WAVE ? cnt - wb : WAVE;
        const uint32_t wsz = lane < limw ? S.wc1[lane] - S.wc0[lane] : 0u;
        const uint32_t msz = wsz >= 2 ? wsz : 0u;
        const uint32_t incl = wave_incl_scan_u32(msz);
        wtotal = (uint32_t)__shfl((int)incl, WAVE - 1);
        S.wpre[lane] = incl - msz;
        __builtin_amdgcn_wave_barrier();
        npre = 0;
        if (wtotal > 0) precompute(0);
      }
      const int off = p - wb;
      const int lim = cnt - wb < WAVE ? cnt - wb : WAVE;
      const bool valid = lane >= off && lane < lim;
      const uint32_t c0 = S.wc0[lane], c1 = S.wc1[lane];
      const uint32_t sz = valid ? c1 - c0 : 0;
      const uint64_t multi = ballot(sz >= 2);
      const int first_multi = multi ? __ffsll((unsigned long long)multi) - 1 : lim;
      const int nbulk = first_multi - off;
      if (nbulk > 0) {
        int take = nbulk;
        bool stop_here = false;
        if (a.early_stop_on && h == k_c && t_low >= a.t_low) {
          int j = a.b_min - b_proc - 1;
          j = j < 0 ? 0 : j;
          if (j < nbulk) {
            take = j + 1;
            stop_here = true;
          }
        }
        const bool single = lane >= off && lane < off + take && sz == 1;
        const uint64_t sm = ballot(single);
        if (single) out[ndir + popc64(sm & lanemask_lt())] = c0;
        ndir += popc64(sm);
        b_proc += take;
        p += take;
        if (stop_here) {
          stop = true;
          break;
        }
      }
      if (multi != 0 && p == wb + first_multi) {
        // a multi-cluster bucket forms its bin's C_z: batches of B_batch
        b_proc += 1;
        const uint32_t mc0 = S.wc0[first_multi], mc1 = S.wc1[first_multi];
        for (uint32_t v = mc0; v < mc1 && !stop;) {
          uint32_t take = mc1 - v < (uint32_t)a.b_batch ? mc1 - v : (uint32_t)a.b_batch;
          npend = (int)take;
          run_batch((int)(S.wpre[first_multi] + (v - mc0)), v);
          v += take;
        }
        if (!stop && full_and_quiet()) stop = true;
        p += 1;
      }
    }
  } else {
    for (int z = 0; z <= z_last && !stop; ++z) {
      b_proc += 1;
      while (p < cnt) {
        if (!have_window || p >= wb + WAVE) load_window();
        const int off = p - wb;
        // bins are sorted, so the probes of bin z from p are the slots [off, off + run)
        const bool in_run = lane >= off && wb + lane < cnt && S.wbin[lane] == z;
        const int run = popc64(ballot(in_run));
        if (run == 0) break;
        const uint32_t c0 = S.wc0[lane], c1 = S.wc1[lane];
        const uint32_t sz = in_run ? c1 - c0 : 0;
        // single-cluster buckets go to C_dir in probe order
        const bool single = sz == 1;
        const uint64_t sm = ballot(single);
        if (single) out[ndir + popc64(sm & lanemask_lt())] = c0;
        ndir += popc64(sm);
        // clusters of multi-cluster buckets feed the batches (not after a stop)
        if (!stop) {
          const uint32_t msz = sz >= 2 ? sz : 0;
          const uint32_t incl = wave_incl_scan_u32(msz);
          const uint32_t total = __shfl(incl, WAVE - 1);
          S.wpre[lane] = in_run ? incl - msz : 0xffffffffu;
          __builtin_amdgcn_wave_barrier();
          uint32_t v = 0;
          while (v < total && !stop) {
            uint32_t take = (uint32_t)(a.b_batch - npend);
            if (take > total - v) take = total - v;
            if ((uint32_t)lane < take) {
              const uint32_t vi = v + lane;
              // last slot of the run whose prefix is <= vi: zero-size slots share
              // the prefix of the next non-empty one, so this is the owner
              int lo = off, hi = off + run - 1;
              while (lo < hi) {
                int mid = (lo + hi + 1) >> 1;
                if (S.wpre[mid] <= vi) lo = mid; else hi = mid - 1;
              }
              S.pend[npend + lane] = S.wc0[lo] + (vi - S.wpre[lo]);
            }
            __builtin_amdgcn_wave_barrier();
            npend += (int)take;
            v += take;
            if (npend == a.b_batch) run_batch(-1, 0u);
          }
        }
        p += run;
        if (off + run < WAVE) break;  // bin z ends inside this window
      }
      if (!stop && npend > 0) run_batch(-1, 0u);
      npend = 0;
      if (!stop && full_and_quiet()) stop = true;
    }
  }

  if (fastm) normalize(cut_last);
  if (abort_q) {  // unreachable (each query has its pass from k_probe): an empty list, never a stale one
    if (lane == 0) {
      a.redo[q] = a.pass + 1;
      a.nclus[q] = 0;
    }
    return;
  }
  flush(hh, hbn);
  for (int i = lane; i < h; i += WAVE) out[ndir + i] = (uint32_t)H[i];
  if (lane == 0) {
    a.nclus[q] = ndir + h;
    if (a.qstats) {
      int32_t *st = a.qstats + q * NR_QSTATS;
      st[NR_QS_PROBES] = cnt;
      st[NR_QS_CLUSTERS] = ndir + h;
      st[NR_QS_DIRECT] = ndir;
      st[NR_QS_SCORED] = n_scored;
      st[NR_QS_STOPPED] = stop ? 1 : 0;
      st[NR_QS_BATCHES] = n_batches;
    }
  }
  if (a.ph_on) {
    // the shared schedule's pair counts for this query, now that its list is
    // final (the wave reads back what it wrote above)
    __threadfence_block();
    pair_hist_wave(a.ph, q, out, ndir + h);
  }
}

// One query per block; a pass of a tiered route skips the queries assigned
// to another pass
template <bool BUF>
__global__ void __launch_bounds__(64) k_route(RouteArgs a) {
  const int64_t q = blockIdx.x;
  if (q < a.nq && (!a.tiered || a.redo[q] == a.pass)) route_query<BUF>(a, q);
}

size_t route_lds_bytes(int k_c, int pst) {
  // the staging buffer only for heaps past the light first pass's size
  const size_t buf = k_c > ROUTE_LIGHT_HEAP ? WAVE : 0;
  return sizeof(RouteLds) + sizeof(uint64_t) * ((size_t)k_c + buf) + 3 * sizeof(uint32_t) * (size_t)pst;
}

hipError_t launch_route(const RouteArgs &a, hipStream_t s, hipStream_t aux, hipEvent_t fork,
                        hipEvent_t join) {
  if (a.nq <= 0) return hipSuccess;
  // the probe kernel has looked up every probe's bucket range (lk) and, when
  // K_c is past the first heap, written each query's pass (redo)
  // A heap of at most ROUTE_LIGHT_HEAP keys in LDS lets more waves share a
  // CU.  When K_c is larger, each query goes to the pass with the smallest
  // heap (ROUTE_LIGHT_HEAP, ROUTE_MID_HEAP, K_c) that holds every cluster it
  // could score; every pass runs Algorithm 2 whole for its queries, and the
  // passes with larger heaps (few, long queries) run beside the first on the
  // second stream when there is one.
  auto launch = [&](const RouteArgs &b0, int hcap, int pass, hipStream_t st) -> hipError_t {
    RouteArgs b = b0;
    b.hcap = hcap;
    b.pass = pass;
    // stage every probe's range in LDS while the block stays within 48 KiB
    const size_t fixed = route_lds_bytes(hcap, 0);
    const size_t budget = 48 * 1024;
    const size_t room = fixed < budget ? (budget - fixed) / (3 * sizeof(uint32_t)) : 0;
    b.pst = (int)(room < (size_t)b.P ? room : (size_t)b.P);
    const size_t lds = route_lds_bytes(hcap, b.pst);
    const void *fn = hcap > ROUTE_LIGHT_HEAP ? (const void *)k_route<true>
                                             : (const void *)k_route<false>;
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    if (hcap > ROUTE_LIGHT_HEAP)
      hipLaunchKernelGGL(k_route<true>, dim3((unsigned)b.nq), dim3(64), lds, st, b);
    else
      hipLaunchKernelGGL(k_route<false>, dim3((unsigned)b.nq), dim3(64), lds, st, b);
    return hipGetLastError();
  };
  int tiers[3];
  const int nt = route_tiers(a.k_c, tiers);
  if (nt == 1) return launch(a, a.k_c, 0, s);
  hipError_t e = hipSuccess;
  RouteArgs b = a;
  b.tiered = 1;
  if (aux && fork && join) {
    if (e == hipSuccess) e = hipEventRecord(fork, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(aux, fork, 0);
    for (int t = 1; t < nt && e == hipSuccess; ++t) e = launch(b, tiers[t], t, aux);
    if (e == hipSuccess) e = hipEventRecord(join, aux);
    if (e == hipSuccess) e = launch(b, tiers[0], 0, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, join, 0);
    return e;
  }
  for (int t = 0; t < nt && e == hipSuccess; ++t) e = launch(b, tiers[t], t, s);
  return e;
}

}  // namespace nr
