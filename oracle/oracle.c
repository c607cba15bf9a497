/*
 * NeuRoute search oracle -- TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared -pthread.
 * -ffp-contract=off keeps every a*b+c as two roundings unless the code calls
 * fmaf() explicitly, so the arithmetic below is exactly what is written.
 */
#define _POSIX_C_SOURCE 200809L
#include "oracle.h"

#include <float.h>
#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

/* ------------------------------------------------------------------------ */
/* Encoder forward pass (Sec. 3.2.1; architecture Sec. 4.5 and App. A):      */
/* hidden layers Linear -> BatchNorm (eval, folded to an affine) -> ReLU,    */
/* last layer Linear.  Accumulation in fp64, logits rounded to fp32 once.    */
/* ------------------------------------------------------------------------ */

static int64_t layer_param_floats(const or_encoder *enc, int l) {
  int64_t in = enc->widths[l], out = enc->widths[l + 1];
  int hidden = l + 1 < enc->n_layers;
  return out * in + out + (hidden ? 2 * out : 0);
}

static void encode_one(const or_encoder *enc, const void *x, int64_t qi, float *logit, double *mag,
                       double *buf_a, double *buf_b) {
  int d = enc->widths[0];
  for (int j = 0; j < d; ++j) {
    double v = enc->in_dtype == OR_U8 ? (double)((const uint8_t *)x)[qi * d + j]
                                      : (double)((const float *)x)[qi * d + j];
    buf_a[j] = v;
  }
  const float *p = enc->params;
  double *in = buf_a, *out = buf_b;
  for (int l = 0; l < enc->n_layers; ++l) {
    int nin = enc->widths[l], nout = enc->widths[l + 1];
    int hidden = l + 1 < enc->n_layers;
    const float *W = p, *bias = p + (int64_t)nout * nin;
    const float *bs = bias + nout, *bsh = bs + nout;
    for (int o = 0; o < nout; ++o) {
      double z = 0.0, m = 0.0;
      for (int i = 0; i < nin; ++i) {
        double t = in[i] * (double)W[(int64_t)o * nin + i];
        z += t;
        m += fabs(t);
      }
      if (l == 0) { z *= enc->input_scale; m *= enc->input_scale; }
      z += (double)bias[o];
      m += fabs((double)bias[o]);
      if (hidden) {
        z = z * (double)bs[o] + (double)bsh[o];
        out[o] = z > 0.0 ? z : 0.0;
      } else {
        logit[o] = (float)z;
        if (mag) mag[o] = m;
      }
    }
    p += layer_param_floats(enc, l);
    double *t = in; in = out; out = t;
  }
}

static int max_width(const or_encoder *enc) {
  int w = 0;
  for (int l = 0; l <= enc->n_layers; ++l) if (enc->widths[l] > w) w = enc->widths[l];
  return w;
}

int or_encode(const or_encoder *enc, const void *x, int64_t nq, float *logits, double *mag) {
  if (!enc || enc->n_layers < 1 || (!x && nq > 0) || nq < 0) return OR_EINVAL;
  int w = max_width(enc), b = enc->widths[enc->n_layers];
  double *a = malloc(sizeof(double) * w), *c = malloc(sizeof(double) * w);
  if (!a || !c) { free(a); free(c); return OR_ENOMEM; }
  for (int64_t q = 0; q < nq; ++q)
    encode_one(enc, x, q, logits + q * b, mag ? mag + q * b : NULL, a, c);
  free(a); free(c);
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1: bucket enumeration around the base address.                 */
/*   a_q[j] = [l_q[j] >= tau_j]  (Eq. 10);  b_0 = BucketId(a_q), bit j = dim j */
/*   delta_q[j] = |l_q[j] - tau_j|                                           */
/*   S = the L_sel dims with smallest delta (ties: lower dim first)          */
/*   every flip set D of S with 1 <= |D| <= R_max and score s <= S_max, with */
/*   s = sum of delta over D (fp32, added in increasing rank order)          */
/* The probe sequence is the base followed by the flip sets in ascending     */
/* (s, rank-mask) order, cut to the first P entries; a rank-mask has bit r   */
/* set when S[r] is flipped.  bin = Bin(s) for finite S_max (equal-width     */
/* bins), else the position in the sequence (each probe its own bin).        */
/* ------------------------------------------------------------------------ */

typedef struct { float s; uint32_t m; } flipset;

static int cmp_flipset(const void *a, const void *b) {
  const flipset *x = a, *y = b;
  if (x->s < y->s) return -1;
  if (x->s > y->s) return 1;
  return (x->m > y->m) - (x->m < y->m);
}

typedef struct { float v; int j; } dimdev;

static int cmp_dimdev(const void *a, const void *b) {
  const dimdev *x = a, *y = b;
  if (x->v < y->v) return -1;
  if (x->v > y->v) return 1;
  return (x->j > y->j) - (x->j < y->j);
}

static int popcount32(uint32_t v) {
  int c = 0;
  while (v) { v &= v - 1; ++c; }
  return c;
}

static int probes_one(const float *l, int b, const float *tau, int l_sel, int r_max,
                      float s_max, int n_bins, int P, uint32_t *codes, float *costs, int32_t *bins,
                      flipset *all) {
  uint32_t b0 = 0;
  dimdev dd[32];
  for (int j = 0; j < b; ++j) {
    if (l[j] >= tau[j]) b0 |= 1u << j;             /* a_q[j] */
    dd[j].v = fabsf(l[j] - tau[j]);                /* delta_q[j] */
    dd[j].j = j;
  }
  qsort(dd, b, sizeof(dimdev), cmp_dimdev);         /* SmallestKIndices */
  int S[32];
  float dS[32];
  for (int r = 0; r < l_sel; ++r) { S[r] = dd[r].j; dS[r] = dd[r].v; }

  int finite = isfinite(s_max);
  int64_t cnt = 0;
  uint32_t nm = (uint32_t)1 << l_sel;               /* l_sel <= 24 here */
  for (uint32_t m = 0; m < nm; ++m) {
    int pc = popcount32(m);
    if (pc > r_max) continue;
    float s = 0.0f;
    for (int r = 0; r < l_sel; ++r)
      if (m >> r & 1u) s = s + dS[r];
    if (m != 0 && !(s <= s_max)) continue;          /* the base is always kept */
    all[cnt].s = s;
    all[cnt].m = m;
    ++cnt;
  }
  qsort(all, cnt, sizeof(flipset), cmp_flipset);
  int n = cnt < P ? (int)cnt : P;
  float bin_scale = finite ? (float)n_bins / s_max : 0.0f;
  for (int i = 0; i < n; ++i) {
    uint32_t code = b0;
    for (int r = 0; r < l_sel; ++r)
      if (all[i].m >> r & 1u) code ^= 1u << S[r];   /* ApplyFlips */
    codes[i] = code;
    costs[i] = all[i].s;
    if (finite) {
      int z = (int)floorf(all[i].s * bin_scale);
      bins[i] = z < n_bins - 1 ? z : n_bins - 1;
    } else {
      bins[i] = i;
    }
  }
  return n;
}

static int probe_args_ok(int b, int l_sel, int r_max, float s_max, int n_bins, int P) {
  if (b < 1 || b > 31 || l_sel < 0 || l_sel > b || l_sel > 24 || r_max < 0 || P < 1) return 0;
  if (isnan(s_max) || s_max < 0.0f) return 0;
  if (isfinite(s_max) && (n_bins < 1 || s_max <= 0.0f)) return 0;
  return 1;
}

int or_probes(const float *logits, int64_t nq, int32_t b, const float *tau,
              int32_t l_sel, int32_t r_max, float s_max, int32_t n_bins, int32_t P,
              uint32_t *codes, float *costs, int32_t *bins, int32_t *counts) {
  if (!probe_args_ok(b, l_sel, r_max, s_max, n_bins, P) || nq < 0) return OR_EINVAL;
  flipset *all = malloc(sizeof(flipset) * ((size_t)1 << l_sel));
  if (!all) return OR_ENOMEM;
  for (int64_t q = 0; q < nq; ++q)
    counts[q] = probes_one(logits + q * b, b, tau, l_sel, r_max, s_max, n_bins, P,
                           codes + q * P, costs + q * P, bins + q * P, all);
  free(all);
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Gate margin curve M(x) (Sec. 3.4 "Centroid gating margin"): monotone      */
/* piecewise-linear through the knots, constant outside them.  Inside        */
/* segment i: fmaf(x - x_i, slope_i, y_i) clamped to [y_i, y_{i+1}], with    */
/* slope_i = (y_{i+1} - y_i) / (x_{i+1} - x_i) in fp32.                      */
/* ------------------------------------------------------------------------ */

float or_margin(const or_route_params *prm, float x) {
  int m = prm->m_knots;
  if (m <= 0) return 0.0f;
  const float *X = prm->m_x, *Y = prm->m_y;
  if (m == 1 || x <= X[0]) return Y[0];
  if (x >= X[m - 1]) return Y[m - 1];
  int i = 0;
  while (i + 1 < m - 1 && X[i + 1] <= x) ++i;
  float slope = (Y[i + 1] - Y[i]) / (X[i + 1] - X[i]);
  float v = fmaf(x - X[i], slope, Y[i]);
  if (v < Y[i]) v = Y[i];
  if (v > Y[i + 1]) v = Y[i + 1];
  return v;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 2: centroid-stage cluster enumeration with calibrated gating.  */
/* Readings:                                                                */
/*  - bins are visited in increasing order; every bin (also an empty one)   */
/*    increments b_proc;                                                    */
/*  - a probed bucket with exactly one cluster goes to C_dir when its bin    */
/*    is visited; empty buckets add nothing;                                */
/*  - C_z lists the clusters of the bin's multi-cluster buckets in probe     */
/*    order, then cluster id; batches are consecutive runs of <= B_batch;    */
/*  - d_cent is the squared L2 distance in logit space, summed over dims in  */
/*    increasing order as acc = fmaf(t, t, acc), t = l_j - mu_cj;            */
/*  - KeepTopKUnderGate: H <- the K_c smallest (d, cluster) of H u batch     */
/*    among entries with d <= theta (pruning H as theta tightens);          */
/*  - u_heap = batch entries that are in H afterwards; u_front = those of    */
/*    them with d <= d_min + alpha_front * M(d_min);                         */
/*  - a batch is low quality when u_heap < U_heap AND u_front < U_front      */
/*    (OR when lowq_or); t_low counts consecutive low-quality batches;       */
/*  - "H is full" means |H| == K_c.                                          */
/* C(q) = C_dir (in visiting order) followed by H in (d, cluster) order.    */
/* ------------------------------------------------------------------------ */

typedef struct { float d; uint32_t c; int from_batch; } hentry;

static int cmp_hentry(const void *a, const void *b) {
  const hentry *x = a, *y = b;
  if (x->d < y->d) return -1;
  if (x->d > y->d) return 1;
  return (x->c > y->c) - (x->c < y->c);
}

static float centroid_distance(const float *l, const float *mu, int b) {
  float acc = 0.0f;
  for (int j = 0; j < b; ++j) {
    float t = l[j] - mu[j];
    acc = fmaf(t, t, acc);
  }
  return acc;
}

static int route_one(const float *l, int b, const uint32_t *codes, const int32_t *bins, int count,
                     const uint32_t *bc_off, const float *centroids, const or_route_params *prm,
                     int k_c, uint32_t *out, int64_t cap, or_route_stats *st, hentry *H,
                     hentry *work, uint32_t *cz) {
  memset(st, 0, sizeof(*st));
  st->n_probes = count;
  int h = 0, n_dir = 0;
  float d_min = INFINITY;
  int b_proc = 0, t_low = 0, stop = 0;
  int finite = isfinite(prm->s_max);
  int n_bins = finite ? prm->n_bins : count;
  int p = 0;
#define FULL_AND_QUIET() \
  (prm->early_stop_on && h == k_c && b_proc >= prm->b_min && t_low >= prm->t_low)

  for (int z = 0; z < n_bins && !stop; ++z) {
    b_proc += 1;
    int p_end = p;
    while (p_end < count && bins[p_end] == z) ++p_end;
    /* singleton buckets of this bin go straight to C_dir */
    int nz = 0;
    for (int i = p; i < p_end; ++i) {
      uint32_t c0 = bc_off[codes[i]], c1 = bc_off[(int64_t)codes[i] + 1];
      if (c1 > c0) st->n_nonempty++;
      if (c1 - c0 == 1) {
        if (n_dir >= cap) return -1;
        out[n_dir++] = c0;
        st->n_singleton++;
      } else if (c1 - c0 >= 2) {
        for (uint32_t c = c0; c < c1; ++c) cz[nz++] = c;   /* MapBucketsToClusters */
      }
    }
    for (int s0 = 0; s0 < nz && !stop; s0 += prm->b_batch) {
      int nb = nz - s0 < prm->b_batch ? nz - s0 : prm->b_batch;
      st->n_batches++;
      st->n_scored += nb;
      float bd[4096];
      float dm = INFINITY;
      for (int i = 0; i < nb; ++i) {
        uint32_t c = cz[s0 + i];
        bd[i] = centroid_distance(l, centroids + (int64_t)c * b, b);
        if (bd[i] < dm) dm = bd[i];
      }
      if (dm < d_min) d_min = dm;
      float M = or_margin(prm, d_min);
      float theta = prm->gate_on ? d_min + M : INFINITY;
      float am = prm->alpha_front * M;
      float theta_f = d_min + am;
      /* KeepTopKUnderGate */
      int w = 0;
      for (int i = 0; i < h; ++i)
        if (H[i].d <= theta) { work[w] = H[i]; work[w].from_batch = 0; ++w; }
      for (int i = 0; i < nb; ++i)
        if (bd[i] <= theta) { work[w].d = bd[i]; work[w].c = cz[s0 + i]; work[w].from_batch = 1; ++w; }
      qsort(work, w, sizeof(hentry), cmp_hentry);
      h = w < k_c ? w : k_c;
      int u_heap = 0, u_front = 0;
      for (int i = 0; i < h; ++i) {
        H[i] = work[i];
        if (work[i].from_batch) {
          ++u_heap;
          if (work[i].d <= theta_f) ++u_front;
        }
      }
      int low = prm->lowq_or ? (u_heap < prm->u_heap || u_front < prm->u_front)
                             : (u_heap < prm->u_heap && u_front < prm->u_front);
      t_low = low ? t_low + 1 : 0;
      if (FULL_AND_QUIET()) stop = 1;
    }
    if (!stop && FULL_AND_QUIET()) stop = 1;
    p = p_end;
    st->bins_done = z + 1;
  }
#undef FULL_AND_QUIET
  st->stopped = stop;
  st->h_size = h;
  st->n_dir = n_dir;
  if (n_dir + h > cap) return -1;
  for (int i = 0; i < h; ++i) out[n_dir + i] = H[i].c;
  return n_dir + h;
}

int or_route(const float *logits, int64_t nq, int32_t b,
             const uint32_t *codes, const int32_t *bins, const int32_t *counts, int32_t P,
             const uint32_t *bc_off, const float *centroids, int64_t n_clusters,
             const or_route_params *prm, uint32_t *clus, int64_t cap, int32_t *n_clus,
             or_route_stats *stats) {
  if (nq < 0 || b < 1 || P < 1 || prm->k_c < 1 || prm->b_batch < 1 || prm->b_batch > 4096)
    return OR_EINVAL;
  int k_c = prm->k_c < n_clusters ? prm->k_c : (int)n_clusters;
  if (k_c < 1) k_c = 1;
  int64_t wn = (int64_t)k_c + prm->b_batch;
  int64_t czn = n_clusters > 0 ? n_clusters : 1;
  hentry *H = malloc(sizeof(hentry) * wn), *work = malloc(sizeof(hentry) * wn);
  uint32_t *cz = malloc(sizeof(uint32_t) * czn);
  int rc = OR_OK;
  if (!H || !work || !cz) { rc = OR_ENOMEM; goto done; }
  for (int64_t q = 0; q < nq; ++q) {
    or_route_stats st;
    int n = route_one(logits + q * b, b, codes + q * P, bins + q * P, counts[q], bc_off,
                      centroids, prm, k_c, clus + q * cap, cap, &st, H, work, cz);
    if (n < 0) { rc = OR_EINVAL; goto done; }
    n_clus[q] = n;
    if (stats) stats[q] = st;
  }
done:
  free(H); free(work); free(cz);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* Exact refinement (Sec. 3.4 intro, Sec. 3.5): every row of every cluster  */
/* of C(q) gets its squared Euclidean distance to q in the original space;  */
/* the k smallest by (distance, original id) are returned, padded with      */
/* (-1, +inf).  uint8: exact int64; fp32: fp64 accumulation.                */
/* ------------------------------------------------------------------------ */

typedef struct { double d; int64_t id; } cand;

static int cand_less(double d1, int64_t i1, double d2, int64_t i2) {
  return d1 < d2 || (d1 == d2 && i1 < i2);
}

static void topk_push(cand *top, int *n, int k, double d, int64_t id) {
  if (*n == k && !cand_less(d, id, top[k - 1].d, top[k - 1].id)) return;
  int i = *n < k ? (*n)++ : k - 1;
  while (i > 0 && cand_less(d, id, top[i - 1].d, top[i - 1].id)) { top[i] = top[i - 1]; --i; }
  top[i].d = d;
  top[i].id = id;
}

static double row_distance(const void *rows, int64_t r, const void *queries, int64_t q, int d,
                           int dtype) {
  if (dtype == OR_U8) {
    const uint8_t *x = (const uint8_t *)rows + r * d, *y = (const uint8_t *)queries + q * d;
    int64_t acc = 0;
    for (int j = 0; j < d; ++j) { int64_t t = (int64_t)x[j] - (int64_t)y[j]; acc += t * t; }
    return (double)acc;
  }
  const float *x = (const float *)rows + r * d, *y = (const float *)queries + q * d;
  double acc = 0.0;
  for (int j = 0; j < d; ++j) { double t = (double)x[j] - (double)y[j]; acc += t * t; }
  return acc;
}

static void write_topk(const cand *top, int n, int k, int64_t *ids, float *dists) {
  for (int i = 0; i < k; ++i) {
    if (i < n) { ids[i] = top[i].id; dists[i] = (float)top[i].d; }
    else { ids[i] = -1; dists[i] = INFINITY; }
  }
}

static int64_t refine_one(const void *rows, int d, int dtype, const int64_t *row_ids,
                          const uint64_t *cl_off, const void *queries, int64_t q,
                          const uint32_t *cl, int ncl, int k, int64_t *ids, float *dists,
                          cand *top) {
  int n = 0;
  int64_t total = 0;
  for (int i = 0; i < ncl; ++i) {
    uint32_t c = cl[i];
    for (uint64_t r = cl_off[c]; r < cl_off[(int64_t)c + 1]; ++r) {
      double dist = row_distance(rows, (int64_t)r, queries, q, d, dtype);
      topk_push(top, &n, k, dist, row_ids ? row_ids[r] : (int64_t)r);
      ++total;
    }
  }
  write_topk(top, n, k, ids, dists);
  return total;
}

int or_refine(const void *rows, int32_t d, int32_t dtype, const int64_t *row_ids,
              const uint64_t *cl_off, const void *queries, int64_t nq,
              const uint32_t *clus, int64_t cap, const int32_t *n_clus, int32_t k,
              int64_t *out_ids, float *out_dists, int64_t *n_cand) {
  if (k < 1 || d < 1 || nq < 0) return OR_EINVAL;
  cand *top = malloc(sizeof(cand) * k);
  if (!top) return OR_ENOMEM;
  for (int64_t q = 0; q < nq; ++q) {
    int64_t t = refine_one(rows, d, dtype, row_ids, cl_off, queries, q, clus + q * cap, n_clus[q],
                           k, out_ids + q * k, out_dists + q * k, top);
    if (n_cand) n_cand[q] = t;
  }
  free(top);
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Whole search and brute force, split over threads by query ranges.        */
/* ------------------------------------------------------------------------ */

typedef struct {
  const or_encoder *enc; const float *tau; int b;
  const void *rows; int d; int dtype; const int64_t *row_ids;
  const uint32_t *bc_off; const uint64_t *cl_off; const float *centroids; int64_t n_clusters;
  const void *queries; int64_t q0, q1; int k; int l_sel, r_max, P;
  const or_route_params *prm;
  int64_t *out_ids; float *out_dists; int64_t *n_cand;
  double secs[4]; int rc;
} search_job;

static double now_s(void) {
  struct timespec ts;
  clock_gettime(CLOCK_MONOTONIC, &ts);
  return ts.tv_sec + 1e-9 * ts.tv_nsec;
}

static void *search_worker(void *arg) {
  search_job *J = arg;
  int b = J->b, P = J->P;
  int k_c = J->prm->k_c < J->n_clusters ? J->prm->k_c : (int)J->n_clusters;
  if (k_c < 1) k_c = 1;
  int64_t cap = (int64_t)P + k_c;
  float *lg = malloc(sizeof(float) * b);
  uint32_t *codes = malloc(sizeof(uint32_t) * P);
  float *costs = malloc(sizeof(float) * P);
  int32_t *bins = malloc(sizeof(int32_t) * P);
  uint32_t *clus = malloc(sizeof(uint32_t) * cap);
  int w = max_width(J->enc);
  double *ba = malloc(sizeof(double) * w), *bb = malloc(sizeof(double) * w);
  J->rc = OR_OK;
  if (!lg || !codes || !costs || !bins || !clus || !ba || !bb) { J->rc = OR_ENOMEM; goto out; }
  for (int64_t q = J->q0; q < J->q1; ++q) {
    int32_t cnt, ncl;
    int rc = OR_OK;
    double t0 = now_s();
    encode_one(J->enc, J->queries, q, lg, NULL, ba, bb);
    double t1 = now_s();
    rc |= or_probes(lg, 1, b, J->tau, J->l_sel, J->r_max, J->prm->s_max, J->prm->n_bins, P,
                    codes, costs, bins, &cnt);
    double t2 = now_s();
    rc |= or_route(lg, 1, b, codes, bins, &cnt, P, J->bc_off, J->centroids, J->n_clusters,
                   J->prm, clus, cap, &ncl, NULL);
    double t3 = now_s();
    rc |= or_refine(J->rows, J->d, J->dtype, J->row_ids, J->cl_off,
                    (const char *)J->queries + q * J->d * (J->dtype == OR_U8 ? 1 : 4), 1, clus,
                    cap, &ncl, J->k, J->out_ids + q * J->k, J->out_dists + q * J->k,
                    J->n_cand ? J->n_cand + q : NULL);
    double t4 = now_s();
    J->secs[0] += t1 - t0; J->secs[1] += t2 - t1; J->secs[2] += t3 - t2; J->secs[3] += t4 - t3;
    if (rc != OR_OK) { J->rc = OR_EINVAL; goto out; }
  }
out:
  free(lg); free(codes); free(costs); free(bins); free(clus); free(ba); free(bb);
  return NULL;
}

int or_search(const or_encoder *enc, const float *tau, int32_t b,
              const void *rows, int32_t d, int32_t dtype, const int64_t *row_ids,
              const uint32_t *bc_off, const uint64_t *cl_off, const float *centroids,
              int64_t n_clusters, const void *queries, int64_t nq, int32_t k,
              int32_t l_sel, int32_t r_max, int32_t P, const or_route_params *prm,
              int32_t n_threads, int64_t *out_ids, float *out_dists, int64_t *n_cand,
              double *stage_seconds) {
  if (n_threads < 1) n_threads = 1;
  if (nq < 0 || k < 1 || enc->widths[0] != d || enc->widths[enc->n_layers] != b) return OR_EINVAL;
  search_job *jobs = calloc(n_threads, sizeof(search_job));
  pthread_t *th = calloc(n_threads, sizeof(pthread_t));
  if (!jobs || !th) { free(jobs); free(th); return OR_ENOMEM; }
  for (int t = 0; t < n_threads; ++t) {
    search_job *J = &jobs[t];
    J->enc = enc; J->tau = tau; J->b = b; J->rows = rows; J->d = d; J->dtype = dtype;
    J->row_ids = row_ids; J->bc_off = bc_off; J->cl_off = cl_off; J->centroids = centroids;
    J->n_clusters = n_clusters; J->queries = queries; J->k = k; J->l_sel = l_sel;
    J->r_max = r_max; J->P = P; J->prm = prm; J->out_ids = out_ids; J->out_dists = out_dists;
    J->n_cand = n_cand;
    J->q0 = nq * t / n_threads;
    J->q1 = nq * (t + 1) / n_threads;
    pthread_create(&th[t], NULL, search_worker, J);
  }
  int rc = OR_OK;
  if (stage_seconds) memset(stage_seconds, 0, 4 * sizeof(double));
  for (int t = 0; t < n_threads; ++t) {
    pthread_join(th[t], NULL);
    if (jobs[t].rc != OR_OK) rc = jobs[t].rc;
    if (stage_seconds) for (int s = 0; s < 4; ++s) stage_seconds[s] += jobs[t].secs[s];
  }
  free(jobs); free(th);
  return rc;
}

typedef struct {
  const void *rows; int64_t n; int d; int dtype; const int64_t *row_ids;
  const void *queries; int64_t q0, q1; int k; int64_t *ids; float *dists; int rc;
} brute_job;

static void *brute_worker(void *arg) {
  brute_job *J = arg;
  cand *top = malloc(sizeof(cand) * J->k);
  if (!top) { J->rc = OR_ENOMEM; return NULL; }
  for (int64_t q = J->q0; q < J->q1; ++q) {
    int n = 0;
    for (int64_t r = 0; r < J->n; ++r)
      topk_push(top, &n, J->k, row_distance(J->rows, r, J->queries, q, J->d, J->dtype),
                J->row_ids ? J->row_ids[r] : r);
    write_topk(top, n, J->k, J->ids + q * J->k, J->dists + q * J->k);
  }
  free(top);
  J->rc = OR_OK;
  return NULL;
}

int or_bruteforce(const void *rows, int64_t n, int32_t d, int32_t dtype, const int64_t *row_ids,
                  const void *queries, int64_t nq, int32_t k, int32_t n_threads,
                  int64_t *out_ids, float *out_dists) {
  if (n < 0 || d < 1 || k < 1 || nq < 0) return OR_EINVAL;
  if (n_threads < 1) n_threads = 1;
  brute_job *jobs = calloc(n_threads, sizeof(brute_job));
  pthread_t *th = calloc(n_threads, sizeof(pthread_t));
  if (!jobs || !th) { free(jobs); free(th); return OR_ENOMEM; }
  for (int t = 0; t < n_threads; ++t) {
    brute_job *J = &jobs[t];
    J->rows = rows; J->n = n; J->d = d; J->dtype = dtype; J->row_ids = row_ids;
    J->queries = queries; J->k = k; J->ids = out_ids; J->dists = out_dists;
    J->q0 = nq * t / n_threads; J->q1 = nq * (t + 1) / n_threads;
    pthread_create(&th[t], NULL, brute_worker, J);
  }
  int rc = OR_OK;
  for (int t = 0; t < n_threads; ++t) { pthread_join(th[t], NULL); if (jobs[t].rc) rc = jobs[t].rc; }
  free(jobs); free(th);
  return rc;
}
