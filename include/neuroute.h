/*
 * neuroute.h -- C ABI of the MI355X (gfx950) batched query-time search of
 * NeuRoute (arXiv 2608.15438).
 *
 * The search returns, for each query q, the k database rows S_k(q) that the
 * method deems nearest under the Euclidean distance (problem statement,
 * Sec. 3.1, Eq. 1-2).  It runs the five query-time steps of the paper:
 *   1. encoder forward pass to logits l_q            (Sec. 3.2.1; Sec. 4.5 "Architecture")
 *   2. binarisation a_j = [l_j >= tau_j] (Eq. 10), deviation scores
 *      delta_j = |l_j - tau_j| and the ordered probe sequence of bucket
 *      enumeration                                    (Sec. 3.4.1, Algorithm 1)
 *   3. bucket lookup in a CSR directory               (Sec. 3.3 "Bucket allocation"; Sec. 3.4 "Implementation")
 *   4. centroid stage with calibrated gate theta = d_min + M(d_min) and
 *      heap-quality early stop                        (Sec. 3.4.2, Algorithm 2)
 *   5. exact refinement of C(q) = C_dir u C_cent in the original space to a
 *      per-query top-k                                (Sec. 3.4 intro; Sec. 3.5)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - DEVICE pointers are HIP device memory of the current device, owned by the
 *   caller.  HOST pointers are ordinary host memory, read during the call.
 * - Work is enqueued on `stream` and the call returns after launch.  Argument
 *   and index errors are reported synchronously as an nr_status and nothing is
 *   enqueued; a HIP launch failure is reported as NR_EDEVICE.  Faults inside a
 *   kernel surface at the caller's next synchronisation of the stream.
 * - No C++ exception crosses this interface.  nr_last_error() returns a
 *   thread-local message describing the last failure of the calling thread.
 * - Distances are SQUARED Euclidean distances (squaring does not change the
 *   ranking, Sec. 3.5); uint8 distances are exact integers, fp32 distances
 *   are accumulated in fp32.  Every result row is sorted by (distance, original
 *   id); rows with fewer than k candidates are padded with id -1, distance +inf.
 * - Calls on one index from different streams may overlap; each stream gets
 *   its own workspace.  The index itself is read-only after upload.
 * - Limits: 1 <= k <= 64, 1 <= probe_budget <= 4096, 1 <= b <= 30,
 *   L_sel <= min(b, 32), 1 <= B_batch <= 64, K_c limited by LDS (16384),
 *   encoder widths <= 4096; anything beyond returns NR_EUNSUPPORTED.
 */
#ifndef NEUROUTE_H
#define NEUROUTE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NR_OK = 0,
  NR_EINVAL = 1,         /* bad argument */
  NR_ENOMEM = 2,         /* device or host allocation failed */
  NR_EDEVICE = 3,        /* a HIP call failed */
  NR_EUNSUPPORTED = 4,   /* valid but beyond the limits above */
  NR_ECORRUPT = 5        /* index arrays fail validation at upload */
} nr_status;

typedef enum { NR_U8 = 0, NR_F32 = 1 } nr_dtype;

#define NR_MAX_LAYERS 8
#define NR_MAX_KNOTS 32
#define NR_MAX_K 64
#define NR_MAX_PROBES 4096

typedef struct nr_index nr_index;   /* opaque, library-owned */

/*
 * Index description (index construction, Sec. 3.3).  Rows are stored permuted
 * so that every bucket-local cluster is one contiguous row span:
 *   bucket (code) c   -> clusters [bc_off[c], bc_off[c+1])
 *   cluster g         -> rows     [cl_off[g], cl_off[g+1])
 *   permuted row r    -> original id row_ids[r]
 * Code bit j is latent dimension j.  The encoder has n_layers linear layers:
 * hidden layers are Linear -> eval-mode BatchNorm folded to a per-channel
 * affine (bn_scale, bn_shift; NULL = identity) -> ReLU; the last layer is
 * Linear and yields the b logits.  The input is multiplied by input_scale
 * (1/255 for uint8 rows).
 */
typedef struct {
  int64_t n;                      /* database rows, >= 1 */
  int32_t d;                      /* E_dim; d * sizeof(element) must be a multiple of 16 */
  int32_t dtype;                  /* nr_dtype of rows and queries */
  int32_t b;                      /* L_dim = number of code bits */
  int32_t n_layers;               /* 1..NR_MAX_LAYERS */
  const int32_t *widths;          /* HOST [n_layers+1]; widths[0] = d, widths[n_layers] = b */
  const float *const *weights;    /* HOST [n_layers] -> HOST [widths[l+1] x widths[l]], row-major */
  const float *const *biases;     /* HOST [n_layers] -> HOST [widths[l+1]]; NULL array or entry = 0 */
  const float *const *bn_scale;   /* HOST [n_layers] -> HOST [widths[l+1]] (hidden layers); NULL = 1 */
  const float *const *bn_shift;   /* HOST, as bn_scale; NULL = 0 */
  float input_scale;
  const float *tau;               /* HOST [b] binarisation thresholds (median per dim, Sec. 3.2.3) */
  /* DEVICE arrays, BORROWED: they must stay valid and unchanged until
   * nr_index_free.  They are never copied (the payload may be ~128 GB). */
  const void *rows;               /* [n x d] permuted payload, 16-byte aligned */
  const int64_t *row_ids;         /* [n] original id of each permuted row (a permutation of 0..n-1) */
  const uint32_t *bc_off;         /* [2^b + 1] non-decreasing, bc_off[0] = 0, bc_off[2^b] = n_clusters */
  const uint64_t *cl_off;         /* [n_clusters + 1] non-decreasing, cl_off[0] = 0, cl_off[n_clusters] = n */
  const float *centroids;         /* [n_clusters x b] cluster centroids in latent space */
  int64_t n_clusters;             /* >= 1, < 2^32 */
  /* Payload layout.  head_bytes = 0: `rows` is row-major [n x row_bytes].
   * Otherwise `rows` starts with a head plane [n x head_bytes] holding the
   * first head_bytes bytes of every permuted row, followed by
   *   head_copy = 0: a tail plane [n x (row_bytes - head_bytes)] (the rest of
   *                  every row; no byte is stored twice), or
   *   head_copy = 1: the whole row-major payload [n x row_bytes] (the heads
   *                  are stored twice; whole rows stay aligned to their size).
   * head_bytes is 16, 32, 64 or 128 and, with head_copy = 0, at most
   * row_bytes - 16.  The shared refinement reads only the heads of the
   * candidate rows that cannot enter a top-k (see NR_REFINE_SHARED). */
  int32_t head_bytes;
  int32_t head_copy;
} nr_index_desc;

/*
 * Query-time knobs of Algorithms 1 and 2 (the "gate params").  Alg. 1 keeps
 * flip sets of the l_sel least stable dimensions with at most r_max flips and
 * score <= s_max; with finite s_max the scores are put in n_bins equal-width
 * bins, with s_max = +inf every probe is its own bin.  The probe sequence is
 * ordered by (score, rank mask) and cut to probe_budget entries.  Alg. 2
 * scores centroids of multi-cluster buckets in batches of <= b_batch, keeps
 * the k_c best under the gate d <= d_min + M(d_min) (gate_on), and stops
 * (early_stop_on) once the heap is full, at least b_min bins were visited and
 * t_low consecutive batches were low quality: fewer than u_heap entries kept
 * OR (lowq_or = 1) / AND (lowq_or = 0) fewer than u_front of them within
 * d_min + alpha_front * M(d_min).  With u_heap = u_front = 1 the OR reading
 * means "no entry reached the front" (alpha_front decides) and the AND
 * reading "no entry was kept" (alpha_front plays no part); the Python
 * binding defaults to the OR reading.  M is piecewise linear through m_knots
 * knots (m_x strictly increasing, m_y non-decreasing), constant outside them,
 * and 0 when m_knots == 0; distances are squared L2 in latent space.
 */
typedef struct {
  int32_t l_sel;
  int32_t r_max;
  float s_max;
  int32_t n_bins;
  int32_t k_c;
  int32_t b_batch;
  int32_t b_min;
  int32_t t_low;
  int32_t u_heap;
  int32_t u_front;
  float alpha_front;
  int32_t gate_on;
  int32_t early_stop_on;
  int32_t lowq_or;
  int32_t refine_mode;   /* NR_REFINE_AUTO / _PER_QUERY / _SHARED (same results) */
  int32_t shared_seed_rows; /* shared schedule: rows of each list's leading clusters
                               kept for the query's own pass (>= k); 0: 4096, or
                               1024 for rows longer than 1024 bytes */
  int32_t m_knots;
  float m_x[NR_MAX_KNOTS];
  float m_y[NR_MAX_KNOTS];
} nr_params;

/* How step 5 is scheduled; both give the same top-k.  PER_QUERY refines each
 * query's candidate rows on their own.  SHARED refines, per query, only the
 * leading clusters of its list (at least shared_seed_rows rows); the exact
 * top-k of those rows bounds the final k-th entry.  Every later (cluster,
 * query) pair goes to one scan over the batch, grouped by cluster: each row's
 * head (the first NR_WORK_HEAD_BYTES bytes) is read once and compared with
 * the bounds of all queries listing its cluster; only rows whose head leaves
 * some query open are read whole, and those at or before the bound are merged
 * into the query's result.  AUTO picks SHARED for batches of at least 512
 * queries.  Distances of rows longer than 1024 bytes are summed per 1 KB slab
 * (each slab reduced over its lanes, the slabs added in order) under both
 * schedules, so the two still agree bit for bit. */
enum { NR_REFINE_AUTO = 0, NR_REFINE_PER_QUERY = 1, NR_REFINE_SHARED = 2 };

/* Per-query counters written by nr_search_ex when `qstats` is not NULL. */
#define NR_QSTATS 8
enum {
  NR_QS_PROBES = 0,      /* probes in the sequence */
  NR_QS_CLUSTERS = 1,    /* |C(q)| */
  NR_QS_DIRECT = 2,      /* |C_dir(q)| */
  NR_QS_SCORED = 3,      /* centroids scored */
  NR_QS_STOPPED = 4,     /* 1 if the early stop fired */
  NR_QS_ROWS = 5,        /* rows refined (candidates), low 32 bits */
  NR_QS_TILES = 6,       /* refinement tiles */
  NR_QS_BATCHES = 7      /* centroid batches */
};

/* Upload an index: validates the description and the device CSR arrays
 * (monotone offsets, bounds, row_ids a permutation), copies the encoder and
 * tau to the device and borrows the DEVICE arrays.  Synchronises `stream`.
 * On success *out owns the library's copies until nr_index_free.  With n = 0
 * and every DEVICE array NULL the index holds only the encoder and tau:
 * nr_encode works on it (to encode a base for index construction), the
 * search entry points return NR_EINVAL. */
nr_status nr_index_upload(const nr_index_desc *desc, nr_index **out, hipStream_t stream);

/* Release an index and its workspaces (synchronises the device). */
nr_status nr_index_free(nr_index *index);

/* Batched search (all five steps).  queries: DEVICE [nq x d] of the index
 * dtype; out_ids: DEVICE int64 [nq x k]; out_dists: DEVICE fp32 [nq x k]. */
nr_status nr_search(const nr_index *index, const void *queries, int64_t nq, int32_t k,
                    int32_t probe_budget, const nr_params *params, int64_t *out_ids,
                    float *out_dists, hipStream_t stream);

/* As nr_search; logits (DEVICE fp32 [nq x b]) replace step 1 when not NULL;
 * qstats (DEVICE int32 [nq x NR_QSTATS]) receives per-query counters when not
 * NULL. */
nr_status nr_search_ex(const nr_index *index, const void *queries, const float *logits,
                       int64_t nq, int32_t k, int32_t probe_budget, const nr_params *params,
                       int64_t *out_ids, float *out_dists, int32_t *qstats, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the search
 * of nr_search_ex (logits optional, no per-query counters) without any
 * allocation.  Its working buffers live in one fixed device array of
 * NR_NOALLOC_SCRATCH_BYTES per GPU, which the library maps when it first
 * uploads an index on that GPU and which stays held until the process ends.
 * The batch runs in chunks of as many queries as that array holds (about
 * 1,500 at P = 304, K_c = 3000, k = 10); refinement always uses the
 * per-query schedule, whatever params->refine_mode says (every schedule
 * returns the same lists).  All calls on one GPU share the array and it keeps
 * the last call's contents: calls that overlap in time on one GPU (other
 * streams or threads) race, so the caller must serialise them.  Returns
 * NR_EUNSUPPORTED when one query's buffers would not fit in the array.  Not
 * covered by nr_last_work or the stage timers. */
#define NR_NOALLOC_SCRATCH_BYTES (64u << 20)
nr_status nr_search_noalloc(const nr_index *index, const void *queries, const float *logits,
                            int64_t nq, int32_t k, int32_t probe_budget, const nr_params *params,
                            int64_t *out_ids, float *out_dists, hipStream_t stream);

/* Step 1 only: logits DEVICE fp32 [nq x b]. */
nr_status nr_encode(const nr_index *index, const void *queries, int64_t nq, float *logits,
                    hipStream_t stream);

/* Step 2 only (Algorithm 1): for each query the first counts[q] <= probe_budget
 * entries of codes/costs/bins (DEVICE [nq x probe_budget]) hold the ordered
 * probe sequence; the rest is unspecified. */
nr_status nr_probe(const nr_index *index, const float *logits, int64_t nq, int32_t probe_budget,
                   const nr_params *params, uint32_t *codes, float *costs, int32_t *bins,
                   int32_t *counts, hipStream_t stream);

/* Steps 2-4: candidate clusters C(q) = C_dir (visiting order) followed by
 * C_cent in (distance, cluster) order.  clusters: DEVICE uint32 [nq x cap],
 * n_clusters: DEVICE int32 [nq].  cap must be >= nr_route_capacity(). */
nr_status nr_route(const nr_index *index, const float *logits, int64_t nq, int32_t probe_budget,
                   const nr_params *params, uint32_t *clusters, int32_t *n_clusters, int64_t cap,
                   hipStream_t stream);

/* Capacity a C(q) list can need: probe_budget + min(k_c, n_clusters). */
int64_t nr_route_capacity(const nr_index *index, int32_t probe_budget, const nr_params *params);

/* Step 5 only: exact top-k over the rows of the given clusters (same layout
 * as nr_route's output). */
nr_status nr_refine(const nr_index *index, const void *queries, int64_t nq, int32_t k,
                    const uint32_t *clusters, const int32_t *n_clusters, int64_t cap,
                    int64_t *out_ids, float *out_dists, hipStream_t stream);

/* Calibration inputs (Sec. 3.4 "Calibration": "Bucket-score cutoff" and
 * "Centroid gating margin"), for calibration queries with known top-K target
 * rows (from a higher-recall run of the search, or exact k-NN):
 *   logits      DEVICE fp32 [nq x b] of the calibration queries;
 *   target_ids  DEVICE int64 [nq x K], original row ids (< 0: no target), K <= 64;
 *   scores      DEVICE fp32 [nq x K] out: the score Algorithm 1 gives each
 *               target's bucket under (l_sel, r_max) -- bit for bit the cost
 *               of that bucket in the probe sequence -- or +inf when the
 *               enumeration cannot reach it;
 *   margin_xy   DEVICE fp32 [nq x 2] out: x = the smallest squared latent
 *               distance from the query to any centroid of a bucket holding a
 *               target, y = the distance of the farthest target's cluster
 *               minus x (x = +inf, y = 0 when the query has no target).
 * The first call on an index builds its inverse permutation (4 bytes per row,
 * freed with the index).  Fitting S_max and M(x) from these arrays is the
 * caller's (quantiles of a few thousand numbers). */
nr_status nr_calibrate(const nr_index *index, const float *logits, int64_t nq,
                       const int64_t *target_ids, int32_t K, int32_t l_sel, int32_t r_max,
                       float *scores, float *margin_xy, hipStream_t stream);

/* Encoder training with the selective similarity loss L_sim (Sec. 3.2.2,
 * the loss of Eq. "similarityconfig" with the mask of Eq. 8), for one
 * mini-batch of B <= 65536 rows.
 * nr_pair_sqdist: out DEVICE fp32 [B x B] = squared Euclidean distances of the
 *   rows of x (DEVICE fp32 [B x D], the inputs as the encoder sees them),
 *   diagonal 0, symmetric bit for bit, computed as |x_i|^2 + |x_j|^2 -
 *   2 x_i.x_j on the fp32 matrix cores after centring the batch on its mean;
 *   ws: DEVICE fp32 scratch of nr_pair_sqdist_ws(B, D) floats.
 * nr_lsim_grad: given those distances (S_emb = their square roots) and the
 *   latents lat (DEVICE fp32 [B x L], L <= 32), with m_ij = [i != j and
 *   (S_emb(i,j) <= tau_emb or S_lat(i,j) <= gamma_rho * tau_emb)] and
 *   d_ij = S_lat(i,j) - gamma_rho * S_emb(i,j) (gamma_rho = gamma * sqrt(L/E)):
 *   num_cnt (DEVICE fp64 [2], overwritten) = (sum m d^2, sum m), so that
 *   L_sim = num / cnt; grad_lat (DEVICE fp32 [B x L]) = cnt * dL_sim/dlat
 *   with the mask held fixed, i.e. sum_j 4 m_ij d_ij (l_i - l_j) / S_lat(i,j)
 *   (d2_emb must be symmetric, as nr_pair_sqdist writes it).  grad_lat and
 *   the mask count are the same bit for bit on every call with the same
 *   inputs; the numerator's last bits may vary (a double-precision atomic). */
size_t nr_pair_sqdist_ws(int64_t B, int32_t D);
nr_status nr_pair_sqdist(const float *x, int64_t B, int32_t D, float *ws, float *out,
                         hipStream_t stream);
nr_status nr_lsim_grad(const float *d2_emb, const float *lat, int64_t B, int32_t L,
                       float gamma_rho, float tau_emb, double *num_cnt, float *grad_lat,
                       hipStream_t stream);

/* ---- Index construction on the GPU (Sec. 3.3 "Bucket allocation" and
 * "In-bucket clustering"; thresholds, Sec. 3.2.3).  Untimed, run once.
 * The latents of the base rows come from nr_encode on an encoder-only index
 * (nr_index_upload with n = 0 and every DEVICE array NULL).  All arrays are
 * DEVICE memory unless marked HOST; calls synchronise `stream` where they
 * return HOST values.  The k-means of multi-cluster buckets: the sample is
 * the first min(|B|, sample_per_cluster * K_B) members ordered by
 * (mix32(id, seed), id); k-means++ from its first member, each further centre
 * drawn by the bucket's uniform U[r] with probability proportional to
 * floor(D^2 * 2^20) (capped at 2^30); then `lloyd` Lloyd passes over the
 * bucket; distances and sums in fp64 in a fixed order; clusters left empty are
 * dropped.  Rows of a cluster are stored in original-id order. */
enum { NR_CLUSTER_NONE = 0, NR_CLUSTER_CAPACITY = 1, NR_CLUSTER_FIXED = 2,
       NR_CLUSTER_PER_BUCKET = 3 };

/* tau [b] = per latent dimension the lower median ((ns - 1) / 2-th smallest)
 * of logits [ns x b]. */
nr_status nr_build_tau(const float *logits, int64_t ns, int32_t b, float *tau, hipStream_t stream);

/* codes [m] = Eq. 10 codes of logits [m x b] under tau [b]; sizes [2^b] is
 * incremented per code (zero it before the first of several calls). */
nr_status nr_build_codes(const float *logits, int64_t m, int32_t b, const float *tau,
                         uint32_t *codes, uint32_t *sizes, hipStream_t stream);

/* Clusters per bucket K_B from the bucket sizes [2^b] of n rows: rule
 * NR_CLUSTER_CAPACITY ceil(size / param), NR_CLUSTER_FIXED min(size, param),
 * NR_CLUSTER_PER_BUCKET capacity t = max(1, round-half-even(mean non-empty
 * size / param)), NR_CLUSTER_NONE min(size, 1).  kb [2^b] out; mlist [2^b]
 * out: the codes with K_B >= 2, ascending, in its first n_multi entries. */
typedef struct {
  int64_t max_clusters;   /* sum of K_B */
  int64_t n_multi;        /* buckets with K_B >= 2 */
  int32_t kmax;           /* largest K_B */
  uint32_t t;             /* capacity used (rules CAPACITY and PER_BUCKET) */
} nr_build_plan_info;
nr_status nr_build_plan(const uint32_t *sizes, int64_t n, int32_t b, int32_t rule, uint32_t param,
                        uint32_t *kb, uint32_t *mlist, nr_build_plan_info *info /* HOST */,
                        hipStream_t stream);

typedef struct {
  int64_t n;
  int32_t b;
  const float *logits;      /* [n x b] latents by original id */
  const uint32_t *codes;    /* [n] */
  const uint32_t *sizes;    /* [2^b] */
  const uint32_t *kb;       /* [2^b] from nr_build_plan */
  const uint32_t *mlist;    /* [n_multi] from nr_build_plan */
  int64_t max_clusters, n_multi;
  int32_t kmax;
  const double *uniforms;   /* [n_multi x kmax] the k-means++ draws, fp64 in (0, 1) */
  uint32_t seed;
  int32_t lloyd;            /* >= 1 */
  int32_t sample_per_cluster;
} nr_build_desc;

/* The index arrays: row_ids [n] (rows in (code, cluster, id) order),
 * bc_off [2^b + 1], cl_off [max_clusters + 1], centroids [max_clusters x b]
 * (fp32 means of the members' latents); *n_clusters (HOST) the clusters kept:
 * the first n_clusters + 1 / n_clusters entries of cl_off / centroids are the
 * index's.  Working memory is allocated and freed inside the call. */
nr_status nr_build_index(const nr_build_desc *desc, int64_t *row_ids, uint32_t *bc_off,
                         uint64_t *cl_off, float *centroids, int64_t *n_clusters,
                         hipStream_t stream);

/* Stage timing with HIP events on the launch stream (off by default).
 * nr_profile_read synchronises the recorded events and returns the summed
 * milliseconds per stage and the number of timed searches since the last
 * reset.  Stages, in launch order:
 *   encode, probe,
 *   route   (shared schedule: also the per-query pair counts, taken by the
 *            route kernel once a query's list is final),
 *   plan    (per-query tiles; shared schedule: seed-pass tiles),
 *   refine  (the per-query refinement kernel; shared schedule: own pass),
 *   merge   (per-query merge; shared schedule: own-pass merge),
 *   shared_prep, shared_scan, shared_open, shared_merge (shared schedule
 *   only; shared_open is the pass over fp32 rows longer than 1024 bytes that
 *   finishes the (row, query) pairs the scan's first 1 KB slab left open).
 *   The scan's preparation runs on a second stream of the library's, beside
 *   the seed pass, so shared_prep counts only the part the seed pass did not
 *   hide; shared_merge includes the per-query redo of queries that lost
 *   survivors. */
#define NR_STAGES 10
nr_status nr_profile_enable(nr_index *index, int32_t on);
nr_status nr_profile_read(nr_index *index, double *stage_ms, int64_t *n_searches, int32_t reset);

/* Work of the last search on `stream` (its last query chunk), synchronising
 * the stream.  Writes min(n_work, NR_WORK) counters into `work` (host):
 *   NR_WORK_TILES          tiles of the per-query refinement kernel
 *   NR_WORK_ROWS           candidate rows summed over queries (sum of |rows of C(q)|)
 *   NR_WORK_ROWS_READ      rows the refinement read from the index
 *   NR_WORK_OWN_ROWS       rows refined by the per-query kernel (all of them for
 *                          the per-query schedule; the own pass for the shared one)
 *   NR_WORK_SHARED_ROWS    rows of shared clusters, each read once by the scan
 *   NR_WORK_SHARED_PAIRS   (query, shared cluster) pairs scored by the scan
 *   NR_WORK_SURVIVORS      rows the scan kept for the merge (before capping)
 *   NR_WORK_FLAGGED        queries recomputed after their survivors overflowed
 *   NR_WORK_FALLBACK_ROWS  rows read by that recomputation
 *   NR_WORK_SHARED_PAIR_ROWS rows scored by the scan, summed over its pairs
 *   NR_WORK_FULL_ROWS      rows the scan read past their head (it left a query open)
 *   NR_WORK_HEAD_BYTES     bytes of a row the scan reads for every row (its head)
 *   NR_WORK_BODY_BYTES     bytes the scan read from those rows: whole rows (for
 *                          fp32 rows longer than 1024 bytes, their first 1 KB slab)
 *   NR_WORK_OPEN_BYTES     row bytes the open-pair pass read: per (row, query) pair
 *                          the first slab left at or before its bound, the further
 *                          1 KB slabs until its running sum passes the bound
 *   NR_WORK_REFINE_BYTES   row bytes the per-query kernel read: whole rows; for fp32
 *                          rows longer than 1024 bytes the 1 KB slabs it read before
 *                          the row's running sum passed the tile list's k-th key
 * ROWS_READ = OWN_ROWS + SHARED_ROWS + FALLBACK_ROWS and
 * ROWS = OWN_ROWS + SHARED_PAIR_ROWS. */
enum {
  NR_WORK_TILES = 0,
  NR_WORK_ROWS = 1,
  NR_WORK_ROWS_READ = 2,
  NR_WORK_OWN_ROWS = 3,
  NR_WORK_SHARED_ROWS = 4,
  NR_WORK_SHARED_PAIRS = 5,
  NR_WORK_SURVIVORS = 6,
  NR_WORK_FLAGGED = 7,
  NR_WORK_FALLBACK_ROWS = 8,
  NR_WORK_SHARED_PAIR_ROWS = 9,
  NR_WORK_FULL_ROWS = 10,
  NR_WORK_HEAD_BYTES = 11,
  NR_WORK_BODY_BYTES = 12,
  NR_WORK_OPEN_BYTES = 13,
  NR_WORK_REFINE_BYTES = 14,
  NR_WORK = 15
};
nr_status nr_last_work(nr_index *index, hipStream_t stream, int64_t *work, int32_t n_work);

/* Bandwidth self-check (not part of the search): one pass of 16-byte loads
 * over `bytes` (a multiple of 16) of the DEVICE buffer `buf`, on `stream`.
 * `sink` is a DEVICE uint32 that the kernel may write.  Timing it gives the
 * achievable streaming read rate of the device the index lives on. */
nr_status nr_stream_read(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t stream);

const char *nr_status_string(nr_status status);
const char *nr_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* NEUROUTE_H */
