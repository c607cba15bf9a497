/*
 * NeuRoute search oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-purpose CPU implementation of the batched query-time
 * search of NeuRoute (arXiv 2608.15438), used to check the GPU path and to
 * time a CPU baseline.  Only the test suite, the smoke check and the bench's
 * CPU-baseline leg may load it; the product library never does.  It shares no
 * code, header or table with the GPU path.
 *
 * Stages (paper section in brackets):
 *   or_encode     encoder forward pass               [Sec. 3.2.1, Sec. 4.5 "Architecture"]
 *   or_probes     bucket enumeration, Algorithm 1    [Sec. 3.4.1, Eq. 10, deviation scores]
 *   or_route      centroid stage, Algorithm 2        [Sec. 3.4.2]
 *   or_refine     exact refinement to top-k          [Sec. 3.4 intro, Sec. 3.5]
 *   or_search     all of the above, threaded over queries
 *   or_bruteforce exact k-NN over the whole base     [Sec. 3.1, Eq. 1-2]
 *
 * Readings where the paper is silent are listed in the repository design notes
 * and repeated at the functions that take them.
 */
#ifndef NEUROUTE_ORACLE_H
#define NEUROUTE_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OR_OK = 0, OR_EINVAL = 1, OR_ENOMEM = 2 };
enum { OR_U8 = 0, OR_F32 = 1 };

/* Encoder: n_layers linear layers; hidden layers are Linear -> (folded eval
 * BatchNorm affine) -> ReLU, the last layer is Linear and yields the logits.
 * params is one flat fp32 buffer, per layer l (in = widths[l], out = widths[l+1]):
 *   W[out*in] (row-major, out x in), bias[out], and for hidden layers also
 *   bn_scale[out], bn_shift[out].  Inputs are multiplied by input_scale. */
typedef struct {
  int32_t n_layers;
  const int32_t *widths;   /* [n_layers + 1] */
  const float *params;
  double input_scale;
  int32_t in_dtype;        /* OR_U8 or OR_F32 */
} or_encoder;

/* Alg. 2 knobs and the gate margin curve M(x). */
typedef struct {
  int32_t n_bins;          /* used when s_max is finite */
  float s_max;             /* +inf: every probe is its own bin */
  int32_t k_c, b_batch, b_min, t_low, u_heap, u_front;
  float alpha_front;
  int32_t gate_on, early_stop_on, lowq_or;
  int32_t m_knots;         /* 0: M == 0 */
  const float *m_x, *m_y;  /* knots, x strictly increasing, y non-decreasing */
} or_route_params;

typedef struct {            /* per query */
  int32_t n_probes, n_nonempty, n_singleton, n_scored, n_batches, bins_done, stopped, h_size, n_dir;
} or_route_stats;

int or_encode(const or_encoder *enc, const void *x, int64_t nq, float *logits, double *mag);

int or_probes(const float *logits, int64_t nq, int32_t b, const float *tau,
              int32_t l_sel, int32_t r_max, float s_max, int32_t n_bins, int32_t p_budget,
              uint32_t *codes, float *costs, int32_t *bins, int32_t *counts);

float or_margin(const or_route_params *prm, float x);

int or_route(const float *logits, int64_t nq, int32_t b,
             const uint32_t *codes, const int32_t *bins, const int32_t *counts, int32_t p_budget,
             const uint32_t *bc_off, const float *centroids, int64_t n_clusters,
             const or_route_params *prm, uint32_t *clus, int64_t cap, int32_t *n_clus,
             or_route_stats *stats);

int or_refine(const void *rows, int32_t d, int32_t dtype, const int64_t *row_ids,
              const uint64_t *cl_off, const void *queries, int64_t nq,
              const uint32_t *clus, int64_t cap, const int32_t *n_clus, int32_t k,
              int64_t *out_ids, float *out_dists, int64_t *n_cand);

int or_search(const or_encoder *enc, const float *tau, int32_t b,
              const void *rows, int32_t d, int32_t dtype, const int64_t *row_ids,
              const uint32_t *bc_off, const uint64_t *cl_off, const float *centroids,
              int64_t n_clusters, const void *queries, int64_t nq, int32_t k,
              int32_t l_sel, int32_t r_max, int32_t p_budget, const or_route_params *prm,
              int32_t n_threads, int64_t *out_ids, float *out_dists, int64_t *n_cand,
              double *stage_seconds /* [4]: encode, probes, route, refine (summed over threads) */);

int or_bruteforce(const void *rows, int64_t n, int32_t d, int32_t dtype, const int64_t *row_ids,
                  const void *queries, int64_t nq, int32_t k, int32_t n_threads,
                  int64_t *out_ids, float *out_dists);

#ifdef __cplusplus
}
#endif
#endif
