// Host side of the C ABI declared in include/neuroute.h: argument and index
// validation, device copies of the encoder, per-stream workspaces and the
// launch sequence of the five search steps.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "nr_internal.h"

namespace {

thread_local std::string g_err;

nr_status fail(nr_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIP_OK(call)                                                                      \
  do {                                                                                    \
    hipError_t e_ = (call);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return fail(NR_EDEVICE, "%s failed: %s", #call, hipGetErrorString(e_));           \
  } while (0)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Carves typed sub-buffers out of one device allocation.
struct Carver {
  char *base;
  size_t off = 0;
  template <class T>
  T *take(size_t count) {
    off = align_up(off, 256);
    T *p = reinterpret_cast<T *>(base ? base + off : nullptr);
    off += sizeof(T) * count;
    return p;
  }
};

struct Buffers {
  float *logits, *act0, *act1;
  uint32_t *codes;
  uint2 *lk;
  int32_t *redo;
  float *costs;
  int32_t *bins, *counts;
  uint32_t *clus;
  int32_t *nclus;
  uint32_t *rowpre, *rtot, *tsize;
  int32_t *ntile, *tile_off, *tile_q, *tile_c0, *counter;
  uint32_t *pkey;
  int64_t *pid;
  // shared refinement
  int64_t *own_ids;
  float *own_dists;
  uint32_t *clus_own;
  int32_t *nclus_own;
  int32_t *cseed;
  uint32_t *rfull, *own_rows;
  int32_t *scnt, *flag;
  unsigned long long *pool_cnt;
  uint32_t *pool_q, *pool_key, *poff, *pcur, *pool2_key;
  unsigned long long *open_cnt;
  uint32_t *open_q, *open_key;
  uint64_t *open_row;
  int64_t *pool_id, *pool2_id;
  unsigned long long *counter2;
  uint32_t *skey;
  int64_t *sid;
  uint32_t *pair_q, *hist, *pair_rank, *slist, *hpos, *lpair, *lpm;
  uint64_t *lbase;
  uint32_t *lsz;
  uint32_t *thr_n, *thr_h, *blk_n, *blk_h;
  uint64_t *thr_w, *blk_w, *lmeta;
  uint2 *qnorm;
  uint4 *qrec;
  uint64_t *swork_off;
  int64_t *wstats;
  bool shared;
  hipStream_t aux;   // from the workspace
  hipEvent_t fork, join;
};

struct Shape {
  int64_t nq;   // queries per chunk
  int P, b, k, maxw;
  int64_t cap;
  bool shared = false;
  int64_t n_clusters = 0;
};

Buffers carve(char *base, const Shape &s, size_t *bytes) {
  Carver c{base};
  Buffers B{};  // what is not carved (the second stream and its events) stays null
  B.logits = c.take<float>((size_t)s.nq * s.b);
  B.act0 = c.take<float>((size_t)s.nq * s.maxw);
  B.act1 = c.take<float>((size_t)s.nq * s.maxw);
  B.codes = c.take<uint32_t>((size_t)s.nq * s.P);
  B.costs = c.take<float>((size_t)s.nq * s.P);
  B.bins = c.take<int32_t>((size_t)s.nq * s.P);
  B.lk = c.take<uint2>((size_t)s.nq * s.P);
  B.redo = c.take<int32_t>((size_t)s.nq);
  B.counts = c.take<int32_t>((size_t)s.nq);
  B.clus = c.take<uint32_t>((size_t)s.nq * s.cap);
  B.nclus = c.take<int32_t>((size_t)s.nq);
  B.rowpre = c.take<uint32_t>((size_t)s.nq * (s.cap + 1));
  B.rtot = c.take<uint32_t>((size_t)s.nq);
  B.tsize = c.take<uint32_t>((size_t)s.nq);
  B.ntile = c.take<int32_t>((size_t)s.nq);
  B.tile_off = c.take<int32_t>((size_t)s.nq + 1);
  B.tile_q = c.take<int32_t>((size_t)s.nq * nr::MAX_TILES_PER_QUERY);
  B.tile_c0 = c.take<int32_t>((size_t)s.nq * nr::MAX_TILES_PER_QUERY);
  B.counter = c.take<int32_t>(1);
  B.pkey = c.take<uint32_t>((size_t)s.nq * nr::MAX_TILES_PER_QUERY * s.k);
  B.pid = c.take<int64_t>((size_t)s.nq * nr::MAX_TILES_PER_QUERY * s.k);
  B.shared = s.shared;
  B.rfull = c.take<uint32_t>((size_t)s.nq);
  B.wstats = c.take<int64_t>(7);
  if (s.shared) {
    const size_t nc1 = (size_t)s.n_clusters + 1;
    B.own_ids = c.take<int64_t>((size_t)s.nq * s.k);
    B.own_dists = c.take<float>((size_t)s.nq * s.k);
    B.clus_own = c.take<uint32_t>((size_t)s.nq * s.cap);
    B.nclus_own = c.take<int32_t>((size_t)s.nq);
    B.cseed = c.take<int32_t>((size_t)s.nq);
    B.own_rows = c.take<uint32_t>((size_t)s.nq);
    B.scnt = c.take<int32_t>((size_t)s.nq);
    B.flag = c.take<int32_t>((size_t)s.nq);
    B.counter2 = c.take<unsigned long long>(1);
    B.skey = c.take<uint32_t>((size_t)s.nq * nr::SURVIVOR_CAP);
    B.sid = c.take<int64_t>((size_t)s.nq * nr::SURVIVOR_CAP);
    B.pool_cnt = c.take<unsigned long long>(1);
    B.pool_q = c.take<uint32_t>(nr::SURVIVOR_POOL);
    B.pool_key = c.take<uint32_t>(nr::SURVIVOR_POOL);
    B.pool_id = c.take<int64_t>(nr::SURVIVOR_POOL);
    B.poff = c.take<uint32_t>((size_t)s.nq + 1);
    B.pcur = c.take<uint32_t>((size_t)s.nq);
    B.pool2_key = c.take<uint32_t>(nr::SURVIVOR_POOL);
    B.pool2_id = c.take<int64_t>(nr::SURVIVOR_POOL);
    B.open_cnt = c.take<unsigned long long>(1);
    B.open_q = c.take<uint32_t>(nr::OPEN_PAIRS);
    B.open_key = c.take<uint32_t>(nr::OPEN_PAIRS);
    B.open_row = c.take<uint64_t>(nr::OPEN_PAIRS);
    B.pair_q = c.take<uint32_t>((size_t)s.nq * s.cap);
    B.pair_rank = c.take<uint32_t>((size_t)s.nq * s.cap);
    B.qnorm = c.take<uint2>((size_t)s.nq);
    B.qrec = c.take<uint4>((size_t)s.nq);
    B.hist = c.take<uint32_t>((size_t)nr::hist_words(s.n_clusters));
    B.hpos = c.take<uint32_t>(nc1);
    B.slist = c.take<uint32_t>(nc1);
    B.lpair = c.take<uint32_t>(nc1);
    B.lpm = c.take<uint32_t>(nc1);
    B.lbase = c.take<uint64_t>(nc1);
    B.lsz = c.take<uint32_t>(nc1);
    B.swork_off = c.take<uint64_t>(nc1);
    B.lmeta = c.take<uint64_t>(4);
    const size_t nblk = (size_t)nr::list_blocks(s.n_clusters);
    B.thr_n = c.take<uint32_t>(nblk * nr::LIST_THREADS);
    B.thr_h = c.take<uint32_t>(nblk * nr::LIST_THREADS);
    B.thr_w = c.take<uint64_t>(nblk * nr::LIST_THREADS);
    B.blk_n = c.take<uint32_t>(nblk);
    B.blk_h = c.take<uint32_t>(nblk);
    B.blk_w = c.take<uint64_t>(nblk);
  }
  *bytes = align_up(c.off, 256);
  return B;
}

struct Workspace {
  hipStream_t stream = nullptr;
  char *base = nullptr;
  size_t bytes = 0;
  // the shared schedule's second stream (default priority) and its fork/join events
  hipStream_t aux = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  Buffers last{};
  int64_t last_nq = 0;
  int64_t last_cap = 0;
  // the shared schedule's pair counts are all zero at
  // this address of hist (each search's prep clears what it used); any other
  // carving of the workspace may overwrite them, so it resets this
  const uint32_t *clean_hist = nullptr;
};

struct EventSet {
  hipEvent_t ev[NR_STAGES + 1];
};

}  // namespace

// Working memory of nr_search_noalloc: one fixed array per GPU, part of the
// library's code object, held until the process ends.  Host code never uses
// the name itself (on the host it is only a stand-in for the symbol): the
// device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[NR_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char *g_scratch[MAX_DEVICES] = {};

// The address of `scratch` on the current device `dev`, looked up once per
// device (the library's index upload does it first).
nr_status scratch_address(int dev, char **out) {
  if (dev < 0 || dev >= MAX_DEVICES)
    return fail(NR_EUNSUPPORTED, "device ordinal %d outside [0, %d)", dev, MAX_DEVICES);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(NR_EDEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                  hipGetErrorString(e));
    g_scratch[dev] = static_cast<char *>(p);
  }
  *out = g_scratch[dev];
  return NR_OK;
}

}  // namespace

struct nr_index {
  nr_index_desc d;               // scalars and borrowed device pointers
  std::vector<int32_t> widths;
  float *params = nullptr;       // device copy of all layers
  std::vector<const float *> W, bias, bn_scale, bn_shift;
  float *tau = nullptr;
  uint32_t *row_of_id = nullptr;  // inverse permutation, made by the first calibration
  bool enc_only = false;          // encoder and tau only (index construction)
  int maxw = 0;
  int n_cu = 0;
  std::mutex mu;
  std::deque<Workspace> ws;     // stable addresses: callers keep Workspace pointers
  bool profiling = false;
  std::vector<EventSet> pending;
  double stage_ms[NR_STAGES] = {0};
  int64_t n_timed = 0;
};

namespace {

nr_status workspace_for(nr_index *ix, hipStream_t stream, const Shape &s, Buffers *out,
                        Workspace **wsp) {
  size_t need = 0;
  carve(nullptr, s, &need);
  std::lock_guard<std::mutex> g(ix->mu);
  Workspace *w = nullptr;
  for (auto &x : ix->ws)
    if (x.stream == stream) w = &x;
  if (!w) {
    ix->ws.emplace_back();
    w = &ix->ws.back();
    w->stream = stream;
  }
  if (w->bytes < need) {
    if (w->base) {
      HIP_OK(hipStreamSynchronize(stream));
      HIP_OK(hipFree(w->base));
      w->base = nullptr;
      w->bytes = 0;
    }
    size_t grow = need + need / 4;
    if (hipMalloc(&w->base, grow) != hipSuccess) {
      (void)hipGetLastError();
      w->base = nullptr;
      return fail(NR_ENOMEM, "workspace allocation of %zu bytes failed", grow);
    }
    w->bytes = grow;
    w->clean_hist = nullptr;
  }
  if (s.shared && !w->aux) {
    HIP_OK(hipStreamCreateWithFlags(&w->aux, hipStreamNonBlocking));
    HIP_OK(hipEventCreateWithFlags(&w->fork, hipEventDisableTiming));
    HIP_OK(hipEventCreateWithFlags(&w->join, hipEventDisableTiming));
  }
  size_t dummy;
  *out = carve(w->base, s, &dummy);
  if (!s.shared || out->hist != w->clean_hist) w->clean_hist = nullptr;
  out->aux = w->aux;
  out->fork = w->fork;
  out->join = w->join;
  *wsp = w;
  return NR_OK;
}

int64_t kc_eff(const nr_index *ix, const nr_params *p) {
  int64_t k = p->k_c;
  return k < ix->d.n_clusters ? k : ix->d.n_clusters;
}

nr_status check_params(const nr_index *ix, int32_t P, const nr_params *p) {
  if (!p) return fail(NR_EINVAL, "params is NULL");
  const int b = ix->d.b;
  if (P < 1) return fail(NR_EINVAL, "probe_budget must be >= 1 (got %d)", P);
  if (P > NR_MAX_PROBES) return fail(NR_EUNSUPPORTED, "probe_budget %d > %d", P, NR_MAX_PROBES);
  if (p->l_sel < 0 || p->l_sel > b || p->l_sel > 32)
    return fail(NR_EINVAL, "l_sel %d outside [0, min(b=%d, 32)]", p->l_sel, b);
  if (p->r_max < 0) return fail(NR_EINVAL, "r_max must be >= 0");
  if (std::isnan(p->s_max) || p->s_max < 0.f) return fail(NR_EINVAL, "s_max must be >= 0");
  if (std::isfinite(p->s_max) && (p->n_bins < 1 || p->s_max <= 0.f))
    return fail(NR_EINVAL, "finite s_max needs s_max > 0 and n_bins >= 1");
  if (p->k_c < 1) return fail(NR_EINVAL, "k_c must be >= 1");
  if (kc_eff(ix, p) > nr::MAX_KC)
    return fail(NR_EUNSUPPORTED, "k_c %d exceeds the LDS heap limit %d", p->k_c, nr::MAX_KC);
  if (p->b_batch < 1 || p->b_batch > 64) return fail(NR_EUNSUPPORTED, "b_batch must be in [1, 64]");
  if (p->m_knots < 0 || p->m_knots > NR_MAX_KNOTS)
    return fail(NR_EINVAL, "m_knots must be in [0, %d]", NR_MAX_KNOTS);
  for (int i = 0; i < p->m_knots; ++i) {
    if (!std::isfinite(p->m_x[i]) || !std::isfinite(p->m_y[i]))
      return fail(NR_EINVAL, "margin knot %d is not finite", i);
    if (i > 0 && !(p->m_x[i] > p->m_x[i - 1]))
      return fail(NR_EINVAL, "margin knots must have strictly increasing x");
    if (i > 0 && p->m_y[i] < p->m_y[i - 1])
      return fail(NR_EINVAL, "margin knots must have non-decreasing y");
  }
  if (!std::isfinite(p->alpha_front)) return fail(NR_EINVAL, "alpha_front must be finite");
  if (p->refine_mode < NR_REFINE_AUTO || p->refine_mode > NR_REFINE_SHARED)
    return fail(NR_EINVAL, "refine_mode must be 0, 1 or 2");
  if (p->shared_seed_rows < 0) return fail(NR_EINVAL, "shared_seed_rows must be >= 0");
  return NR_OK;
}

Shape shape_of(const nr_index *ix, int64_t nq, int P, int k, int64_t cap) {
  Shape s;
  s.nq = nq < nr::QUERY_CHUNK ? nq : nr::QUERY_CHUNK;
  s.P = P;
  s.b = ix->d.b;
  s.k = k;
  s.maxw = ix->maxw;
  s.cap = cap;
  return s;
}

size_t elem_size(const nr_index *ix) { return ix->d.dtype == NR_U8 ? 1 : 4; }

// bytes of each row the shared scan's filter reads: the head plane of the
// split layout, else the first 16 dimensions of the row-major row
int scan_head(const nr_index *ix) {
  if (ix->d.head_bytes > 0) return ix->d.head_bytes;
  const int rb = (int)(ix->d.d * (ix->d.dtype == NR_U8 ? 1 : 4));
  const int h = ix->d.dtype == NR_U8 ? 16 : 64;
  return h < rb ? h : rb;
}

// payload addressing for the kernels (row-major or head/tail planes)
nr::RowAddr row_addr(const nr_index *ix) {
  const uint64_t rb = (uint64_t)ix->d.d * elem_size(ix);
  const uint64_t H = ix->d.head_bytes > 0 ? (uint64_t)ix->d.head_bytes : 0;
  const unsigned char *base = (const unsigned char *)ix->d.rows;
  nr::RowAddr r;
  if (H > 0 && !ix->d.head_copy) {  // head plane, then tail plane
    r.h = (int)H;
    r.hb = base;
    r.hs = H;
    r.tb = base + (uint64_t)ix->d.n * H;
    r.ts = rb - H;
  } else {  // row-major rows (after the head plane when it is a copy)
    r.h = (int)rb;
    r.hb = base + (uint64_t)ix->d.n * H;
    r.hs = rb;
    r.tb = r.hb;  // unused: every offset is below h
    r.ts = rb;
  }
  return r;
}

// ----------------------------------------------------------------- stages
hipError_t run_encode(const nr_index *ix, const void *q, int64_t nq, float *logits,
                      const Buffers &B, hipStream_t s) {
  const int L = (int)ix->widths.size() - 1;
  const void *in = q;
  int in_u8 = ix->d.dtype == NR_U8;
  float *bufs[2] = {B.act0, B.act1};
  for (int l = 0; l < L; ++l) {
    nr::EncodeLayerArgs a{};
    a.in = in;
    a.in_u8 = in_u8;
    a.out = l + 1 == L ? logits : bufs[l & 1];
    a.W = ix->W[l];
    a.bias = ix->bias[l];
    a.bn_scale = l + 1 < L ? ix->bn_scale[l] : nullptr;
    a.bn_shift = l + 1 < L ? ix->bn_shift[l] : nullptr;
    a.in_scale = l == 0 ? ix->d.input_scale : 1.0f;
    a.relu = l + 1 < L;
    a.M = nq;
    a.K = ix->widths[l];
    a.N = ix->widths[l + 1];
    hipError_t e = nr::launch_encode_layer(a, s);
    if (e != hipSuccess) return e;
    in = a.out;
    in_u8 = 0;
  }
  return hipSuccess;
}

// with route (a search's buffers): the probe kernel also looks up each
// probe's bucket and assigns each query its route pass, for run_route(...,
// looked_up = true) on the same buffers
hipError_t run_probe(const nr_index *ix, const float *logits, int64_t nq, int P,
                     const nr_params *p, uint32_t *codes, float *costs, int32_t *bins,
                     int32_t *counts, hipStream_t s, const Buffers *route = nullptr) {
  nr::ProbeArgs a{};
  a.logits = logits;
  a.tau = ix->tau;
  a.nq = nq;
  a.b = ix->d.b;
  a.l_sel = p->l_sel;
  a.r_max = p->r_max;
  a.P = P;
  a.finite = std::isfinite(p->s_max) ? 1 : 0;
  a.s_max = p->s_max;
  a.n_bins = a.finite ? p->n_bins : 1;
  a.bin_scale = a.finite ? (float)p->n_bins / p->s_max : 0.0f;
  a.codes = codes;
  a.costs = costs;
  a.bins = bins;
  a.counts = counts;
  if (route) {
    a.bc_off = ix->d.bc_off;
    a.lk = route->lk;
    int tiers[3];
    a.tier_n = nr::route_tiers((int)kc_eff(ix, p), tiers);
    if (a.tier_n > 1) {
      a.tier = route->redo;
      a.tier_h0 = tiers[0];
      a.tier_h1 = a.tier_n > 2 ? tiers[1] : tiers[0];
    }
  }
  return nr::launch_probe(a, s);
}

// after run_probe(..., &B) on the same buffers (it writes B.lk and B.redo)
hipError_t run_route(const nr_index *ix, const float *logits, int64_t nq, int P,
                     const nr_params *p, const Buffers &B, uint32_t *clus, int32_t *nclus,
                     int64_t cap, int32_t *qstats, hipStream_t s,
                     const nr::PairHistArgs *ph = nullptr) {
  nr::RouteArgs a{};
  a.logits = logits;
  a.nq = nq;
  a.b = ix->d.b;
  a.P = P;
  a.bins = B.bins;
  a.counts = B.counts;
  a.lk = B.lk;
  a.redo = B.redo;
  a.centroids = ix->d.centroids;
  a.k_c = (int)kc_eff(ix, p);
  a.b_batch = p->b_batch;
  a.b_min = p->b_min;
  a.t_low = p->t_low;
  a.u_heap = p->u_heap;
  a.u_front = p->u_front;
  a.alpha_front = p->alpha_front;
  a.gate_on = p->gate_on != 0;
  a.early_stop_on = p->early_stop_on != 0;
  a.lowq_or = p->lowq_or != 0;
  a.finite = std::isfinite(p->s_max) ? 1 : 0;
  a.m_knots = p->m_knots;
  for (int i = 0; i < p->m_knots; ++i) {
    a.m_x[i] = p->m_x[i];
    a.m_y[i] = p->m_y[i];
    a.m_slope[i] = i + 1 < p->m_knots ? (p->m_y[i + 1] - p->m_y[i]) / (p->m_x[i + 1] - p->m_x[i])
                                      : 0.0f;
  }
  a.clus = clus;
  a.nclus = nclus;
  a.cap = cap;
  a.qstats = qstats;
  if (ph) {
    a.ph = *ph;
    a.ph_on = 1;
  }
  return nr::launch_route(a, s, B.aux, B.fork, B.join);
}

struct RefineOpts {
  const int32_t *qmask = nullptr;      // only these queries (the others keep their outputs)
  const int32_t *own_cseed = nullptr;  // seed pass of the shared schedule: leading clusters only
  // shared schedule: the scan's prep, started on the second stream once the
  // seed pass is planned (so that it does not slow the planning kernels)
  const nr::SharedArgs *prep = nullptr;
  hipStream_t aux = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};

// ev (may be null): events recorded after the plan, the refinement and the merge
hipError_t run_refine(const nr_index *ix, const void *q, int64_t nq, int k, const uint32_t *clus,
                      const int32_t *nclus, int64_t cap, const Buffers &B, int64_t *out_ids,
                      float *out_dists, int32_t *qstats, hipStream_t s, hipEvent_t *ev,
                      const RefineOpts &o = RefineOpts()) {
  nr::PlanArgs pa{};
  pa.nq = nq;
  pa.clus = clus;
  pa.nclus = nclus;
  pa.cap = cap;
  pa.cl_off = ix->d.cl_off;
  pa.n_clusters = ix->d.n_clusters;
  pa.rowpre = B.rowpre;
  pa.rtot = B.rtot;
  pa.tsize = B.tsize;
  pa.ntile = B.ntile;
  pa.tile_off = B.tile_off;
  pa.tile_q = B.tile_q;
  pa.tile_c0 = B.tile_c0;
  pa.counter = B.counter;
  pa.rfull = (o.qmask || o.own_cseed) ? nullptr : B.rfull;
  pa.qmask = o.qmask;
  pa.own_cseed = o.own_cseed;
  if (o.own_cseed) {
    pa.clus_out = B.clus_own;
    pa.nclus_out = B.nclus_own;
    pa.tile_min = nr::OWN_TILE_MIN_ROWS;
  }
  // the search's refine bytes count from its first refinement launch on (the
  // redo of queries whose survivors overflowed adds to them)
  hipError_t e = o.qmask ? hipSuccess : nr::launch_fill_i32((int32_t *)(B.wstats + 6), 2, 0, s);
  if (e == hipSuccess) e = nr::launch_plan(pa, s);
#ifdef NR_PREP_ON_MAIN
  if (e == hipSuccess && o.prep) {
    e = nr::launch_shared_prep(*o.prep, s);
    if (e == hipSuccess) e = hipEventRecord(o.join, s);
  }
#else
  if (e == hipSuccess && o.prep) {
    e = hipEventRecord(o.fork, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(o.aux, o.fork, 0);
    if (e == hipSuccess) e = nr::launch_shared_prep(*o.prep, o.aux);
    if (e == hipSuccess) e = hipEventRecord(o.join, o.aux);
  }
#endif
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[0], s);
  nr::RefineArgs ra{};
  ra.ra = row_addr(ix);
  ra.row_ids = ix->d.row_ids;
  ra.cl_off = ix->d.cl_off;
  ra.n_clusters = ix->d.n_clusters;
  ra.queries = q;
  ra.nq = nq;
  ra.d = ix->d.d;
  ra.row_bytes = (int)(ix->d.d * elem_size(ix));
  ra.k = k;
  ra.clus = o.own_cseed ? B.clus_own : clus;
  ra.nclus = o.own_cseed ? B.nclus_own : nclus;
  ra.cap = cap;
  ra.rowpre = B.rowpre;
  ra.rtot = B.rtot;
  ra.tsize = B.tsize;
  ra.tile_off = B.tile_off;
  ra.tile_q = B.tile_q;
  ra.tile_c0 = B.tile_c0;
  ra.counter = B.counter;
  ra.pkey = B.pkey;
  ra.pid = B.pid;
  ra.rbytes = (unsigned long long *)(B.wstats + 6);
  // beside the scan's preparation, four blocks per CU (four waves per SIMD)
  // leave its kernels room to run under the seed pass instead of after it
#ifndef NR_REFINE_BLOCKS_BESIDE_PREP
#define NR_REFINE_BLOCKS_BESIDE_PREP 4
#endif
  e = nr::launch_refine(ra, ix->d.dtype, ix->n_cu, o.prep ? NR_REFINE_BLOCKS_BESIDE_PREP : 0, s);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[1], s);
  nr::MergeArgs ma{};
  ma.nq = nq;
  ma.k = k;
  ma.is_u8 = ix->d.dtype == NR_U8;
  ma.tile_off = B.tile_off;
  ma.pkey = B.pkey;
  ma.pid = B.pid;
  ma.rtot = B.rtot;
  ma.out_ids = out_ids;
  ma.out_dists = out_dists;
  ma.qstats = qstats;
  ma.qmask = o.qmask;
  e = nr::launch_merge(ma, s);
  if (e == hipSuccess && ev) (void)hipEventRecord(ev[2], s);
  return e;
}

// Step 5 with the batch-shared schedule (k_shared.hip): pair counts, the own
// pass of every query, cluster-major work units, the shared scan, the merge,
// and the per-query schedule again for the queries whose survivors overflowed.
// ev (may be null): after the own plan, own refinement, own merge, shared
// prep, shared scan, shared merge.
nr::SharedArgs shared_args(const nr_index *ix, const nr_params *p, const void *q, int64_t nq,
                           int k, const uint32_t *clus, const int32_t *nclus, int64_t cap,
                           const Buffers &B, int64_t *out_ids, float *out_dists,
                           int32_t *qstats) {
  nr::SharedArgs a{};
  a.nq = nq;
  a.k = k;
  a.is_u8 = ix->d.dtype == NR_U8;
  a.row_bytes = (int)(ix->d.d * elem_size(ix));
  a.g = nr::SHARED_G;
  a.scan_head = scan_head(ix);
  a.scan_hb = (const unsigned char *)ix->d.rows;  // the head plane, or the rows themselves
  a.scan_hs = ix->d.head_bytes > 0 ? (uint64_t)ix->d.head_bytes : (uint64_t)a.row_bytes;
  const uint32_t seed = p->shared_seed_rows > 0 ? (uint32_t)p->shared_seed_rows
                        : (a.row_bytes > 1024 ? nr::SEED_ROWS_LONG : nr::SEED_ROWS);
  a.seed_min = seed > (uint32_t)k ? seed : (uint32_t)k;
  a.n_clusters = ix->d.n_clusters;
  a.ra = row_addr(ix);
  a.row_ids = ix->d.row_ids;
  a.cl_off = ix->d.cl_off;
  a.queries = q;
  a.clus = clus;
  a.nclus = nclus;
  a.cap = cap;
  a.cseed = B.cseed;
  a.rfull = B.rfull;
  a.rtot = B.rtot;
  a.tile_off = B.tile_off;
  a.own_ids = B.own_ids;
  a.own_dists = B.own_dists;
  a.own_rows = B.own_rows;
  a.hist = B.hist;
  a.hpos = B.hpos;
  a.pair_rank = B.pair_rank;
  a.slist = B.slist;
  a.lpair = B.lpair;
  a.lpm = B.lpm;
  a.lbase = B.lbase;
  a.lsz = B.lsz;
  a.lmeta = B.lmeta;
  a.thr_n = B.thr_n;
  a.thr_h = B.thr_h;
  a.thr_w = B.thr_w;
  a.blk_n = B.blk_n;
  a.blk_h = B.blk_h;
  a.blk_w = B.blk_w;
  // the per-query rows of the whole list are diagnostics: taken here only
  // when the caller asked for per-query statistics
  a.eager_rows = qstats != nullptr;
  a.swork_off = B.swork_off;
  a.pair_q = B.pair_q;
  a.qnorm = B.qnorm;
  a.qrec = B.qrec;
  a.scnt = B.scnt;
  a.skey = B.skey;
  a.sid = B.sid;
  a.flag = B.flag;
  a.pool_cnt = B.pool_cnt;
  a.pool_q = B.pool_q;
  a.pool_key = B.pool_key;
  a.pool_id = B.pool_id;
  a.poff = B.poff;
  a.pcur = B.pcur;
  a.pool2_key = B.pool2_key;
  a.pool2_id = B.pool2_id;
  a.open_cnt = B.open_cnt;
  a.open_q = B.open_q;
  a.open_key = B.open_key;
  a.open_row = B.open_row;
  a.counter = B.counter2;
  a.wstats = B.wstats;
  a.out_ids = out_ids;
  a.out_dists = out_dists;
  a.qstats = qstats;
  return a;
}

// The shared schedule after routing; the route kernel has counted the pairs
// (its pair_hist_wave epilogue, on counts zeroed before it ran).
hipError_t run_refine_shared(const nr_index *ix, const nr::SharedArgs &a, const void *q,
                             int64_t nq, int k, const uint32_t *clus, const int32_t *nclus,
                             int64_t cap, const Buffers &B, int64_t *out_ids, float *out_dists,
                             int32_t *qstats, hipStream_t s, hipEvent_t *ev) {
  // the scan's prep needs only the route's lists and pair counts: it runs on
  // the second stream while the seed pass runs here
  RefineOpts own;
  own.own_cseed = B.cseed;
  own.prep = &a;
  own.aux = B.aux;
  own.fork = B.fork;
  own.join = B.join;
  hipError_t e = run_refine(ix, q, nq, k, clus, nclus, cap, B, B.own_ids, B.own_dists, qstats,
                            s, ev, own);
  if (e != hipSuccess) return e;
  e = hipStreamWaitEvent(s, B.join, 0);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[3], s);  // the part of the prep the seed pass did not hide
  e = nr::launch_shared_refine(a, ix->d.dtype, ix->n_cu, s);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[4], s);
  if (e == hipSuccess) e = nr::launch_scan_open(a, ix->d.dtype, ix->n_cu, s);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[5], s);
  e = nr::launch_shared_merge(a, s);
  if (e != hipSuccess) return e;
  RefineOpts fb;
  fb.qmask = B.flag;
  e = run_refine(ix, q, nq, k, clus, nclus, cap, B, out_ids, out_dists, qstats, s, nullptr, fb);
  if (e == hipSuccess && ev) (void)hipEventRecord(ev[6], s);
  return e;
}

bool use_shared(const nr_index *ix, const nr_params *p, int64_t nq) {
  const int rb = (int)(ix->d.d * elem_size(ix));
  if ((rb + 127) / 128 > nr::SHARED_MAX_NSEG) return false;
  if (p->refine_mode == NR_REFINE_SHARED) return true;
  if (p->refine_mode == NR_REFINE_PER_QUERY) return false;
  return nq >= 512;
}

nr_status check_index(const nr_index *ix) {
  if (!ix) return fail(NR_EINVAL, "index is NULL");
  return NR_OK;
}

// device buffers of one call, freed when it ends
struct DevScratch {
  std::vector<void *> ptrs;
  ~DevScratch() {
    for (void *p : ptrs) (void)hipFree(p);
  }
  template <class T>
  T *get(size_t count) {
    void *p = nullptr;
    if (hipMalloc(&p, sizeof(T) * (count > 0 ? count : 1)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    ptrs.push_back(p);
    return static_cast<T *>(p);
  }
};

// entry points that read the payload or the directory
nr_status check_search_index(const nr_index *ix) {
  if (!ix) return fail(NR_EINVAL, "index is NULL");
  if (ix->enc_only) return fail(NR_EINVAL, "the index holds only an encoder (n = 0)");
  return NR_OK;
}

nr_status make_events(nr_index *ix, EventSet *es) {
  for (int i = 0; i <= NR_STAGES; ++i) HIP_OK(hipEventCreate(&es->ev[i]));
  return NR_OK;
}

}  // namespace

extern "C" {

const char *nr_status_string(nr_status s) {
  switch (s) {
    case NR_OK: return "ok";
    case NR_EINVAL: return "invalid argument";
    case NR_ENOMEM: return "out of memory";
    case NR_EDEVICE: return "device error";
    case NR_EUNSUPPORTED: return "unsupported";
    case NR_ECORRUPT: return "corrupt index";
  }
  return "unknown status";
}

const char *nr_last_error(void) { return g_err.c_str(); }

nr_status nr_stream_read(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t stream) {
  if (!buf || !sink || bytes < 0 || bytes % 16 != 0)
    return fail(NR_EINVAL, "buf and sink must be set and bytes a multiple of 16");
  int dev = 0, n_cu = 0;
  HIP_OK(hipGetDevice(&dev));
  HIP_OK(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
  HIP_OK(nr::launch_stream_read(buf, bytes, sink, n_cu, stream));
  return NR_OK;
}

nr_status nr_index_upload(const nr_index_desc *desc, nr_index **out, hipStream_t stream) {
  if (!desc || !out) return fail(NR_EINVAL, "desc and out must not be NULL");
  *out = nullptr;
  const nr_index_desc &d = *desc;
  // encoder and tau only: no payload, nothing borrowed
  const bool enc_only = d.n == 0 && !d.rows && !d.row_ids && !d.bc_off && !d.cl_off &&
                        !d.centroids;
  if (d.n < 1 && !enc_only) return fail(NR_EINVAL, "n must be >= 1");
  if (d.n >= (int64_t)1 << 32) return fail(NR_EUNSUPPORTED, "n must be < 2^32");
  if (d.d < 1) return fail(NR_EINVAL, "d must be >= 1");
  if (d.dtype != NR_U8 && d.dtype != NR_F32) return fail(NR_EINVAL, "dtype must be NR_U8 or NR_F32");
  const size_t rb = (size_t)d.d * (d.dtype == NR_U8 ? 1 : 4);
  if (rb % 16 != 0) return fail(NR_EUNSUPPORTED, "row size %zu bytes is not a multiple of 16", rb);
  if (rb > 48 * 128) return fail(NR_EUNSUPPORTED, "row size %zu bytes exceeds 6144", rb);
  if (d.b < 1 || d.b > 30) return fail(NR_EUNSUPPORTED, "b must be in [1, 30] (got %d)", d.b);
  if (d.n_layers < 1 || d.n_layers > NR_MAX_LAYERS)
    return fail(NR_EUNSUPPORTED, "n_layers must be in [1, %d]", NR_MAX_LAYERS);
  if (!d.widths || !d.weights || !d.tau) return fail(NR_EINVAL, "widths, weights and tau are required");
  if (d.widths[0] != d.d || d.widths[d.n_layers] != d.b)
    return fail(NR_EINVAL, "widths[0] must equal d and widths[n_layers] must equal b");
  for (int l = 0; l <= d.n_layers; ++l)
    if (d.widths[l] < 1 || d.widths[l] > 4096)
      return fail(NR_EUNSUPPORTED, "encoder width %d outside [1, 4096]", d.widths[l]);
  for (int l = 0; l < d.n_layers; ++l)
    if (!d.weights[l]) return fail(NR_EINVAL, "weights[%d] is NULL", l);
  if (!std::isfinite(d.input_scale)) return fail(NR_EINVAL, "input_scale must be finite");
  if (!enc_only && (!d.rows || !d.row_ids || !d.bc_off || !d.cl_off || !d.centroids))
    return fail(NR_EINVAL, "rows, row_ids, bc_off, cl_off and centroids are required");
  if ((uintptr_t)d.rows % 16 != 0) return fail(NR_EINVAL, "rows must be 16-byte aligned");
  if (d.head_bytes != 0 &&
      ((d.head_bytes != 16 && d.head_bytes != 32 && d.head_bytes != 64 && d.head_bytes != 128) ||
       (size_t)d.head_bytes > (d.head_copy ? rb : rb - 16)))
    return fail(NR_EINVAL, "head_bytes must be 0, 16, 32, 64 or 128, at most the row size "
                           "(row size - 16 without head_copy)");
  if (d.head_copy != 0 && d.head_copy != 1) return fail(NR_EINVAL, "head_copy must be 0 or 1");
  if (!enc_only && (d.n_clusters < 1 || d.n_clusters >= ((int64_t)1 << 32)))
    return fail(NR_EINVAL, "n_clusters must be in [1, 2^32)");

  nr_index *ix = new (std::nothrow) nr_index();
  if (!ix) return fail(NR_ENOMEM, "host allocation failed");
  ix->d = d;
  ix->widths.assign(d.widths, d.widths + d.n_layers + 1);
  // encoder parameters: one device buffer, per layer W, bias, scale, shift
  size_t total = 0;
  std::vector<size_t> offW, offB, offS, offH;
  for (int l = 0; l < d.n_layers; ++l) {
    size_t in = d.widths[l], o = d.widths[l + 1];
    offW.push_back(total); total += in * o;
    offB.push_back(total); total += o;
    offS.push_back(total); total += o;
    offH.push_back(total); total += o;
    ix->maxw = std::max(ix->maxw, (int)o);
  }
  std::vector<float> host(total, 0.0f);
  for (int l = 0; l < d.n_layers; ++l) {
    size_t in = d.widths[l], o = d.widths[l + 1];
    std::memcpy(&host[offW[l]], d.weights[l], sizeof(float) * in * o);
    if (d.biases && d.biases[l]) std::memcpy(&host[offB[l]], d.biases[l], sizeof(float) * o);
    for (size_t i = 0; i < o; ++i) {
      host[offS[l] + i] = (d.bn_scale && d.bn_scale[l]) ? d.bn_scale[l][i] : 1.0f;
      host[offH[l] + i] = (d.bn_shift && d.bn_shift[l]) ? d.bn_shift[l][i] : 0.0f;
    }
  }
  auto cleanup = [&](nr_status s) {
    if (ix->params) (void)hipFree(ix->params);
    if (ix->tau) (void)hipFree(ix->tau);
    delete ix;
    return s;
  };
  if (hipMalloc(&ix->params, sizeof(float) * total) != hipSuccess ||
      hipMalloc(&ix->tau, sizeof(float) * d.b) != hipSuccess) {
    (void)hipGetLastError();
    return cleanup(fail(NR_ENOMEM, "device allocation of the encoder failed"));
  }
  if (hipMemcpy(ix->params, host.data(), sizeof(float) * total, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(ix->tau, d.tau, sizeof(float) * d.b, hipMemcpyHostToDevice) != hipSuccess)
    return cleanup(fail(NR_EDEVICE, "copy of the encoder to the device failed"));
  for (int l = 0; l < d.n_layers; ++l) {
    ix->W.push_back(ix->params + offW[l]);
    ix->bias.push_back(ix->params + offB[l]);
    ix->bn_scale.push_back(ix->params + offS[l]);
    ix->bn_shift.push_back(ix->params + offH[l]);
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ix->n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return cleanup(fail(NR_EDEVICE, "device query failed"));
  {  // the no-alloc entry point's array on this device
    char *sp = nullptr;
    if (nr_status st = scratch_address(dev, &sp)) return cleanup(st);
  }
  if (enc_only) {
    ix->enc_only = true;
    *out = ix;
    return NR_OK;
  }
  // validate the borrowed CSR arrays and the permutation
  uint32_t *bitmap = nullptr;
  int32_t *flags = nullptr;
  const size_t words = (size_t)((d.n + 31) / 32);
  if (hipMalloc(&bitmap, words * 4) != hipSuccess || hipMalloc(&flags, 4) != hipSuccess) {
    (void)hipGetLastError();
    if (bitmap) (void)hipFree(bitmap);
    return cleanup(fail(NR_ENOMEM, "validation buffers could not be allocated"));
  }
  int32_t hflags = 0;
  hipError_t e = hipMemsetAsync(bitmap, 0, words * 4, stream);
  if (e == hipSuccess) e = hipMemsetAsync(flags, 0, 4, stream);
  if (e == hipSuccess)
    e = nr::launch_validate(d.bc_off, (int64_t)1 << d.b, d.cl_off, d.n_clusters, d.row_ids, d.n,
                            bitmap, flags, stream);
  if (e == hipSuccess) e = hipMemcpyAsync(&hflags, flags, 4, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  (void)hipFree(bitmap);
  (void)hipFree(flags);
  if (e != hipSuccess) return cleanup(fail(NR_EDEVICE, "index validation failed: %s", hipGetErrorString(e)));
  if (hflags) {
    std::string what;
    if (hflags & 1) what += " bucket directory (bc_off)";
    if (hflags & 2) what += " cluster offsets (cl_off)";
    if (hflags & 4) what += " row_ids (not a permutation of 0..n-1)";
    return cleanup(fail(NR_ECORRUPT, "index arrays fail validation:%s", what.c_str()));
  }
  *out = ix;
  return NR_OK;
}

nr_status nr_index_free(nr_index *ix) {
  if (!ix) return NR_OK;
  (void)hipDeviceSynchronize();
  for (auto &w : ix->ws) {
    if (w.base) (void)hipFree(w.base);
    if (w.fork) (void)hipEventDestroy(w.fork);
    if (w.join) (void)hipEventDestroy(w.join);
    if (w.aux) (void)hipStreamDestroy(w.aux);
  }
  for (auto &es : ix->pending)
    for (auto &ev : es.ev) (void)hipEventDestroy(ev);
  if (ix->params) (void)hipFree(ix->params);
  if (ix->tau) (void)hipFree(ix->tau);
  if (ix->row_of_id) (void)hipFree(ix->row_of_id);
  delete ix;
  return NR_OK;
}

int64_t nr_route_capacity(const nr_index *ix, int32_t P, const nr_params *p) {
  if (!ix || !p) return 0;
  return (int64_t)P + kc_eff(ix, p);
}

nr_status nr_encode(const nr_index *cix, const void *queries, int64_t nq, float *logits,
                    hipStream_t stream) {
  nr_index *ix = const_cast<nr_index *>(cix);
  if (nr_status s = check_index(ix)) return s;
  if (nq < 0) return fail(NR_EINVAL, "nq must be >= 0");
  if (nq == 0) return NR_OK;
  if (!queries || !logits) return fail(NR_EINVAL, "queries and logits must not be NULL");
  Buffers B;
  Workspace *w;
  Shape sh = shape_of(ix, nq, 1, 1, 1);
  if (nr_status s = workspace_for(ix, stream, sh, &B, &w)) return s;
  for (int64_t q0 = 0; q0 < nq; q0 += sh.nq) {
    int64_t n = nq - q0 < sh.nq ? nq - q0 : sh.nq;
    HIP_OK(run_encode(ix, (const char *)queries + q0 * ix->d.d * elem_size(ix), n,
                      logits + q0 * ix->d.b, B, stream));
  }
  return NR_OK;
}

nr_status nr_probe(const nr_index *cix, const float *logits, int64_t nq, int32_t P,
                   const nr_params *p, uint32_t *codes, float *costs, int32_t *bins,
                   int32_t *counts, hipStream_t stream) {
  if (nr_status s = check_search_index(cix)) return s;
  if (nr_status s = check_params(cix, P, p)) return s;
  if (nq < 0) return fail(NR_EINVAL, "nq must be >= 0");
  if (nq == 0) return NR_OK;
  if (!logits || !codes || !costs || !bins || !counts) return fail(NR_EINVAL, "NULL buffer");
  HIP_OK(run_probe(cix, logits, nq, P, p, codes, costs, bins, counts, stream));
  return NR_OK;
}

nr_status nr_route(const nr_index *cix, const float *logits, int64_t nq, int32_t P,
                   const nr_params *p, uint32_t *clusters, int32_t *n_clusters, int64_t cap,
                   hipStream_t stream) {
  nr_index *ix = const_cast<nr_index *>(cix);
  if (nr_status s = check_search_index(ix)) return s;
  if (nr_status s = check_params(ix, P, p)) return s;
  if (nq < 0) return fail(NR_EINVAL, "nq must be >= 0");
  if (nq == 0) return NR_OK;
  if (!logits || !clusters || !n_clusters) return fail(NR_EINVAL, "NULL buffer");
  if (cap < nr_route_capacity(ix, P, p))
    return fail(NR_EINVAL, "cap %lld < required %lld", (long long)cap,
                (long long)nr_route_capacity(ix, P, p));
  Buffers B;
  Workspace *w;
  Shape sh = shape_of(ix, nq, P, 1, 1);
  if (nr_status s = workspace_for(ix, stream, sh, &B, &w)) return s;
  for (int64_t q0 = 0; q0 < nq; q0 += sh.nq) {
    int64_t n = nq - q0 < sh.nq ? nq - q0 : sh.nq;
    const float *lg = logits + q0 * ix->d.b;
    HIP_OK(run_probe(ix, lg, n, P, p, B.codes, B.costs, B.bins, B.counts, stream, &B));
    HIP_OK(run_route(ix, lg, n, P, p, B, clusters + q0 * cap, n_clusters + q0, cap, nullptr,
                     stream));
  }
  return NR_OK;
}

nr_status nr_refine(const nr_index *cix, const void *queries, int64_t nq, int32_t k,
                    const uint32_t *clusters, const int32_t *n_clusters, int64_t cap,
                    int64_t *out_ids, float *out_dists, hipStream_t stream) {
  nr_index *ix = const_cast<nr_index *>(cix);
  if (nr_status s = check_search_index(ix)) return s;
  if (k < 1) return fail(NR_EINVAL, "k must be >= 1");
  if (k > NR_MAX_K) return fail(NR_EUNSUPPORTED, "k %d > %d", k, NR_MAX_K);
  if (nq < 0 || cap < 1) return fail(NR_EINVAL, "nq must be >= 0 and cap >= 1");
  if (nq == 0) return NR_OK;
  if (!queries || !clusters || !n_clusters || !out_ids || !out_dists)
    return fail(NR_EINVAL, "NULL buffer");
  Buffers B;
  Workspace *w;
  Shape sh = shape_of(ix, nq, 1, k, cap);
  if (nr_status s = workspace_for(ix, stream, sh, &B, &w)) return s;
  for (int64_t q0 = 0; q0 < nq; q0 += sh.nq) {
    int64_t n = nq - q0 < sh.nq ? nq - q0 : sh.nq;
    HIP_OK(run_refine(ix, (const char *)queries + q0 * ix->d.d * elem_size(ix), n, k,
                      clusters + q0 * cap, n_clusters + q0, cap, B, out_ids + q0 * k,
                      out_dists + q0 * k, nullptr, stream, nullptr));
  }
  w->last = B;
  w->last_nq = nq - (nq - 1) / sh.nq * sh.nq;
  w->last_cap = cap;
  return NR_OK;
}

nr_status nr_search_ex(const nr_index *cix, const void *queries, const float *logits,
                       int64_t nq, int32_t k, int32_t P, const nr_params *p, int64_t *out_ids,
                       float *out_dists, int32_t *qstats, hipStream_t stream) {
  nr_index *ix = const_cast<nr_index *>(cix);
  if (nr_status s = check_search_index(ix)) return s;
  if (nr_status s = check_params(ix, P, p)) return s;
  if (k < 1) return fail(NR_EINVAL, "k must be >= 1");
  if (k > NR_MAX_K) return fail(NR_EUNSUPPORTED, "k %d > %d", k, NR_MAX_K);
  if (nq < 0) return fail(NR_EINVAL, "nq must be >= 0");
  if (nq == 0) return NR_OK;
  if (!queries || !out_ids || !out_dists) return fail(NR_EINVAL, "NULL buffer");
  const int64_t cap = nr_route_capacity(ix, P, p);
  Buffers B;
  Workspace *w;
  Shape sh = shape_of(ix, nq, P, k, cap);
  sh.shared = use_shared(ix, p, sh.nq);
  sh.n_clusters = ix->d.n_clusters;
  if (nr_status s = workspace_for(ix, stream, sh, &B, &w)) return s;
  const size_t qrow = ix->d.d * elem_size(ix);
  for (int64_t q0 = 0; q0 < nq; q0 += sh.nq) {
    int64_t n = nq - q0 < sh.nq ? nq - q0 : sh.nq;
    const void *qp = (const char *)queries + q0 * qrow;
    int32_t *qs = qstats ? qstats + q0 * NR_QSTATS : nullptr;
    EventSet es{};
    bool prof = ix->profiling;
    if (prof) {
      if (nr_status s = make_events(ix, &es)) return s;
      HIP_OK(hipEventRecord(es.ev[0], stream));
    }
    const float *lg = logits ? logits + q0 * ix->d.b : B.logits;
    if (!logits) HIP_OK(run_encode(ix, qp, n, B.logits, B, stream));
    if (prof) HIP_OK(hipEventRecord(es.ev[1], stream));
    HIP_OK(run_probe(ix, lg, n, P, p, B.codes, B.costs, B.bins, B.counts, stream, &B));
    if (prof) HIP_OK(hipEventRecord(es.ev[2], stream));
    nr::SharedArgs sa{};
    nr::PairHistArgs ph{};
    if (B.shared) {
      sa = shared_args(ix, p, qp, n, k, B.clus, B.nclus, cap, B, out_ids + q0 * k,
                       out_dists + q0 * k, qs);
      ph = nr::pair_hist_args(sa);
      // pair counts start at zero: cleared in full only for a new
      // workspace (or after a search that stopped early), else by the last prep
      HIP_OK(nr::launch_shared_hist(sa, w->clean_hist != B.hist, stream));
      w->clean_hist = nullptr;
    }
    HIP_OK(run_route(ix, lg, n, P, p, B, B.clus, B.nclus, cap, qs, stream,
                     B.shared ? &ph : nullptr));
    if (prof) HIP_OK(hipEventRecord(es.ev[3], stream));
    if (B.shared) {
      HIP_OK(run_refine_shared(ix, sa, qp, n, k, B.clus, B.nclus, cap, B, out_ids + q0 * k,
                               out_dists + q0 * k, qs, stream, prof ? &es.ev[4] : nullptr));
      w->clean_hist = B.hist;
    } else {
      HIP_OK(run_refine(ix, qp, n, k, B.clus, B.nclus, cap, B, out_ids + q0 * k,
                        out_dists + q0 * k, qs, stream, prof ? &es.ev[4] : nullptr));
      if (prof)
        for (int i = 7; i <= NR_STAGES; ++i) HIP_OK(hipEventRecord(es.ev[i], stream));
    }
    if (prof) {
      std::lock_guard<std::mutex> g(ix->mu);
      ix->pending.push_back(es);
    }
  }
  w->last = B;
  w->last_nq = nq - (nq - 1) / sh.nq * sh.nq;
  w->last_cap = cap;
  return NR_OK;
}

nr_status nr_search_noalloc(const nr_index *cix, const void *queries, const float *logits,
                            int64_t nq, int32_t k, int32_t P, const nr_params *p,
                            int64_t *out_ids, float *out_dists, hipStream_t stream) {
  const nr_index *ix = cix;
  if (nr_status s = check_search_index(ix)) return s;
  if (nr_status s = check_params(ix, P, p)) return s;
  if (k < 1) return fail(NR_EINVAL, "k must be >= 1");
  if (k > NR_MAX_K) return fail(NR_EUNSUPPORTED, "k %d > %d", k, NR_MAX_K);
  if (nq < 0) return fail(NR_EINVAL, "nq must be >= 0");
  if (nq == 0) return NR_OK;
  if (!queries || !out_ids || !out_dists) return fail(NR_EINVAL, "NULL buffer");
  int dev = 0;
  HIP_OK(hipGetDevice(&dev));
  char *base = nullptr;
  if (nr_status s = scratch_address(dev, &base)) return s;
  const int64_t cap = nr_route_capacity(ix, P, p);
  // the largest chunk of queries whose buffers fit in the array (the carved
  // size grows by a fixed amount per query, up to 256-byte alignment per buffer)
  auto need = [&](int64_t nqc) {
    Shape sh = shape_of(ix, nqc, P, k, cap);
    sh.nq = nqc;
    size_t bytes = 0;
    carve(nullptr, sh, &bytes);
    return bytes;
  };
  const size_t limit = NR_NOALLOC_SCRATCH_BYTES;
  if (need(1) > limit)
    return fail(NR_EUNSUPPORTED, "one query needs %zu bytes of working memory, more than the "
                                 "%zu-byte no-alloc array", need(1), limit);
  const size_t per = need(2) - need(1);
  int64_t chunk = per ? (int64_t)((limit - need(1)) / per) + 1 : nr::QUERY_CHUNK;
  if (chunk > nr::QUERY_CHUNK) chunk = nr::QUERY_CHUNK;
  if (chunk > nq) chunk = nq;
  while (chunk > 1 && need(chunk) > limit) --chunk;
  Shape sh = shape_of(ix, chunk, P, k, cap);
  sh.nq = chunk;
  size_t used = 0;
  Buffers B = carve(base, sh, &used);
  const size_t qrow = ix->d.d * elem_size(ix);
  for (int64_t q0 = 0; q0 < nq; q0 += chunk) {
    const int64_t n = nq - q0 < chunk ? nq - q0 : chunk;
    const void *qp = (const char *)queries + q0 * qrow;
    const float *lg = logits ? logits + q0 * ix->d.b : B.logits;
    if (!logits) HIP_OK(run_encode(ix, qp, n, B.logits, B, stream));
    HIP_OK(run_probe(ix, lg, n, P, p, B.codes, B.costs, B.bins, B.counts, stream, &B));
    HIP_OK(run_route(ix, lg, n, P, p, B, B.clus, B.nclus, cap, nullptr, stream));
    HIP_OK(run_refine(ix, qp, n, k, B.clus, B.nclus, cap, B, out_ids + q0 * k,
                      out_dists + q0 * k, nullptr, stream, nullptr));
  }
  return NR_OK;
}

nr_status nr_search(const nr_index *ix, const void *queries, int64_t nq, int32_t k, int32_t P,
                    const nr_params *p, int64_t *out_ids, float *out_dists, hipStream_t stream) {
  return nr_search_ex(ix, queries, nullptr, nq, k, P, p, out_ids, out_dists, nullptr, stream);
}

nr_status nr_calibrate(const nr_index *cix, const float *logits, int64_t nq,
                       const int64_t *target_ids, int32_t K, int32_t l_sel, int32_t r_max,
                       float *scores, float *margin_xy, hipStream_t stream) {
  nr_index *ix = const_cast<nr_index *>(cix);
  if (nr_status s = check_search_index(ix)) return s;
  if (nq < 0) return fail(NR_EINVAL, "nq must be >= 0");
  if (K < 1 || K > NR_MAX_K) return fail(NR_EUNSUPPORTED, "K must be in [1, %d]", NR_MAX_K);
  if (l_sel < 0 || l_sel > ix->d.b || l_sel > 32)
    return fail(NR_EINVAL, "l_sel %d outside [0, min(b=%d, 32)]", l_sel, ix->d.b);
  if (r_max < 0) return fail(NR_EINVAL, "r_max must be >= 0");
  if (nq == 0) return NR_OK;
  if (!logits || !target_ids || !scores || !margin_xy) return fail(NR_EINVAL, "NULL buffer");
  {
    std::lock_guard<std::mutex> g(ix->mu);
    if (!ix->row_of_id) {
      if (hipMalloc(&ix->row_of_id, sizeof(uint32_t) * (size_t)ix->d.n) != hipSuccess) {
        (void)hipGetLastError();
        ix->row_of_id = nullptr;
        return fail(NR_ENOMEM, "inverse permutation (%lld rows) could not be allocated",
                    (long long)ix->d.n);
      }
      HIP_OK(nr::launch_inverse_perm(ix->d.row_ids, ix->d.n, ix->row_of_id, stream));
    }
  }
  nr::CalibArgs a{};
  a.logits = logits;
  a.tau = ix->tau;
  a.nq = nq;
  a.n = ix->d.n;
  a.b = ix->d.b;
  a.l_sel = l_sel;
  a.r_max = r_max;
  a.K = K;
  a.targets = target_ids;
  a.row_of_id = ix->row_of_id;
  a.cl_off = ix->d.cl_off;
  a.n_clusters = ix->d.n_clusters;
  a.n_codes = (int64_t)1 << ix->d.b;
  a.bc_off = ix->d.bc_off;
  a.centroids = ix->d.centroids;
  a.scores = scores;
  a.xy = margin_xy;
  HIP_OK(nr::launch_calib(a, stream));
  return NR_OK;
}

size_t nr_pair_sqdist_ws(int64_t B, int32_t D) {
  return B > 0 && D > 0 ? nr::pair_sqdist_ws_floats(B, D) : 0;
}

nr_status nr_pair_sqdist(const float *x, int64_t B, int32_t D, float *ws, float *out,
                         hipStream_t stream) {
  if (B < 0 || D < 1) return fail(NR_EINVAL, "B must be >= 0 and D >= 1");
  if (B > 65536) return fail(NR_EUNSUPPORTED, "B %lld > 65536", (long long)B);
  if (B == 0) return NR_OK;
  if (!x || !ws || !out) return fail(NR_EINVAL, "NULL buffer");
  HIP_OK(nr::launch_pair_sqdist(x, B, D, ws, out, stream));
  return NR_OK;
}

nr_status nr_lsim_grad(const float *d2_emb, const float *lat, int64_t B, int32_t L,
                       float gamma_rho, float tau_emb, double *num_cnt, float *grad_lat,
                       hipStream_t stream) {
  if (B < 0 || L < 1) return fail(NR_EINVAL, "B must be >= 0 and L >= 1");
  if (L > 32) return fail(NR_EUNSUPPORTED, "L %d > 32", L);
  if (B > 65536) return fail(NR_EUNSUPPORTED, "B %lld > 65536", (long long)B);
  if (!std::isfinite(gamma_rho) || !std::isfinite(tau_emb))
    return fail(NR_EINVAL, "gamma_rho and tau_emb must be finite");
  if (!d2_emb || !lat || !num_cnt || !grad_lat) return fail(NR_EINVAL, "NULL buffer");
  HIP_OK(nr::launch_lsim_grad(d2_emb, lat, B, L, gamma_rho, tau_emb, num_cnt, grad_lat, stream));
  return NR_OK;
}

nr_status nr_build_tau(const float *logits, int64_t ns, int32_t b, float *tau, hipStream_t stream) {
  if (ns < 1 || b < 1 || b > 30) return fail(NR_EINVAL, "ns must be >= 1 and b in [1, 30]");
  if (!logits || !tau) return fail(NR_EINVAL, "NULL buffer");
  HIP_OK(nr::launch_build_tau(logits, ns, b, tau, stream));
  return NR_OK;
}

nr_status nr_build_codes(const float *logits, int64_t m, int32_t b, const float *tau,
                         uint32_t *codes, uint32_t *sizes, hipStream_t stream) {
  if (m < 0 || b < 1 || b > 30) return fail(NR_EINVAL, "m must be >= 0 and b in [1, 30]");
  if (m == 0) return NR_OK;
  if (!logits || !tau || !codes || !sizes) return fail(NR_EINVAL, "NULL buffer");
  HIP_OK(nr::launch_build_codes(logits, m, b, tau, codes, sizes, stream));
  return NR_OK;
}

nr_status nr_build_plan(const uint32_t *sizes, int64_t n, int32_t b, int32_t rule, uint32_t param,
                        uint32_t *kb, uint32_t *mlist, nr_build_plan_info *info,
                        hipStream_t stream) {
  if (n < 1 || n >= ((int64_t)1 << 32)) return fail(NR_EINVAL, "n must be in [1, 2^32)");
  if (b < 1 || b > 30) return fail(NR_EINVAL, "b must be in [1, 30]");
  if (!sizes || !kb || !mlist || !info) return fail(NR_EINVAL, "NULL buffer");
  if (rule < NR_CLUSTER_NONE || rule > NR_CLUSTER_PER_BUCKET)
    return fail(NR_EINVAL, "unknown cluster rule %d", rule);
  if (rule != NR_CLUSTER_NONE && param < 1) return fail(NR_EINVAL, "param must be >= 1");
  const int64_t nb = (int64_t)1 << b;
  DevScratch ds;
  uint32_t *multi = ds.get<uint32_t>(nb + 1), *mpos = ds.get<uint32_t>(nb + 1);
  unsigned long long *cnt = ds.get<unsigned long long>(4);
  uint64_t *blk = ds.get<uint64_t>(nr::build_scan_blocks(nb));
  if (!multi || !mpos || !cnt || !blk) return fail(NR_ENOMEM, "plan scratch allocation failed");
  HIP_OK(nr::launch_fill_i32((int32_t *)cnt, 8, 0, stream));
  uint32_t t = param;
  int r = rule;
  if (rule == NR_CLUSTER_PER_BUCKET) {
    HIP_OK(nr::launch_build_nonempty(sizes, nb, cnt + 3, stream));
    unsigned long long ne = 0;
    HIP_OK(hipMemcpyAsync(&ne, cnt + 3, 8, hipMemcpyDeviceToHost, stream));
    HIP_OK(hipStreamSynchronize(stream));
    const double mean = ne ? (double)n / (double)ne : 0.0;
    const double tt = std::nearbyint(mean / (double)param);  // half to even
    t = tt < 1.0 ? 1u : (uint32_t)tt;
    r = NR_CLUSTER_CAPACITY;
  }
  nr::BuildArgs a{};
  a.b = b;
  a.sizes = sizes;
  a.rule = r;
  a.t = t;
  a.kb = kb;
  a.multi = multi;
  a.mpos = mpos;
  a.mlist = mlist;
  a.stats = cnt;
  a.blk = blk;
  HIP_OK(nr::run_build_plan(a, stream));
  unsigned long long st[3] = {0, 0, 0};
  HIP_OK(hipMemcpyAsync(st, cnt, sizeof(st), hipMemcpyDeviceToHost, stream));
  HIP_OK(hipStreamSynchronize(stream));
  info->max_clusters = (int64_t)st[0];
  info->n_multi = (int64_t)st[1];
  info->kmax = (int32_t)st[2];
  info->t = t;
  return NR_OK;
}

nr_status nr_build_index(const nr_build_desc *d, int64_t *row_ids, uint32_t *bc_off,
                         uint64_t *cl_off, float *centroids, int64_t *n_clusters,
                         hipStream_t stream) {
  if (!d || !row_ids || !bc_off || !cl_off || !centroids || !n_clusters)
    return fail(NR_EINVAL, "NULL argument");
  if (d->n < 1 || d->n >= ((int64_t)1 << 32)) return fail(NR_EINVAL, "n must be in [1, 2^32)");
  if (d->b < 1 || d->b > 30) return fail(NR_EINVAL, "b must be in [1, 30]");
  if (!d->logits || !d->codes || !d->sizes || !d->kb || (d->n_multi > 0 && (!d->mlist ||
      !d->uniforms)))
    return fail(NR_EINVAL, "NULL input array");
  if (d->lloyd < 1) return fail(NR_EINVAL, "lloyd must be >= 1");
  if (d->sample_per_cluster < 1) return fail(NR_EINVAL, "sample_per_cluster must be >= 1");
  if (d->max_clusters < 1 || d->max_clusters >= ((int64_t)1 << 32))
    return fail(NR_EINVAL, "max_clusters must be in [1, 2^32)");
  if (d->n_multi > 0 && d->kmax < 2) return fail(NR_EINVAL, "kmax must be >= 2");
  const int64_t nb = (int64_t)1 << d->b, n = d->n, mc = d->max_clusters;
  DevScratch ds;
  nr::BuildArgs a{};
  a.n = n;
  a.b = d->b;
  a.lg = d->logits;
  a.codes = d->codes;
  a.sizes = d->sizes;
  a.kb = const_cast<uint32_t *>(d->kb);
  a.mlist = const_cast<uint32_t *>(d->mlist);
  a.n_multi = d->n_multi;
  a.U = d->uniforms;
  a.kmax = d->kmax;
  a.seed = d->seed;
  a.lloyd = d->lloyd;
  a.spc = d->sample_per_cluster;
  const int64_t most = std::max(std::max(nb, n), mc) + 1;
  a.blk = ds.get<uint64_t>(nr::build_scan_blocks(most));
  a.kbpre = ds.get<uint64_t>(nb + 1);
  a.boff = ds.get<uint64_t>(nb + 1);
  a.cursor = ds.get<uint32_t>(nb);
  a.nkept = ds.get<uint32_t>(nb);
  a.ncl = ds.get<uint32_t>(nb);
  a.ids = ds.get<uint32_t>(n);
  a.ids_tmp = ds.get<uint32_t>(n);
  a.label = ds.get<uint32_t>(n);
  a.skey = ds.get<uint64_t>(n);
  a.skey_tmp = ds.get<uint64_t>(n);
  a.d2 = ds.get<double>(n);
  a.cent = ds.get<double>((size_t)mc * d->b);
  a.ccnt = ds.get<uint32_t>(mc);
  a.csize = ds.get<uint64_t>(mc);
  if (!a.blk || !a.kbpre || !a.boff || !a.cursor || !a.nkept || !a.ncl || !a.ids || !a.ids_tmp ||
      !a.label || !a.skey || !a.skey_tmp || !a.d2 || !a.cent || !a.ccnt || !a.csize)
    return fail(NR_ENOMEM, "build scratch allocation failed");
  a.bc_off = bc_off;
  a.row_ids = row_ids;
  a.centroids = centroids;
  HIP_OK(nr::run_build_index(a, stream));
  uint32_t ncl = 0;
  HIP_OK(hipMemcpyAsync(&ncl, bc_off + nb, 4, hipMemcpyDeviceToHost, stream));
  HIP_OK(hipStreamSynchronize(stream));
  if ((int64_t)ncl > mc) return fail(NR_ECORRUPT, "more clusters than planned");
  HIP_OK(nr::launch_build_cl_off(a.csize, (int64_t)ncl, cl_off, a.blk, stream));
  HIP_OK(hipStreamSynchronize(stream));
  *n_clusters = ncl;
  return NR_OK;
}

nr_status nr_profile_enable(nr_index *ix, int32_t on) {
  if (nr_status s = check_index(ix)) return s;
  ix->profiling = on != 0;
  return NR_OK;
}

nr_status nr_profile_read(nr_index *ix, double *stage_ms, int64_t *n_searches, int32_t reset) {
  if (nr_status s = check_index(ix)) return s;
  std::lock_guard<std::mutex> g(ix->mu);
  for (auto &es : ix->pending) {
    HIP_OK(hipEventSynchronize(es.ev[NR_STAGES]));
    for (int i = 0; i < NR_STAGES; ++i) {
      float ms = 0.f;
      HIP_OK(hipEventElapsedTime(&ms, es.ev[i], es.ev[i + 1]));
      ix->stage_ms[i] += ms;
    }
    ix->n_timed += 1;
    for (auto &ev : es.ev) (void)hipEventDestroy(ev);
  }
  ix->pending.clear();
  if (stage_ms)
    for (int i = 0; i < NR_STAGES; ++i) stage_ms[i] = ix->stage_ms[i];
  if (n_searches) *n_searches = ix->n_timed;
  if (reset) {
    for (double &v : ix->stage_ms) v = 0.0;
    ix->n_timed = 0;
  }
  return NR_OK;
}

nr_status nr_last_work(nr_index *ix, hipStream_t stream, int64_t *work, int32_t n_work) {
  if (nr_status s = check_index(ix)) return s;
  if (!work || n_work < 0) return fail(NR_EINVAL, "work must be a host array");
  Workspace *w = nullptr;
  {
    std::lock_guard<std::mutex> g(ix->mu);
    for (auto &x : ix->ws)
      if (x.stream == stream) w = &x;
  }
  if (!w || !w->last.tile_off) return fail(NR_EINVAL, "no search has run on this stream");
  const Buffers &B = w->last;
  const size_t nq = (size_t)w->last_nq;
  if (B.shared) {
    HIP_OK(nr::launch_fill_i32((int32_t *)B.wstats, 2, 0, stream));      // wstats[0]
    HIP_OK(nr::launch_fill_i32((int32_t *)(B.wstats + 2), 2, 0, stream));  // wstats[2]
    HIP_OK(nr::launch_unique_rows(B.slist, B.lpm, B.lmeta, ix->d.cl_off, B.wstats, stream));
    HIP_OK(nr::launch_list_rows(B.clus, B.nclus, w->last_cap, (int64_t)nq, ix->d.cl_off,
                                ix->d.n_clusters, B.rfull, stream));
  }
  HIP_OK(hipStreamSynchronize(stream));
  int64_t v[NR_WORK] = {0};
  int32_t t = 0;
  HIP_OK(hipMemcpy(&t, B.tile_off + nq, 4, hipMemcpyDeviceToHost));
  std::vector<uint32_t> full(nq);
  HIP_OK(hipMemcpy(full.data(), B.rfull, 4 * nq, hipMemcpyDeviceToHost));
  for (uint32_t x : full) v[NR_WORK_ROWS] += x;
  HIP_OK(hipMemcpy(&v[NR_WORK_REFINE_BYTES], B.wstats + 6, 8, hipMemcpyDeviceToHost));
  v[NR_WORK_TILES] = t;
  v[NR_WORK_OWN_ROWS] = v[NR_WORK_ROWS];
  if (B.shared) {
    int64_t ws[6] = {0, 0, 0, 0, 0, 0};  // the first six counters
    uint64_t pairs = 0;
    HIP_OK(hipMemcpy(ws, B.wstats, sizeof(ws), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(&pairs, B.lmeta + 1, 8, hipMemcpyDeviceToHost));
    std::vector<uint32_t> own(nq);
    std::vector<int32_t> flag(nq), scnt(nq);
    HIP_OK(hipMemcpy(own.data(), B.own_rows, 4 * nq, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(flag.data(), B.flag, 4 * nq, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(scnt.data(), B.scnt, 4 * nq, hipMemcpyDeviceToHost));
    v[NR_WORK_TILES] += ws[1];
    v[NR_WORK_OWN_ROWS] = 0;
    for (size_t i = 0; i < nq; ++i) {
      v[NR_WORK_OWN_ROWS] += own[i];
      v[NR_WORK_SURVIVORS] += scnt[i];
      if (flag[i]) {
        v[NR_WORK_FLAGGED] += 1;
        v[NR_WORK_FALLBACK_ROWS] += full[i];
      }
    }
    v[NR_WORK_SHARED_ROWS] = ws[0];
    v[NR_WORK_SHARED_PAIRS] = (int64_t)pairs;
    v[NR_WORK_SHARED_PAIR_ROWS] = ws[2];
    v[NR_WORK_FULL_ROWS] = ws[3];
    v[NR_WORK_BODY_BYTES] = ws[4];
    v[NR_WORK_OPEN_BYTES] = ws[5];
    v[NR_WORK_HEAD_BYTES] = scan_head(ix);
  }
  v[NR_WORK_ROWS_READ] = v[NR_WORK_OWN_ROWS] + v[NR_WORK_SHARED_ROWS] + v[NR_WORK_FALLBACK_ROWS];
  for (int i = 0; i < n_work && i < NR_WORK; ++i) work[i] = v[i];
  return NR_OK;
}

}  // extern "C"
