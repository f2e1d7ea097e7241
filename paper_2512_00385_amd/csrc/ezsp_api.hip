// ezsp_api.hip -- the extern "C" entry points declared in include/ezsp.h:
// argument validation on the host, workspace carving, and dispatch to the
// kernel launchers.
#include <math.h>
#include <string.h>

#include "../../include/ezsp.h"
#include "ezsp_internal.h"

namespace ezsp {
const char *last_error_text();
int prof_enable(int on);
int prof_only(const char *name);
int prof_read(const char *name, int64_t *launches, double *ms,
              double *bytes);
}

using namespace ezsp;

namespace {

constexpr int64_t kMaxN = (int64_t)1 << 31;

// Aligns the caller's workspace; Ctl first, then the rest.
Arena open_ws(void *ws, size_t bytes) {
  Arena a;
  uintptr_t p = reinterpret_cast<uintptr_t>(ws);
  uintptr_t q = (p + 255) & ~uintptr_t(255);
  a.base = reinterpret_cast<char *>(q);
  a.cap = (bytes > (q - p)) ? bytes - (q - p) : 0;
  return a;
}

int fail(int code, const char *msg) {
  set_error("%s", msg);
  return code;
}

// Point counts leave room for grids of 256-thread blocks and whole buckets
// of padding in int32 arithmetic.
bool n_ok(int64_t n) { return n >= 1 && n <= kMaxN - 256; }

// Graph tables are indexed with int32: 2*k*n directed entries, and windows
// of up to twice that, must fit.
bool edges_ok(int64_t n, int32_t k) {
  return 4 * n * (int64_t)k < kMaxN - 1;
}

int check_params(int64_t n, int32_t d, const ezsp_params *p) {
  if (!p) return fail(EZSP_ERR_INVALID_ARG, "params is NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (d < 1 || d > 64) return fail(EZSP_ERR_INVALID_ARG, "d must be in 1..64");
  if (p->k < 1 || p->k > 64)
    return fail(EZSP_ERR_INVALID_ARG, "k must be in 1..64");
  if (!edges_ok(n, p->k))
    return fail(EZSP_ERR_INVALID_ARG, "4*k*n must stay below 2^31");
  if ((int64_t)n * d >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "n*d must stay below 2^31");
  if (p->n_levels < 1 || p->n_levels > 16)
    return fail(EZSP_ERR_INVALID_ARG, "n_levels must be in 1..16");
  if (!p->lambdas) return fail(EZSP_ERR_INVALID_ARG, "lambdas is NULL");
  for (int32_t l = 0; l < p->n_levels; ++l)
    if (!isfinite(p->lambdas[l]) || p->lambdas[l] < 0.0)
      return fail(EZSP_ERR_INVALID_ARG, "every lambda must be finite and >= 0");
  if (p->max_rounds < 0)
    return fail(EZSP_ERR_INVALID_ARG, "max_rounds must be >= 0");
  if (p->flags & ~(EZSP_F_ENERGY | EZSP_F_LINK_ISOLATED))
    return fail(EZSP_ERR_INVALID_ARG, "unknown flag bits");
  return EZSP_OK;
}

size_t partition_bytes(int64_t n, int32_t d, int32_t k, bool with_knn,
                       bool link) {
  Arena a;
  a.take<Ctl>(1);
  if (with_knn) {
    KnnWork w;
    knn_reserve(a, (int32_t)n, k, &w);
  }
  ladder_reserve(a, (int32_t)n, d, k, link);
  return a.off + 512;
}

int run_partition(const float *xyz, const int32_t *nbr_in, const float *emb,
                  int64_t n, int32_t d, const ezsp_params *p, int32_t *labels,
                  int64_t *n_comp, double *energy, void *ws, size_t ws_bytes,
                  void *stream) {
  const bool with_knn = xyz != nullptr;
  const bool link = (p->flags & EZSP_F_LINK_ISOLATED) != 0;
  if (link && !with_knn)
    return fail(EZSP_ERR_INVALID_ARG,
                "EZSP_F_LINK_ISOLATED needs the positions (ezsp_partition)");
  if (ws_bytes < partition_bytes(n, d, p->k, with_knn, link))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  LadderArgs g;
  memset(&g, 0, sizeof(g));
  if (with_knn) {
    KnnWork w;
    knn_reserve(a, (int32_t)n, p->k, &w);
    // rows of 4, 8, 12 or 16 floats at a 16-byte aligned base: the kNN
    // kernel copies them into internal order for the ladder on the way
    g.emb_ready = d % 4 == 0 && d <= 16 &&
                  (reinterpret_cast<uintptr_t>(emb) & 15) == 0;
    int rc = check_hip(
        g.emb_ready
            ? knn_launch_emb(xyz, (int32_t)n, p->k, ctl, w, emb, d,
                             ladder_emb_slot(a, (int32_t)n, d, p->k, link),
                             st)
            : knn_launch(xyz, (int32_t)n, p->k, ctl, w, nullptr, nullptr,
                         st),
        "knn launch");
    if (rc) return rc;
    g.nbr = w.nbr_int;
    g.pts = w.pts;
    g.kth = w.kth;
    g.perm = w.perm;
    g.inv = w.inv;
    g.check_nbr = false;
  } else {
    g.nbr = nbr_in;
    g.check_nbr = true;
  }
  g.emb = emb;
  g.n = (int32_t)n;
  g.d = d;
  g.k = p->k;
  g.n_levels = p->n_levels;
  g.lambdas = p->lambdas;
  g.min_size = p->min_size;
  g.max_rounds = p->max_rounds;
  g.want_energy = (p->flags & EZSP_F_ENERGY) != 0;
  g.link = link;
  g.labels = labels;
  g.n_comp = n_comp;
  g.energy = energy;
  return ladder_run(g, ctl, a, st);
}

}  // namespace

extern "C" {

const char *ezsp_status_string(int status) {
  switch (status) {
    case EZSP_OK: return "ok";
    case EZSP_ERR_INVALID_ARG: return "invalid argument";
    case EZSP_ERR_NONFINITE: return "non-finite input";
    case EZSP_ERR_RANGE: return "embeddings out of fixed-point range";
    case EZSP_ERR_WORKSPACE: return "workspace too small";
    case EZSP_ERR_DEVICE: return "device error";
    case EZSP_ERR_NOT_CONVERGED: return "max_rounds reached";
    default: return "unknown status";
  }
}

const char *ezsp_last_error(void) { return last_error_text(); }

int ezsp_profile_enable(int on) { return prof_enable(on); }

int ezsp_profile_only(const char *stage) { return prof_only(stage); }

int ezsp_profile_read(const char *stage, int64_t *launches, double *ms,
                      double *alg_bytes) {
  return prof_read(stage, launches, ms, alg_bytes);
}

size_t ezsp_knn_workspace_size(int64_t n, int32_t k) {
  if (!n_ok(n) || k < 1 || k > 64 || (int64_t)n * k >= kMaxN) return 0;
  Arena a;
  a.take<Ctl>(1);
  KnnWork w;
  knn_reserve(a, (int32_t)n, k, &w);
  return a.off + 512;
}

int ezsp_knn(const float *xyz, int64_t n, int32_t k, int32_t *nbr, float *d2,
             void *ws, size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!xyz || !nbr || !ws)
    return fail(EZSP_ERR_INVALID_ARG, "xyz, nbr and ws must not be NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (k < 1 || k > 64) return fail(EZSP_ERR_INVALID_ARG, "k must be in 1..64");
  if ((int64_t)n * k >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "n*k must stay below 2^31");
  if (ws_bytes < ezsp_knn_workspace_size(n, k))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  KnnWork w;
  knn_reserve(a, (int32_t)n, k, &w);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  // stream-asynchronous: device-detected errors stay in the workspace's
  // control block for ezsp_sync_status
  return check_hip(knn_launch(xyz, (int32_t)n, k, ctl, w, nbr, d2, st),
                   "knn launch");
}

int ezsp_knn_walk_stats(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                        int32_t *group_scans, int32_t *group_nodes, void *ws,
                        size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!xyz || !nbr || !group_scans || !group_nodes || !ws)
    return fail(EZSP_ERR_INVALID_ARG, "pointers must not be NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (k < 1 || k > 64) return fail(EZSP_ERR_INVALID_ARG, "k must be in 1..64");
  if ((int64_t)n * k >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "n*k must stay below 2^31");
  if (ws_bytes < ezsp_knn_workspace_size(n, k))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  KnnWork w;
  knn_reserve(a, (int32_t)n, k, &w);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  return check_hip(knn_launch_stats(xyz, (int32_t)n, k, ctl, w, nbr,
                                    group_scans, group_nodes, st),
                   "knn launch");
}

int ezsp_sync_status(const void *ws, size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!ws && ws_bytes == 0) {  // the static scratch of ezsp_knn_noalloc
    void *p = nullptr;
    const int rc = noalloc_scratch(&p);
    if (rc) return rc;
    ws = p;
    ws_bytes = kNoallocScratchBytes;
  }
  if (!ws || ws_bytes < sizeof(Ctl) + 256)
    return fail(EZSP_ERR_INVALID_ARG, "ws must be a call's workspace");
  Arena a = open_ws(const_cast<void *>(ws), ws_bytes);
  return device_status(a.take<Ctl>(1), static_cast<hipStream_t>(stream));
}

size_t ezsp_partition_workspace_size(int64_t n, int32_t d,
                                     const ezsp_params *p) {
  if (!p || !n_ok(n) || d < 1 || d > 64 || p->k < 1 || p->k > 64 ||
      !edges_ok(n, p->k))
    return 0;
  return partition_bytes(n, d, p->k, true,
                         (p->flags & EZSP_F_LINK_ISOLATED) != 0);
}

int ezsp_partition(const float *xyz, const float *emb, int64_t n, int32_t d,
                   const ezsp_params *p, int32_t *labels, int64_t *n_comp,
                   double *energy, void *ws, size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!xyz || !emb || !labels || !n_comp || !ws)
    return fail(EZSP_ERR_INVALID_ARG,
                "xyz, emb, labels, n_comp and ws must not be NULL");
  int rc = check_params(n, d, p);
  if (rc) return rc;
  return run_partition(xyz, nullptr, emb, n, d, p, labels, n_comp, energy, ws,
                       ws_bytes, stream);
}

int ezsp_partition_from_knn(const int32_t *nbr, const float *emb, int64_t n,
                            int32_t d, const ezsp_params *p, int32_t *labels,
                            int64_t *n_comp, double *energy, void *ws,
                            size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!nbr || !emb || !labels || !n_comp || !ws)
    return fail(EZSP_ERR_INVALID_ARG,
                "nbr, emb, labels, n_comp and ws must not be NULL");
  int rc = check_params(n, d, p);
  if (rc) return rc;
  return run_partition(nullptr, nbr, emb, n, d, p, labels, n_comp, energy, ws,
                       ws_bytes, stream);
}

size_t ezsp_component_stats_workspace_size(int64_t n, int64_t n_comp,
                                           int32_t d) {
  if (!n_ok(n) || n_comp < 1 || n_comp >= kMaxN || d < 1 || d > 64 ||
      n_comp * d >= kMaxN)
    return 0;
  Arena a;
  a.take<Ctl>(1);
  stats_reserve(a, (int32_t)n, n_comp, d);
  return a.off + 512;
}

int ezsp_component_stats(const int32_t *labels, int64_t n, int64_t n_comp,
                         const float *emb, int32_t d, const float *xyz,
                         int64_t *size, float *emb_mean, float *centroid,
                         void *ws, size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!labels || !emb || !size || !emb_mean || !ws)
    return fail(EZSP_ERR_INVALID_ARG,
                "labels, emb, size, emb_mean and ws must not be NULL");
  if (xyz && !centroid)
    return fail(EZSP_ERR_INVALID_ARG, "centroid must be given with xyz");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (d < 1 || d > 64) return fail(EZSP_ERR_INVALID_ARG, "d must be in 1..64");
  if (n_comp < 1 || n_comp >= kMaxN || n_comp * d >= kMaxN || n * d >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "n_comp out of range");
  if (ws_bytes < ezsp_component_stats_workspace_size(n, n_comp, d))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  return stats_run(labels, (int32_t)n, (int32_t)n_comp, emb, d, xyz, size,
                   emb_mean, centroid, ctl, a, st);
}

size_t ezsp_grid_subsample_workspace_size(int64_t n) {
  if (!n_ok(n)) return 0;
  Arena a;
  a.take<Ctl>(1);
  grid_reserve(a, (int32_t)n);
  return a.off + 512;
}

int ezsp_grid_subsample(const float *xyz, int64_t n, float h, int32_t *keep,
                        int64_t *n_keep, void *ws, size_t ws_bytes,
                        void *stream) {
  set_error("%s", "");
  if (!xyz || !keep || !n_keep || !ws)
    return fail(EZSP_ERR_INVALID_ARG,
                "xyz, keep, n_keep and ws must not be NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (!(h > 0.0f) || !isfinite(h))
    return fail(EZSP_ERR_INVALID_ARG, "h must be finite and > 0");
  if (ws_bytes < ezsp_grid_subsample_workspace_size(n))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  return grid_run(xyz, (int32_t)n, h, keep, n_keep, ctl, a, st);
}

size_t ezsp_edge_loss_workspace_size(int64_t n, int32_t k) {
  if (!n_ok(n) || k < 1 || k > 64 || n * (int64_t)k >= kMaxN) return 0;
  Arena a;
  a.take<Ctl>(1);
  loss_reserve(a, (int32_t)n, k);
  return a.off + 512;
}

int ezsp_edge_loss(const float *emb, int64_t n, int32_t d, const int32_t *nbr,
                   int32_t k, const int32_t *cls, const uint32_t *word,
                   double tau, double rho, float *affinity, float *grad,
                   uint8_t *sampled, ezsp_loss_stats *out, void *ws,
                   size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!emb || !nbr || !cls || !word || !out || !ws)
    return fail(EZSP_ERR_INVALID_ARG,
                "emb, nbr, cls, word, out and ws must not be NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (d < 1 || d > 1024)
    return fail(EZSP_ERR_INVALID_ARG, "d must be in 1..1024");
  if (k < 1 || k > 64 || n * (int64_t)k >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "k must be in 1..64 with n*k below 2^31");
  if (n * (int64_t)d >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "n*d must stay below 2^31");
  if (!(tau > 0.0) || !isfinite(tau))
    return fail(EZSP_ERR_INVALID_ARG, "tau must be finite and > 0");
  if (!(rho >= 0.0 && rho <= 1.0))
    return fail(EZSP_ERR_INVALID_ARG, "rho must be in [0, 1]");
  if (ws_bytes < ezsp_edge_loss_workspace_size(n, k))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  LossArgs g;
  g.emb = emb;
  g.n = (int32_t)n;
  g.d = d;
  g.nbr = nbr;
  g.k = k;
  g.cls = cls;
  g.word = word;
  g.tau = tau;
  g.rho = rho;
  g.affinity = affinity;
  g.grad = grad;
  g.sampled = sampled;
  LossResult r;
  int rc = loss_run(g, &r, ctl, a, st);
  if (rc) return rc;
  out->loss = r.loss;
  out->n_edges = r.n_edges;
  out->n_intra = r.n_intra;
  out->n_inter = r.n_inter;
  out->n_intra_kept = r.n_intra_kept;
  return EZSP_OK;
}

size_t ezsp_purity_workspace_size(int64_t n, int64_t n_comp, int32_t n_cls) {
  if (!n_ok(n) || n_comp < 1 || n_comp >= kMaxN || n_cls < 1 ||
      n_comp > ((int64_t)1 << 62) / n_cls)
    return 0;
  Arena a;
  a.take<Ctl>(1);
  purity_reserve(a, (int32_t)n, (int32_t)n_comp, n_cls);
  return a.off + 512;
}

int ezsp_purity(const int32_t *labels, int64_t n, int64_t n_comp,
                const int32_t *cls, int32_t n_cls, int32_t *majority,
                double *iou, ezsp_purity_stats *out, void *ws,
                size_t ws_bytes, void *stream) {
  set_error("%s", "");
  if (!labels || !cls || !out || !ws)
    return fail(EZSP_ERR_INVALID_ARG,
                "labels, cls, out and ws must not be NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (n_comp < 1 || n_comp >= kMaxN || n_cls < 1 ||
      n_comp > ((int64_t)1 << 62) / n_cls)
    return fail(EZSP_ERR_INVALID_ARG, "n_comp or n_cls out of range");
  if (ws_bytes < ezsp_purity_workspace_size(n, n_comp, n_cls))
    return fail(EZSP_ERR_WORKSPACE, "workspace smaller than the queried size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  Arena a = open_ws(ws, ws_bytes);
  Ctl *ctl = a.take<Ctl>(1);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, ctl);
  PurityResult r;
  int rc = purity_run(labels, (int32_t)n, (int32_t)n_comp, cls, n_cls,
                      majority, iou, &r, ctl, a, st);
  if (rc) return rc;
  out->miou = r.miou;
  out->purity = r.purity;
  out->n_present = r.n_present;
  return EZSP_OK;
}

int ezsp_embed_mlp(const uint16_t *x, int64_t n, int32_t d_in, int32_t d_hid,
                   int32_t d_out, const uint16_t *w1, const float *b1,
                   const uint16_t *w2, const float *b2, const uint16_t *w3,
                   const float *b3, float *out, void *stream) {
  set_error("%s", "");
  if (!x || !w1 || !b1 || !w2 || !b2 || !w3 || !b3 || !out)
    return fail(EZSP_ERR_INVALID_ARG, "no pointer may be NULL");
  if (!n_ok(n)) return fail(EZSP_ERR_INVALID_ARG, "n must be in [1, 2^31 - 256]");
  if (d_in < 1 || d_in > 8 || d_hid != 32 || d_out < 1 || d_out > 32)
    return fail(EZSP_ERR_INVALID_ARG,
                "the MLP is d_in (1..8) -> 32 -> 32 -> d_out (1..32)");
  if (n * (int64_t)d_out >= kMaxN || n * (int64_t)d_in >= kMaxN)
    return fail(EZSP_ERR_INVALID_ARG, "n*d_out must stay below 2^31");
  return mlp_run(x, (int32_t)n, d_in, d_out, w1, b1, w2, b2, w3, b3, out,
                 static_cast<hipStream_t>(stream));
}

}  // extern "C"
