/*
 * ezsp.h -- C ABI of the MI355X (gfx950) EZ-SP partition library.
 *
 * The library computes the partition step of EZ-SP (arXiv 2512.00385):
 * the exact k-nearest-neighbour adjacency of a point cloud, then the
 * round-synchronous parallel merge of adjacent components that greedily
 * lowers the contour-regularised energy
 *
 *   Omega = sum_p |f_p - y_p|^2 + lambda * sum_(p,q) w_pq [y_p != y_q]
 *                                                   (Sec. 3.2, Eq. gmpp)
 *
 * with the merge gain of Prop. 1 (Eq. delta), Steps 0-4 of Sec. 3.2
 * ("Parallel Implementation"; App. Alg. A-1 and A-2), repeated over a ladder
 * of regularisation strengths (Sec. 3.2, "Hierarchical Partition").
 *
 * Conventions shared by every entry point
 *   - Every array pointer is a DEVICE pointer unless marked (host).  The
 *     caller owns every buffer.  The library allocates nothing on the device:
 *     all scratch memory comes from the caller's workspace `ws` of
 *     `ws_bytes` bytes (size from the matching *_workspace_size query;
 *     any alignment, the library aligns internally).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All device work is enqueued on it.
 *   - ezsp_knn, ezsp_component_stats and ezsp_embed_mlp are
 *     stream-asynchronous: they validate their arguments, enqueue their
 *     kernels and return; their outputs are ready once `stream` reaches
 *     that point, and their workspace must stay allocated until then.
 *     Errors the device detects (a non-finite coordinate, a label out of
 *     range) are kept in the call's workspace and reported by
 *     ezsp_sync_status.  The entry points that return host values
 *     (ezsp_partition, ezsp_partition_from_knn, ezsp_grid_subsample,
 *     ezsp_edge_loss, ezsp_purity) synchronise `stream` before they return
 *     and report device errors themselves; their outputs are complete when
 *     they return EZSP_OK.
 *   - Arguments are validated on the host before anything is launched; an
 *     invalid argument returns EZSP_ERR_INVALID_ARG and touches no memory.
 *   - On any status other than EZSP_OK the outputs are unspecified.
 *   - Calls on different streams with different workspaces may run
 *     concurrently; the only global state is the thread-local message of
 *     ezsp_last_error().
 *   - Arrays are row-major and contiguous: xyz is n*3 fp32, emb is n*d fp32.
 */
#ifndef EZSP_H
#define EZSP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EZSP_OK = 0,
  EZSP_ERR_INVALID_ARG = -1,   /* bad size, pointer, parameter            */
  EZSP_ERR_NONFINITE = -2,     /* NaN or Inf in xyz or emb                */
  EZSP_ERR_RANGE = -3,         /* embeddings too large for the exact
                                  fixed-point sums (shift F < 16)         */
  EZSP_ERR_WORKSPACE = -4,     /* ws_bytes below the queried size         */
  EZSP_ERR_DEVICE = -5,        /* a HIP call failed, or an internal
                                  consistency check on the device tripped */
  EZSP_ERR_NOT_CONVERGED = -6  /* a level reached max_rounds merge rounds */
} ezsp_status;

/* Flags of ezsp_params.flags. */
#define EZSP_F_ENERGY 1u /* fill energy[] (Eq. gmpp per level) */
/* prepare_graph's linking of isolated nodes (App. Alg. A-2), ezsp_partition
 * only: at the start of every round with more than one node, each node
 * without an edge gets an edge of weight 1 to each of its min(k, nodes - 1)
 * nearest nodes, by the squared distance of their centroids (exact int64
 * fixed-point position sums, fp64 means and distance), ties to the
 * superpoint with the smaller smallest point index; a pair linked from both
 * ends is one edge.  The energy's cut term stays on the input graph.  Needs
 * a workspace queried with the flag set; rounds of small graphs then run as
 * separate launches instead of in one kernel. */
#define EZSP_F_LINK_ISOLATED 2u

typedef struct {
  int32_t k;                /* neighbours per point, 1..64                   */
  int32_t n_levels;         /* L >= 1 (at most 16)                           */
  const double *lambdas;    /* (host) L regularisation strengths, finite,
                               >= 0; level l merges with lambdas[l]          */
  const int64_t *min_size;  /* (host) L minimum superpoint sizes s_min, or
                               NULL.  A component smaller than s_min may
                               merge along its best edge even when the gain
                               is not positive (Step 1); values <= 1 disable */
  int32_t max_rounds;       /* merge rounds allowed per level; 0 = 256       */
  uint32_t flags;           /* EZSP_F_* bits                                 */
} ezsp_params;

/* ---- kNN adjacency (Sec. 3.1: a graph linking every point to its k
 * nearest neighbours; Sec. 4.1: unit edge weights) ----------------------- */

size_t ezsp_knn_workspace_size(int64_t n, int32_t k);

/* Exact k nearest neighbours of every point (stream-asynchronous).
 *   xyz  n*3 fp32 (in)
 *   nbr  n*k int32 (out): row p lists the k points q != p with the smallest
 *        (d2(p,q), q), in increasing order, where
 *        d2 = fma(dz, dz, fma(dy, dy, dx*dx)), dx = x_q - x_p, IEEE fp32,
 *        each multiply, subtract and fused multiply-add one rounding.  Ties in d2 go to
 *        the smaller index.  When n-1 < k the row ends in -1 entries.
 *   d2   n*k fp32 (out, nullable): the matching squared distances, +inf
 *        where nbr is -1.
 * Errors returned: INVALID_ARG (n < 1, n > 2^31 - 256, k outside 1..64, NULL
 *         pointer), WORKSPACE, DEVICE (a launch failed).
 * Errors through ezsp_sync_status(ws): NONFINITE, DEVICE. */
int ezsp_knn(const float *xyz, int64_t n, int32_t k, int32_t *nbr, float *d2,
             void *ws, size_t ws_bytes, void *stream);

/* ezsp_knn (same nbr, workspace and errors) with the statistics of its
 * tree walk, for inspection outside timed work: points are sorted into
 * Morton order, cut into buckets of 16 consecutive points, and groups of 64
 * consecutive points (four buckets) walk the box tree together; group g
 * (0 <= g < ceil(n / 64)) gets
 *   group_scans[g]  the buckets whose candidates it scanned, its own
 *                   included
 *   group_nodes[g]  the inner tree nodes it entered
 * (both int32, device memory, written in full).  Stream-asynchronous. */
int ezsp_knn_walk_stats(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                        int32_t *group_scans, int32_t *group_nodes, void *ws,
                        size_t ws_bytes, void *stream);

/* ---- partition (Sec. 3.2: Eq. gmpp, Prop. 1, Steps 0-4, hierarchical
 * partition; App. Alg. A-1, A-2) ----------------------------------------- */

size_t ezsp_partition_workspace_size(int64_t n, int32_t d,
                                     const ezsp_params *p);

/* kNN graph of xyz (as ezsp_knn, one undirected edge of weight 1 per
 * neighbouring pair), then the merge ladder on the embeddings.
 *   xyz     n*3 fp32 (in)
 *   emb     n*d fp32 (in), 1 <= d <= 64
 *   labels  L*n int32 (out): row l holds every point's superpoint at level
 *           l, numbered 0..n_comp[l]-1 in increasing order of each
 *           superpoint's smallest point index
 *   n_comp  (host) L int64 (out): superpoints per level
 *   energy  (host) L double (out, nullable; written when EZSP_F_ENERGY is
 *           set): Omega of Eq. gmpp for level l with lambdas[l], each
 *           superpoint's value being its mean embedding
 * Component means and sums are exact: embeddings enter as int64 fixed point
 * S = rint(e * 2^F), F = min(40, 61 - ceil(log2 n) - max(0, ceil(log2 A))),
 * A = max |e|; gains are fp64 in a fixed operation order, so decisions do not
 * depend on summation order.  Conflict removal keeps, per component, the
 * candidate edge with the largest gain, ties to the smaller neighbour (in the
 * order of smallest point index).
 * Errors: INVALID_ARG (also when 4*k*n >= 2^31: the adjacency tables are
 *         int32-indexed), NONFINITE, RANGE (F < 16), WORKSPACE, DEVICE,
 *         NOT_CONVERGED. */
int ezsp_partition(const float *xyz, const float *emb, int64_t n, int32_t d,
                   const ezsp_params *p, int32_t *labels, int64_t *n_comp,
                   double *energy, void *ws, size_t ws_bytes, void *stream);

/* The merge ladder on a given neighbour table instead of xyz.
 *   nbr  n*k int32 (in): entries in [-1, n); -1 and q == p are ignored,
 *        repeated entries count once.  The graph is the set of unordered
 *        pairs {p, q} with q in row p or p in row q, each of weight 1.
 * Other arguments and errors as ezsp_partition (p->k is the row length). */
int ezsp_partition_from_knn(const int32_t *nbr, const float *emb, int64_t n,
                            int32_t d, const ezsp_params *p, int32_t *labels,
                            int64_t *n_comp, double *energy, void *ws,
                            size_t ws_bytes, void *stream);

/* ---- per-superpoint attributes (Sec. 3.2: mean embedding Y_P of each
 * superpoint; App. Alg. A-2, component_attributes) ----------------------- */

size_t ezsp_component_stats_workspace_size(int64_t n, int64_t n_comp,
                                           int32_t d);

/* Size, mean embedding and centroid of every superpoint of a labelling
 * (stream-asynchronous).
 *   labels    n int32 (in), each in [0, n_comp)
 *   emb       n*d fp32 (in); xyz n*3 fp32 (in, nullable)
 *   size      n_comp int64 (out)
 *   emb_mean  n_comp*d fp32 (out): ((double)sum S / size) * 2^-F rounded to
 *             fp32, S the fixed point of emb with F by the rule above
 *             (0 for an empty superpoint)
 *   centroid  n_comp*3 fp32 (out, NULL when xyz is NULL): the same for xyz
 *             with its own F
 * Errors returned: INVALID_ARG, WORKSPACE, DEVICE (a launch failed).
 * Errors through ezsp_sync_status(ws): INVALID_ARG (a label outside
 *         [0, n_comp)), NONFINITE, RANGE, DEVICE. */
int ezsp_component_stats(const int32_t *labels, int64_t n, int64_t n_comp,
                         const float *emb, int32_t d, const float *xyz,
                         int64_t *size, float *emb_mean, float *centroid,
                         void *ws, size_t ws_bytes, void *stream);

/* ---- grid subsampling (Sec. 4.1: every cloud is subsampled on a regular
 * grid before it is partitioned) ------------------------------------------ */

size_t ezsp_grid_subsample_workspace_size(int64_t n);

/* Keeps one point per occupied cell of a regular grid of spacing h.
 *   xyz      n*3 fp32 (in)
 *   h        cell size, finite and > 0
 *   keep     n int32 (out): the first *n_keep entries are the kept point
 *            indices in increasing order; the rest is unspecified
 *   n_keep   (host, out) number of kept points
 * A point's cell is floor((x_i - o_i) / h) on each axis, computed in IEEE
 * fp32 (one subtraction, one correctly rounded division), o the
 * coordinate-wise minimum of xyz; each cell keeps its smallest point index.
 * Errors: INVALID_ARG, NONFINITE, RANGE (2^21 or more cells on an axis),
 *         WORKSPACE, DEVICE. */
int ezsp_grid_subsample(const float *xyz, int64_t n, float h, int32_t *keep,
                        int64_t *n_keep, void *ws, size_t ws_bytes,
                        void *stream);

/* ---- affinity and contrastive edge loss (Sec. 3.1, Eq. softmax and
 * Eq. loss) --------------------------------------------------------------- */

typedef struct {
  double loss;          /* Eq. loss summed over the sampled pairs          */
  int64_t n_edges;      /* unordered pairs of the kNN relation             */
  int64_t n_intra;      /* pairs whose end points share a class            */
  int64_t n_inter;      /* the others; every inter pair is sampled         */
  int64_t n_intra_kept; /* intra pairs in the sample                       */
} ezsp_loss_stats;

size_t ezsp_edge_loss_workspace_size(int64_t n, int32_t k);

/* Affinity a_pq = exp(-|e_p - e_q| / tau) and the contrastive loss
 *   L = sum_intra -log a_pq + sum_inter -log(1 - a_pq)
 * over the unordered pairs of a neighbour table, intra pairs sampled.
 *   emb       n*d fp32 (in), d in 1..1024
 *   nbr       n*k int32 (in), k in 1..64: neighbour ids in [0, n) or -1
 *             (empty slot)
 *   cls       n int32 (in): class of every point (only equality matters)
 *   word      n*k uint32 (in): one random word per slot
 *   tau       temperature, finite and > 0; rho in [0, 1]
 *   affinity  n*k fp32 (out, nullable): a for every non-empty slot, 0 for
 *             empty ones
 *   grad      n*d fp32 (out, nullable): dL/d emb
 *   sampled   n*k uint8 (out, nullable): 1 where the slot owns a pair of
 *             the sample
 *   out       (host, out) the loss and the pair counts
 * A pair {p, q} belongs to the smallest slot p*k + j listing it, and that
 * slot's word draws it.  With rho < 1 the sample keeps the
 * m = min(n_intra, floor(rho * n_inter / (1 - rho))) intra pairs with the
 * smallest (word, slot); rho = 1 keeps them all.  -log a is evaluated as
 * d / tau and -log(1 - a) as -log(-expm1(-d / tau)); the gradient of
 * |e_p - e_q| at e_p = e_q is taken as 0.  Distances, affinities and the
 * gradient are fp32 (the gradient is accumulated with atomics, so its last
 * bits vary between runs); the loss is summed in fp64.
 * Errors: INVALID_ARG (also a neighbour id outside [-1, n), detected on the
 *         device), NONFINITE, WORKSPACE, DEVICE. */
int ezsp_edge_loss(const float *emb, int64_t n, int32_t d, const int32_t *nbr,
                   int32_t k, const int32_t *cls, const uint32_t *word,
                   double tau, double rho, float *affinity, float *grad,
                   uint8_t *sampled, ezsp_loss_stats *out, void *ws,
                   size_t ws_bytes, void *stream);

/* ---- purity and oracle mIoU (Sec. 4.2 "Metrics") ------------------------- */

typedef struct {
  double miou;       /* mean over the classes present of the IoU between
                        the classes and the superpoints' majority classes */
  double purity;     /* share of points whose class is their superpoint's
                        majority class                                     */
  int64_t n_present; /* classes that occur in cls                          */
} ezsp_purity_stats;

size_t ezsp_purity_workspace_size(int64_t n, int64_t n_comp, int32_t n_cls);

/* Gives every superpoint its majority class and scores that labelling.
 *   labels    n int32 (in), each in [0, n_comp)
 *   cls       n int32 (in), each in [0, n_cls)
 *   majority  n_comp int32 (out, nullable): majority class, ties to the
 *             smallest class, -1 for an empty superpoint
 *   iou       n_cls fp64 (out, nullable): TP / (|cls = c| + |pred = c| - TP),
 *             NaN for a class absent from cls
 *   out       (host, out) mIoU (IoUs summed in class order), purity
 * Errors: INVALID_ARG (also ids out of range, detected on the device),
 *         WORKSPACE, DEVICE. */
int ezsp_purity(const int32_t *labels, int64_t n, int64_t n_comp,
                const int32_t *cls, int32_t n_cls, int32_t *majority,
                double *iou, ezsp_purity_stats *out, void *ws,
                size_t ws_bytes, void *stream);

/* ---- point-embedding MLP (stand-in for the embedding network of
 * Sec. 3.1 on the LiDAR-sweep workload) ----------------------------------- */

/* out[p] = L3(h2), h2 = bf16(relu(L2(h1))), h1 = bf16(relu(L1(x[p]))),
 * L(v) = v W + b: a per-point MLP d_in -> 32 -> 32 -> d_out on the matrix
 * cores.  bf16 = round to nearest even; products of bfloat16 values are
 * accumulated in fp32 (the summation order is the matrix unit's).
 *   x    n*d_in bfloat16 bit patterns (in), d_in in 1..8
 *   w1   d_in*32, w2 32*32, w3 32*d_out bfloat16 bits, row k = input k
 *   b1   32, b2 32, b3 d_out fp32
 *   out  n*d_out fp32 (out), d_out in 1..32
 * d_hid must be 32.  Needs no workspace.  Stream-asynchronous; the device
 * detects no errors.
 * Errors: INVALID_ARG, DEVICE (the launch failed). */
int ezsp_embed_mlp(const uint16_t *x, int64_t n, int32_t d_in, int32_t d_hid,
                   int32_t d_out, const uint16_t *w1, const float *b1,
                   const uint16_t *w2, const float *b2, const uint16_t *w3,
                   const float *b3, float *out, void *stream);

/* ---- kNN without a workspace --------------------------------------------- */

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): ezsp_knn
 * with its scratch in a static device array of 160 MiB instead of a caller
 * workspace.  Same arguments, results and errors as ezsp_knn (bit-identical
 * outputs); stream-asynchronous, device-detected errors through
 * ezsp_sync_status(NULL, 0, stream).  The call allocates nothing: no
 * hipMalloc, hipFree or other allocating routine.  Sizes whose
 * ezsp_knn_workspace_size(n, k) exceeds 160 MiB (about 1.5M points at
 * k = 10) return EZSP_ERR_INVALID_ARG.  Each GPU the library runs on holds
 * its own copy of the array until the process ends; every call on one GPU
 * uses that copy, so calls that overlap on one GPU (other streams, other
 * threads) race. */
int ezsp_knn_noalloc(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                     float *d2, void *stream);

/* ---- diagnostics --------------------------------------------------------- */

/* Synchronises `stream` and returns the status of the errors the device
 * detected in the last call that used the workspace `ws` (ws_bytes as
 * passed to that call), or, with ws = NULL and ws_bytes = 0, in the last
 * ezsp_knn_noalloc call on the current device: EZSP_OK, or the error with
 * its detail in ezsp_last_error().  For the stream-asynchronous entry
 * points; the others report device errors themselves. */
int ezsp_sync_status(const void *ws, size_t ws_bytes, void *stream);

/* Static text for a status code. */
const char *ezsp_status_string(int status);

/* Detail of the last error on the calling thread ("" if none). */
const char *ezsp_last_error(void);

/* Per-stage timing with HIP events recorded on the caller's stream around
 * the launches of each stage ("knn_query", "morton_sort", "graph_build",
 * "select", "union", "stats", "contract", "compose", "tail", "link",
 * "grid_subsample", "edge_loss", "purity", "embed_mlp").  Off by default; a
 * diagnostic for benchmarks.  ezsp_profile_enable(1) clears the totals and
 * starts recording, ezsp_profile_enable(0) stops.  ezsp_profile_read gives
 * the number of recorded launches of `stage`, their summed duration in
 * milliseconds and the summed algorithmic bytes the stage has to move (its
 * input and output arrays, each counted once; host pointers, each
 * nullable); it returns -1, with zeros, for a stage never recorded.
 * Process-wide state: not for concurrent callers. */
int ezsp_profile_enable(int on);
int ezsp_profile_read(const char *stage, int64_t *launches, double *ms,
                      double *alg_bytes);

/* Restricts the event recording to one stage (NULL or "" = every stage,
 * the default); the other stages still add their algorithmic bytes.  Lets a
 * benchmark time one stage inside otherwise untouched steps.  Returns 0.
 * Process-wide state like the above. */
int ezsp_profile_only(const char *stage);

#ifdef __cplusplus
}
#endif
#endif /* EZSP_H */
