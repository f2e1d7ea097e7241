/*
 * ezsp_oracle.h -- plain sequential CPU oracle for the EZ-SP partition step.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the GPU path; it is
 * never called by the product library.  Only the test-suite, the smoke check
 * and the CPU-baseline leg of the benchmark may load it.  It shares no code,
 * header, table or helper with the HIP path.
 *
 * What it computes (arXiv 2512.00385):
 *   - the undirected k-nearest-neighbour adjacency, weights w = 1
 *     (Sec. 3.1 "Semantic Transition Prediction", Sec. 4.1 "Implementation
 *     Details");
 *   - the contour-regularised energy  Omega = sum_p |f_p - y_p|^2
 *       + lambda * sum_(p,q) w_pq [y_p != y_q]          (Sec. 3.2, Eq. gmpp);
 *   - the merge gain  Delta(P,Q) = -|P||Q|/(|P|+|Q|) |f_P - f_Q|^2
 *       + lambda * w_PQ                                  (Prop. 1, Eq. delta);
 *   - the round-synchronous parallel merge: candidate merges, conflict
 *     removal, weakly-connected-component merging, recalibration
 *     (Sec. 3.2 "Parallel Implementation", Steps 0-4; App. Alg. A-1, A-2),
 *     applied recursively over a ladder of regularisation strengths
 *     (Sec. 3.2 "Hierarchical Partition");
 *   - the grid subsampling applied before partitioning (Sec. 4.1);
 *   - the pairwise affinity and the contrastive edge loss with intra-edge
 *     dropping (Sec. 3.1, Eq. softmax, Eq. loss);
 *   - partition purity and oracle mIoU (Sec. 4.2 "Metrics");
 *   - a random-weight point-embedding MLP standing in for the embedding
 *     network of Sec. 3.1 (reading R20).
 *
 * Readings taken where the paper is silent (each one is listed, with the
 * reason, in the design notes of the repository):
 *   R1  kNN excludes the point itself by index; d2 is IEEE fp32,
 *       d2 = fma(dz, dz, fma(dy, dy, dx*dx)) with dx = x_q - x_p, fp32;
 *       neighbours ordered by (d2, index); -1 padding when n-1 < k.
 *   R2  the graph is the union of the kNN relations, one edge per unordered
 *       pair, w = 1.
 *   R3  component sums are exact int64 fixed point, S = rint(e * 2^F); means
 *       and gains are fp64 in a fixed operation order.
 *   R4  component ids are ordered by their smallest member index.
 *   R5  conflict removal keeps, per node, the incident candidate edge that is
 *       largest under (Delta desc, lo asc, hi asc).
 *   R6  |P| < s_min is strict; s_min <= 1 disables it.
 *   R7  linking of isolated nodes (prepare_graph), when asked for: at the
 *       start of every round with more than one node, each node without an
 *       edge gets an edge of weight 1 to each of its min(k, nn-1) nearest
 *       nodes (squared distance of exact fixed-point centroids in fp64, then
 *       the smaller id); a pair linked from both ends is one edge.
 *   R8  the cut term counts edges whose end points lie in different
 *       components.
 *   R9  level l+1 starts from level l's contracted graph and statistics.
 *   R10 Delta > 0 is strict.
 *   R13 grid cells are floor((x_i - o_i) / h) in IEEE fp32 with o the
 *       coordinate-wise minimum; each cell keeps its smallest point index.
 *   R14 loss edges are the unordered kNN pairs; an edge belongs to the
 *       smallest slot p*k + j that lists it, whose random word draws it.
 *   R15 rho < 1 keeps the m = min(n_intra, floor(rho*n_inter/(1-rho)))
 *       intra edges with the smallest (word, slot); rho = 1 keeps all.
 *   R16 -log(a) = d/tau, -log(1 - a) = -log(-expm1(-d/tau)), summed.
 *   R17 the gradient of |e_p - e_q| at e_p = e_q is 0.
 *   R18 majority ties go to the smallest class; IoU over the classes present
 *       in the ground truth; purity = matched points / n.
 *   R20 the embedding MLP: bfloat16 inputs, weights and hidden activations
 *       (round to nearest even), exact dot products, fp32 biases, ReLU after
 *       the hidden layers.
 *
 * Conventions: all pointers are host pointers owned by the caller.
 * Functions return 0 on success and a negative code on error:
 *   -1 invalid argument, -2 non-finite input, -3 fixed-point range,
 *   -4 out of memory, -6 round cap reached.
 */
#ifndef EZSP_ORACLE_H
#define EZSP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- kNN (Sec. 3.1, Sec. 4.1; reading R1) -------------------------------- */

/* Brute force over all pairs.  nbr: n*k int32 (out), d2: n*k fp32 (out,
 * nullable). */
int or_knn_brute(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                 float *d2);

/* Brute force for the single query point p (k entries). */
int or_knn_one(const float *xyz, int64_t n, int32_t k, int64_t p,
               int32_t *nbr, float *d2);

/* Exact kNN through a k-d tree; same output as or_knn_brute. */
int or_knn_kdtree(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                  float *d2);

/* ---- graph (reading R2) -------------------------------------------------- */

/* Unique undirected edges of the kNN relation, sorted by (lo, hi), w = 1.
 * lo, hi, w: capacity n*k.  Returns the edge count or a negative code. */
int64_t or_graph(const int32_t *nbr, int64_t n, int32_t k, int32_t *lo,
                 int32_t *hi, int64_t *w);

/* ---- fixed point (reading R3) -------------------------------------------- */

/* F = min(40, 61 - ceil(log2 n) - max(0, ceil(log2 A))), A = max |e|.
 * Returns F, or -2 on a non-finite value, -3 when F < 16. */
int or_fixed_shift(const float *emb, int64_t n, int32_t d);

/* S[p*d+i] = rint(e[p*d+i] * 2^F), round half to even. */
void or_quantize(const float *emb, int64_t n, int32_t d, int32_t F,
                 int64_t *S);

/* ---- one merge round, exposed step by step ------------------------------- */

/* Eq. delta for every edge.  size: nn, S: nn*d (fixed point). */
void or_gains(int64_t ne, const int32_t *lo, const int32_t *hi,
              const int64_t *w, const int64_t *size, const int64_t *S,
              int32_t d, int32_t F, double lambda, double *delta);

/* Steps 1-2: target[v] = other end of v's retained edge, or -1. */
void or_select(int64_t nn, int64_t ne, const int32_t *lo, const int32_t *hi,
               const double *delta, const int64_t *size, int64_t min_size,
               int32_t *target);

/* Step 3: weakly connected components of {v -> target[v]}, numbered by
 * smallest member (reading R4).  Returns the component count. */
int64_t or_components(int64_t nn, const int32_t *target, int32_t *label);

/* Step 4: component sizes and sums, and the contracted edge list (sorted by
 * (lo, hi), self loops dropped, weights of parallel edges added).
 * out arrays: size_out nc, S_out nc*d, lo/hi/w_out capacity ne.
 * Returns the contracted edge count. */
int64_t or_contract(int64_t nn, int64_t ne, const int32_t *lo,
                    const int32_t *hi, const int64_t *w, const int64_t *size,
                    const int64_t *S, int32_t d, const int32_t *label,
                    int64_t nc, int64_t *size_out, int64_t *S_out,
                    int32_t *lo_out, int32_t *hi_out, int64_t *w_out);

/* ---- the ladder (Steps 0-4 per level; hierarchical partition) ------------ */

typedef struct {
  int32_t level;
  int32_t round;
  int64_t n_nodes;     /* nodes entering the round                       */
  int64_t n_edges;     /* undirected edges entering the round            */
  int64_t n_choosing;  /* nodes that kept an outgoing merge edge         */
  int64_t n_comp;      /* components after the round                     */
  double min_gap;      /* smallest relative gap between a node's best and
                          second-best candidate gain (1 when < 2 cands)  */
  double min_sign;     /* smallest |Delta_best| / (f*ss + lambda*w)      */
} or_round_log;

/* Full ladder on a given graph.
 *   emb      n*d fp32 embeddings
 *   lo,hi,w  ne undirected edges (any order, no self loops, no duplicates)
 *   lambdas  L regularisation strengths; min_size L values or NULL
 *   labels   L*n int32 (out), canonical per level
 *   n_comp   L (out); energy L (out, nullable)
 *   log      capacity log_cap (nullable); *log_len receives the count
 * Returns 0, or a negative code (-6 when max_rounds is reached). */
int or_partition(const float *emb, int64_t n, int32_t d, int64_t ne,
                 const int32_t *lo, const int32_t *hi, const int64_t *w,
                 int32_t L, const double *lambdas, const int64_t *min_size,
                 int32_t max_rounds, int32_t *labels, int64_t *n_comp,
                 double *energy, or_round_log *log, int64_t log_cap,
                 int64_t *log_len);

/* The same ladder with prepare_graph's linking of isolated nodes (reading
 * R7): xyz n*3 fp32 positions, link_k >= 1 neighbours per isolated node. */
int or_partition_linked(const float *emb, const float *xyz, int64_t n,
                        int32_t d, int64_t ne, const int32_t *lo,
                        const int32_t *hi, const int64_t *w, int32_t L,
                        const double *lambdas, const int64_t *min_size,
                        int32_t link_k, int32_t max_rounds, int32_t *labels,
                        int64_t *n_comp, double *energy, or_round_log *log,
                        int64_t log_cap, int64_t *log_len);

/* One linking step (reading R7) on nn nodes and ne edges: size nn, Sx nn*3
 * int64 position sums.  lo_out/hi_out (capacity nn*k) receive the new pairs
 * sorted by (lo, hi).  Returns their count. */
int64_t or_link_isolated(int64_t nn, int64_t ne, const int32_t *lo,
                         const int32_t *hi, const int64_t *size,
                         const int64_t *Sx, int32_t k, int32_t *lo_out,
                         int32_t *hi_out);

/* Eq. gmpp evaluated for a labelling (direct form, fp64).  Means are the
 * fixed-point means ((double)S_C / |C|) * 2^-F.  The cut term runs over the
 * given edges. */
double or_energy(const float *emb, int64_t n, int32_t d, int32_t F,
                 const int32_t *label, int64_t nc, int64_t ne,
                 const int32_t *lo, const int32_t *hi, const int64_t *w,
                 double lambda);

/* Per-component size, mean embedding and centroid for a labelling.
 * Means: ((double)sum_fixed / size) * 2^-F rounded to fp32, F from
 * or_fixed_shift on emb; centroids the same with their own F from xyz. */
int or_component_stats(const int32_t *label, int64_t n, int64_t nc,
                       const float *emb, int32_t d, const float *xyz,
                       int64_t *size, float *mean, float *centroid);

/* ---- grid subsampling (Sec. 4.1; reading R13) ---------------------------- */

/* keep: capacity n, receives the kept point indices in increasing order.
 * Returns the kept count, or -1 (bad argument), -2 (non-finite coordinate),
 * -3 (a cell index reaches 2^21 on some axis). */
int64_t or_grid_subsample(const float *xyz, int64_t n, float h,
                          int32_t *keep);

/* ---- affinity and contrastive loss (Sec. 3.1; readings R14-R17) ---------- */

typedef struct {
  double loss;          /* Eq. loss over the sampled edges              */
  int64_t n_edges;      /* unordered kNN pairs                          */
  int64_t n_intra;      /* pairs with equal classes                     */
  int64_t n_inter;      /* pairs with different classes (all sampled)   */
  int64_t n_intra_kept; /* intra pairs in the sample                    */
} or_loss_out;

/*   emb       n*d fp32        nbr  n*k int32 (-1 = empty slot)
 *   cls       n int32 class   word n*k uint32 random words, one per slot
 *   affinity  n*k fp64 out (nullable): Eq. softmax per slot, 0 when empty
 *   grad      n*d fp64 out (nullable): d loss / d emb
 *   sampled   n*k out (nullable): 1 where the slot owns a sampled edge */
int or_edge_loss(const float *emb, int64_t n, int32_t d, const int32_t *nbr,
                 int32_t k, const int32_t *cls, const uint32_t *word,
                 double tau, double rho, double *affinity, double *grad,
                 uint8_t *sampled, or_loss_out *out);

/* ---- purity and oracle mIoU (Sec. 4.2 "Metrics"; reading R18) ------------- */

typedef struct {
  double miou;       /* mean IoU over the classes present          */
  double purity;     /* points whose class is their superpoint's majority, / n */
  int64_t n_present; /* classes present in the ground truth         */
} or_purity_out;

/* label n in [0, nc), cls n in [0, n_cls); majority nc out (nullable, -1 for
 * an empty component); iou n_cls out (nullable, NaN for absent classes). */
int or_purity(const int32_t *label, int64_t n, int64_t nc, const int32_t *cls,
              int32_t n_cls, int32_t *majority, double *iou,
              or_purity_out *out);

/* ---- point-embedding MLP (stand-in for Sec. 3.1's embedding; R20) ------- */

/* Round to the nearest bfloat16 value (8 significant bits), ties to even. */
double or_round_bf16(double v);

/* out[p] = L3(bf16(relu(L2(bf16(relu(L1(x[p]))))))), L(v) = v W + b with
 * exact dot products.  x n*d_in, w1 d_in*d_hid, w2 d_hid*d_hid,
 * w3 d_hid*d_out as bfloat16 bits (row k = input k); biases fp32; out
 * n*d_out fp64 (the exact last-layer sum). */
int or_embed_mlp(const uint16_t *x, int64_t n, int32_t d_in, int32_t d_hid,
                 int32_t d_out, const uint16_t *w1, const float *b1,
                 const uint16_t *w2, const float *b2, const uint16_t *w3,
                 const float *b3, double *out);

#ifdef __cplusplus
}
#endif
#endif /* EZSP_ORACLE_H */
