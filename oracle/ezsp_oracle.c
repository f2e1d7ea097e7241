/*
 * ezsp_oracle.c -- plain sequential CPU oracle for the EZ-SP partition step
 * (arXiv 2512.00385).  TEST INFRASTRUCTURE ONLY: see ezsp_oracle.h.
 *
 * Written for readability, not speed: one thread, plain loops, qsort.
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared.
 * No FMA contraction is allowed anywhere in this file: every fp32 and fp64
 * operation below is a single correctly rounded IEEE operation.
 */
#include "ezsp_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_EINVAL (-1)
#define OR_ENONFINITE (-2)
#define OR_ERANGE (-3)
#define OR_ENOMEM (-4)
#define OR_ENOTCONV (-6)

/* ======================================================================== */
/* kNN.  Sec. 3.1 builds an undirected graph linking each point to its k     */
/* nearest neighbours; Sec. 4.1 uses w_pq = 1.  Reading R1 fixes the         */
/* arithmetic and the order.                                                 */
/* ======================================================================== */

/* Squared distance between points p and q, IEEE fp32, fixed order:
 * fma(dz, dz, fma(dy, dy, dx * dx)), each fma one rounding (C99 fmaf). */
static float sqdist(const float *xyz, int64_t p, int64_t q) {
  float dx = xyz[3 * q + 0] - xyz[3 * p + 0];
  float dy = xyz[3 * q + 1] - xyz[3 * p + 1];
  float dz = xyz[3 * q + 2] - xyz[3 * p + 2];
  float xx = dx * dx;
  return fmaf(dz, dz, fmaf(dy, dy, xx));
}

/* A sorted list of the k best (d2, index) pairs seen so far. */
typedef struct {
  int32_t k, count;
  float *d2;
  int32_t *idx;
} best_list;

static int pair_less(float da, int32_t ia, float db, int32_t ib) {
  return da < db || (da == db && ia < ib);
}

static void best_consider(best_list *L, float d2, int32_t j) {
  int32_t pos;
  if (L->count == L->k) {
    if (!pair_less(d2, j, L->d2[L->k - 1], L->idx[L->k - 1])) return;
    pos = L->k - 1; /* the current worst falls off */
  } else {
    pos = L->count++;
  }
  while (pos > 0 && pair_less(d2, j, L->d2[pos - 1], L->idx[pos - 1])) {
    L->d2[pos] = L->d2[pos - 1];
    L->idx[pos] = L->idx[pos - 1];
    --pos;
  }
  L->d2[pos] = d2;
  L->idx[pos] = j;
}

static void best_write(const best_list *L, int32_t *nbr, float *d2) {
  for (int32_t j = 0; j < L->k; ++j) {
    if (j < L->count) {
      nbr[j] = L->idx[j];
      if (d2) d2[j] = L->d2[j];
    } else {
      nbr[j] = -1;
      if (d2) d2[j] = INFINITY;
    }
  }
}

static int check_knn_args(const float *xyz, int64_t n, int32_t k) {
  if (!xyz || n < 1 || n > INT32_MAX || k < 1 || k > 64) return OR_EINVAL;
  for (int64_t i = 0; i < 3 * n; ++i)
    if (!isfinite(xyz[i])) return OR_ENONFINITE;
  return OR_OK;
}

int or_knn_one(const float *xyz, int64_t n, int32_t k, int64_t p,
               int32_t *nbr, float *d2) {
  if (!xyz || n < 1 || k < 1 || k > 64 || p < 0 || p >= n || !nbr)
    return OR_EINVAL;
  float bd[64];
  int32_t bi[64];
  best_list L = {k, 0, bd, bi};
  for (int64_t q = 0; q < n; ++q)
    if (q != p) best_consider(&L, sqdist(xyz, p, q), (int32_t)q);
  best_write(&L, nbr, d2);
  return OR_OK;
}

int or_knn_brute(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                 float *d2) {
  int rc = check_knn_args(xyz, n, k);
  if (rc) return rc;
  if (!nbr) return OR_EINVAL;
  for (int64_t p = 0; p < n; ++p)
    or_knn_one(xyz, n, k, p, nbr + p * k, d2 ? d2 + p * k : NULL);
  return OR_OK;
}

/* --- k-d tree --------------------------------------------------------------
 * Each inner node splits its points at the median coordinate of the axis
 * with the largest extent: the left child holds coordinates <= split, the
 * right child coordinates >= split.  A far child is skipped only when the
 * fp32 square of the query-to-plane distance is strictly larger than the
 * current k-th d2.  Because IEEE subtraction, squaring and addition are
 * monotone, that plane term never exceeds the d2 of any point behind the
 * plane, so the skip can never drop a neighbour or a tie. */

typedef struct {
  int64_t begin, end;  /* range in perm                      */
  int64_t left, right; /* children, -1 for a leaf            */
  int32_t axis;
  float split;
} kd_node;

typedef struct {
  const float *xyz;
  int32_t *perm;
  kd_node *nodes;
  int64_t n_nodes, cap;
} kd_tree;

static float kd_coord(const kd_tree *t, int64_t i, int32_t axis) {
  return t->xyz[3 * (int64_t)t->perm[i] + axis];
}

static void kd_swap(int32_t *perm, int64_t a, int64_t b) {
  int32_t tmp = perm[a];
  perm[a] = perm[b];
  perm[b] = tmp;
}

/* Place the element of rank nth of perm[lo, hi) (by coordinate) at nth, with
 * smaller-or-equal coordinates before it and larger-or-equal after it.
 * Three-way partitioning keeps runs of equal coordinates linear. */
static void kd_select(kd_tree *t, int32_t axis, int64_t lo, int64_t hi,
                      int64_t nth) {
  while (hi - lo > 1) {
    float a = kd_coord(t, lo, axis);
    float b = kd_coord(t, lo + (hi - lo) / 2, axis);
    float c = kd_coord(t, hi - 1, axis);
    float pivot = (a < b) ? ((b < c) ? b : ((a < c) ? c : a))
                          : ((a < c) ? a : ((b < c) ? c : b));
    int64_t lt = lo, i = lo, gt = hi;
    while (i < gt) {
      float v = kd_coord(t, i, axis);
      if (v < pivot)
        kd_swap(t->perm, lt++, i++);
      else if (v > pivot)
        kd_swap(t->perm, i, --gt);
      else
        ++i;
    }
    if (nth < lt)
      hi = lt;
    else if (nth >= gt)
      lo = gt;
    else
      return;
  }
}

#define KD_LEAF 8

static int64_t kd_build(kd_tree *t, int64_t begin, int64_t end) {
  int64_t id = t->n_nodes++;
  kd_node *nd = &t->nodes[id];
  nd->begin = begin;
  nd->end = end;
  nd->left = nd->right = -1;
  nd->axis = 0;
  nd->split = 0.0f;
  if (end - begin <= KD_LEAF) return id;
  float lo3[3], hi3[3];
  for (int a = 0; a < 3; ++a) lo3[a] = hi3[a] = kd_coord(t, begin, a);
  for (int64_t i = begin + 1; i < end; ++i)
    for (int a = 0; a < 3; ++a) {
      float v = kd_coord(t, i, a);
      if (v < lo3[a]) lo3[a] = v;
      if (v > hi3[a]) hi3[a] = v;
    }
  int32_t axis = 0;
  double ext = (double)hi3[0] - (double)lo3[0];
  for (int a = 1; a < 3; ++a) {
    double e = (double)hi3[a] - (double)lo3[a];
    if (e > ext) {
      ext = e;
      axis = a;
    }
  }
  if (ext == 0.0) return id; /* all points coincide: keep as one leaf */
  int64_t mid = begin + (end - begin) / 2;
  kd_select(t, axis, begin, end, mid);
  float split = kd_coord(t, mid, axis);
  int64_t l = kd_build(t, begin, mid);
  int64_t r = kd_build(t, mid, end);
  nd = &t->nodes[id]; /* nodes array is preallocated; pointer stays valid */
  nd->axis = axis;
  nd->split = split;
  nd->left = l;
  nd->right = r;
  return id;
}

static void kd_search(const kd_tree *t, int64_t node, int64_t qi,
                      best_list *L) {
  const kd_node *nd = &t->nodes[node];
  if (nd->left < 0) {
    for (int64_t i = nd->begin; i < nd->end; ++i) {
      int64_t j = t->perm[i];
      if (j != qi) best_consider(L, sqdist(t->xyz, qi, j), (int32_t)j);
    }
    return;
  }
  float diff = t->xyz[3 * qi + nd->axis] - nd->split;
  int64_t near = (diff <= 0.0f) ? nd->left : nd->right;
  int64_t far = (diff <= 0.0f) ? nd->right : nd->left;
  kd_search(t, near, qi, L);
  float plane = diff * diff;
  if (L->count < L->k || plane <= L->d2[L->k - 1]) kd_search(t, far, qi, L);
}

int or_knn_kdtree(const float *xyz, int64_t n, int32_t k, int32_t *nbr,
                  float *d2) {
  int rc = check_knn_args(xyz, n, k);
  if (rc) return rc;
  if (!nbr) return OR_EINVAL;
  kd_tree t;
  t.xyz = xyz;
  t.cap = 2 * n + 1;
  t.n_nodes = 0;
  t.perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  t.nodes = (kd_node *)malloc(sizeof(kd_node) * (size_t)t.cap);
  if (!t.perm || !t.nodes) {
    free(t.perm);
    free(t.nodes);
    return OR_ENOMEM;
  }
  for (int64_t i = 0; i < n; ++i) t.perm[i] = (int32_t)i;
  kd_build(&t, 0, n);
  float bd[64];
  int32_t bi[64];
  for (int64_t p = 0; p < n; ++p) {
    best_list L = {k, 0, bd, bi};
    kd_search(&t, 0, p, &L);
    best_write(&L, nbr + p * k, d2 ? d2 + p * k : NULL);
  }
  free(t.perm);
  free(t.nodes);
  return OR_OK;
}

/* ======================================================================== */
/* Graph (reading R2): one undirected edge per unordered kNN pair, w = 1.    */
/* ======================================================================== */

typedef struct {
  int32_t lo, hi;
  int64_t w;
} edge_t;

static int edge_cmp(const void *a, const void *b) {
  const edge_t *x = (const edge_t *)a, *y = (const edge_t *)b;
  if (x->lo != y->lo) return (x->lo < y->lo) ? -1 : 1;
  if (x->hi != y->hi) return (x->hi < y->hi) ? -1 : 1;
  return 0;
}

/* Sort edges by (lo, hi) and add up the weights of equal pairs in place.
 * Returns the number of distinct pairs. */
static int64_t sort_and_merge(edge_t *e, int64_t m) {
  if (m == 0) return 0;
  qsort(e, (size_t)m, sizeof(edge_t), edge_cmp);
  int64_t out = 0;
  for (int64_t i = 1; i < m; ++i) {
    if (e[i].lo == e[out].lo && e[i].hi == e[out].hi)
      e[out].w += e[i].w;
    else
      e[++out] = e[i];
  }
  return out + 1;
}

int64_t or_graph(const int32_t *nbr, int64_t n, int32_t k, int32_t *lo,
                 int32_t *hi, int64_t *w) {
  if (!nbr || n < 1 || k < 1 || !lo || !hi || !w) return OR_EINVAL;
  edge_t *e = (edge_t *)malloc(sizeof(edge_t) * (size_t)(n * k));
  if (!e) return OR_ENOMEM;
  int64_t m = 0;
  for (int64_t p = 0; p < n; ++p)
    for (int32_t j = 0; j < k; ++j) {
      int32_t q = nbr[p * k + j];
      if (q < 0 || q == p) continue;
      e[m].lo = (q < p) ? q : (int32_t)p;
      e[m].hi = (q < p) ? (int32_t)p : q;
      e[m].w = 1;
      ++m;
    }
  if (m > 0) qsort(e, (size_t)m, sizeof(edge_t), edge_cmp);
  int64_t out = 0;
  for (int64_t i = 0; i < m; ++i) {
    if (out > 0 && e[i].lo == lo[out - 1] && e[i].hi == hi[out - 1])
      continue; /* a duplicate pair keeps weight 1 */
    lo[out] = e[i].lo;
    hi[out] = e[i].hi;
    w[out] = 1;
    ++out;
  }
  free(e);
  return out;
}

/* ======================================================================== */
/* Fixed point (reading R3).                                                 */
/* ======================================================================== */

static int32_t ceil_log2_int(int64_t n) { /* smallest c with 2^c >= n */
  int32_t c = 0;
  while (((int64_t)1 << c) < n) ++c;
  return c;
}

static int32_t ceil_log2_pos(double a) { /* a > 0 */
  int e;
  double m = frexp(a, &e); /* a = m * 2^e, m in [0.5, 1) */
  return (m == 0.5) ? e - 1 : e;
}

int or_fixed_shift(const float *emb, int64_t n, int32_t d) {
  if (!emb || n < 1 || d < 1) return OR_EINVAL;
  double A = 0.0;
  for (int64_t i = 0; i < n * d; ++i) {
    if (!isfinite(emb[i])) return OR_ENONFINITE;
    double v = fabs((double)emb[i]);
    if (v > A) A = v;
  }
  int32_t ca = (A > 0.0) ? ceil_log2_pos(A) : 0;
  if (ca < 0) ca = 0;
  int32_t F = 61 - ceil_log2_int(n) - ca;
  if (F > 40) F = 40;
  if (F < 16) return OR_ERANGE;
  return F;
}

void or_quantize(const float *emb, int64_t n, int32_t d, int32_t F,
                 int64_t *S) {
  for (int64_t i = 0; i < n * d; ++i)
    S[i] = (int64_t)llrint(ldexp((double)emb[i], F));
}

/* ======================================================================== */
/* One round: Eq. delta, Steps 1-2, Step 3, Step 4.                          */
/* ======================================================================== */

/* Mean of component v along dimension i: ((double)S / size) * 2^-F. */
static double fixed_mean(const int64_t *S, const int64_t *size, int32_t d,
                         int64_t v, int32_t i, double scale) {
  double q = (double)S[v * d + i] / (double)size[v];
  return q * scale;
}

/* Prop. 1: Delta(P,Q) = lambda*w_PQ - |P||Q|/(|P|+|Q|) * |Y_P - Y_Q|^2. */
static double edge_gain(int32_t a, int32_t b, int64_t w, const int64_t *size,
                        const int64_t *S, int32_t d, double scale,
                        double lambda, double *f_out, double *ss_out) {
  double sa = (double)size[a];
  double sb = (double)size[b];
  double f = (sa * sb) / (sa + sb);
  double ss = 0.0;
  for (int32_t i = 0; i < d; ++i) {
    double diff = fixed_mean(S, size, d, a, i, scale) -
                  fixed_mean(S, size, d, b, i, scale);
    double sq = diff * diff;
    ss = ss + sq;
  }
  if (f_out) *f_out = f;
  if (ss_out) *ss_out = ss;
  double cut = lambda * (double)w;
  double fit = f * ss;
  return cut - fit;
}

void or_gains(int64_t ne, const int32_t *lo, const int32_t *hi,
              const int64_t *w, const int64_t *size, const int64_t *S,
              int32_t d, int32_t F, double lambda, double *delta) {
  double scale = ldexp(1.0, -F);
  for (int64_t e = 0; e < ne; ++e)
    delta[e] = edge_gain(lo[e], hi[e], w[e], size, S, d, scale, lambda, NULL,
                         NULL);
}

/* Reading R5: the order used by conflict removal. */
static int edge_better(int64_t e, int64_t f, const int32_t *lo,
                       const int32_t *hi, const double *delta) {
  if (delta[e] != delta[f]) return delta[e] > delta[f];
  if (lo[e] != lo[f]) return lo[e] < lo[f];
  return hi[e] < hi[f];
}

static int is_candidate(double delta, int64_t size_v, int64_t min_size) {
  return delta > 0.0 || size_v < min_size; /* Step 1 (strict, R6, R10) */
}

void or_select(int64_t nn, int64_t ne, const int32_t *lo, const int32_t *hi,
               const double *delta, const int64_t *size, int64_t min_size,
               int32_t *target) {
  int64_t *best = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nn > 0 ? nn : 1));
  for (int64_t v = 0; v < nn; ++v) best[v] = -1;
  for (int64_t e = 0; e < ne; ++e) {
    int32_t ends[2] = {lo[e], hi[e]};
    for (int s = 0; s < 2; ++s) {
      int32_t v = ends[s];
      if (!is_candidate(delta[e], size[v], min_size)) continue;
      if (best[v] < 0 || edge_better(e, best[v], lo, hi, delta)) best[v] = e;
    }
  }
  for (int64_t v = 0; v < nn; ++v) {
    int64_t e = best[v];
    target[v] = (e < 0) ? -1 : ((lo[e] == v) ? hi[e] : lo[e]);
  }
  free(best);
}

static int32_t uf_find(int32_t *parent, int32_t v) {
  while (parent[v] != v) {
    parent[v] = parent[parent[v]];
    v = parent[v];
  }
  return v;
}

int64_t or_components(int64_t nn, const int32_t *target, int32_t *label) {
  int32_t *parent = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nn > 0 ? nn : 1));
  int32_t *newid = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nn > 0 ? nn : 1));
  for (int64_t v = 0; v < nn; ++v) {
    parent[v] = (int32_t)v;
    newid[v] = -1;
  }
  for (int64_t v = 0; v < nn; ++v) {
    if (target[v] < 0) continue;
    int32_t a = uf_find(parent, (int32_t)v), b = uf_find(parent, target[v]);
    if (a != b) parent[a] = b;
  }
  int64_t nc = 0;
  for (int64_t v = 0; v < nn; ++v) { /* increasing v: smallest member first */
    int32_t r = uf_find(parent, (int32_t)v);
    if (newid[r] < 0) newid[r] = (int32_t)nc++;
    label[v] = newid[r];
  }
  free(parent);
  free(newid);
  return nc;
}

int64_t or_contract(int64_t nn, int64_t ne, const int32_t *lo,
                    const int32_t *hi, const int64_t *w, const int64_t *size,
                    const int64_t *S, int32_t d, const int32_t *label,
                    int64_t nc, int64_t *size_out, int64_t *S_out,
                    int32_t *lo_out, int32_t *hi_out, int64_t *w_out) {
  memset(size_out, 0, sizeof(int64_t) * (size_t)nc);
  memset(S_out, 0, sizeof(int64_t) * (size_t)(nc * d));
  for (int64_t v = 0; v < nn; ++v) {
    int32_t c = label[v];
    size_out[c] += size[v];
    for (int32_t i = 0; i < d; ++i) S_out[c * d + i] += S[v * d + i];
  }
  edge_t *e = (edge_t *)malloc(sizeof(edge_t) * (size_t)(ne > 0 ? ne : 1));
  int64_t m = 0;
  for (int64_t j = 0; j < ne; ++j) {
    int32_t A = label[lo[j]], B = label[hi[j]];
    if (A == B) continue; /* edge inside a merged component */
    e[m].lo = (A < B) ? A : B;
    e[m].hi = (A < B) ? B : A;
    e[m].w = w[j];
    ++m;
  }
  m = sort_and_merge(e, m);
  for (int64_t j = 0; j < m; ++j) {
    lo_out[j] = e[j].lo;
    hi_out[j] = e[j].hi;
    w_out[j] = e[j].w;
  }
  free(e);
  return m;
}

/* ======================================================================== */
/* Energy, Eq. gmpp (direct form; reading R8).                               */
/* ======================================================================== */

double or_energy(const float *emb, int64_t n, int32_t d, int32_t F,
                 const int32_t *label, int64_t nc, int64_t ne,
                 const int32_t *lo, const int32_t *hi, const int64_t *w,
                 double lambda) {
  int64_t *size = (int64_t *)calloc((size_t)(nc > 0 ? nc : 1), sizeof(int64_t));
  int64_t *S = (int64_t *)calloc((size_t)(nc > 0 ? nc * d : 1), sizeof(int64_t));
  for (int64_t p = 0; p < n; ++p) {
    int32_t c = label[p];
    size[c] += 1;
    for (int32_t i = 0; i < d; ++i)
      S[c * d + i] += (int64_t)llrint(ldexp((double)emb[p * d + i], F));
  }
  double scale = ldexp(1.0, -F);
  double fid = 0.0;
  for (int64_t p = 0; p < n; ++p) {
    int32_t c = label[p];
    for (int32_t i = 0; i < d; ++i) {
      double mu = fixed_mean(S, size, d, c, i, scale);
      double r = (double)emb[p * d + i] - mu;
      double sq = r * r;
      fid = fid + sq;
    }
  }
  double cut = 0.0;
  for (int64_t e = 0; e < ne; ++e)
    if (label[lo[e]] != label[hi[e]]) cut = cut + (double)w[e];
  free(size);
  free(S);
  double reg = lambda * cut;
  return fid + reg;
}

/* ======================================================================== */
/* prepare_graph's linking of isolated nodes (App. Alg. A-2).  Reading R7:   */
/* when more than one node is left, every node without an edge gets an edge */
/* of weight 1 to each of its min(k, nn - 1) nearest other nodes, nearest by */
/* the squared distance of their centroids and then by the smaller id; a    */
/* pair linked from both ends is one edge.  Centroids are exact: position   */
/* sums in int64 fixed point, c = (double)Sx / |P| per axis, and the        */
/* squared distance ((dx*dx) + (dy*dy)) + (dz*dz) in fp64.                   */
/* ======================================================================== */

typedef struct {
  double d2;
  int32_t id;
} near_rec;

static int near_cmp(const void *x, const void *y) {
  const near_rec *a = (const near_rec *)x, *b = (const near_rec *)y;
  if (a->d2 != b->d2) return (a->d2 < b->d2) ? -1 : 1;
  return (a->id < b->id) ? -1 : (a->id > b->id);
}

static double centroid_axis(const int64_t *Sx, const int64_t *size, int64_t v,
                            int a) {
  return (double)Sx[3 * v + a] / (double)size[v];
}

int64_t or_link_isolated(int64_t nn, int64_t ne, const int32_t *lo,
                         const int32_t *hi, const int64_t *size,
                         const int64_t *Sx, int32_t k, int32_t *lo_out,
                         int32_t *hi_out) {
  if (nn < 2 || k < 1) return 0;
  char *has = (char *)calloc((size_t)nn, 1);
  near_rec *nr = (near_rec *)malloc(sizeof(near_rec) * (size_t)nn);
  if (!has || !nr) {
    free(has);
    free(nr);
    return OR_ENOMEM;
  }
  for (int64_t e = 0; e < ne; ++e) has[lo[e]] = has[hi[e]] = 1;
  int64_t take = (k < nn - 1) ? k : nn - 1;
  edge_t *L = NULL;
  int64_t m = 0, cap = 0;
  for (int64_t v = 0; v < nn; ++v) {
    if (has[v]) continue;
    int64_t c = 0;
    for (int64_t u = 0; u < nn; ++u) {
      if (u == v) continue;
      double dx = centroid_axis(Sx, size, u, 0) - centroid_axis(Sx, size, v, 0);
      double dy = centroid_axis(Sx, size, u, 1) - centroid_axis(Sx, size, v, 1);
      double dz = centroid_axis(Sx, size, u, 2) - centroid_axis(Sx, size, v, 2);
      double xx = dx * dx, yy = dy * dy, zz = dz * dz;
      double t = xx + yy;
      nr[c].d2 = t + zz;
      nr[c].id = (int32_t)u;
      ++c;
    }
    qsort(nr, (size_t)c, sizeof(near_rec), near_cmp);
    if (m + take > cap) {
      cap = 2 * (m + take);
      edge_t *t = (edge_t *)realloc(L, sizeof(edge_t) * (size_t)cap);
      if (!t) {
        free(L);
        free(has);
        free(nr);
        return OR_ENOMEM;
      }
      L = t;
    }
    for (int64_t i = 0; i < take; ++i) {
      int32_t u = nr[i].id;
      L[m].lo = (u < v) ? u : (int32_t)v;
      L[m].hi = (u < v) ? (int32_t)v : u;
      L[m].w = 1;
      ++m;
    }
  }
  /* one edge per pair; both ends were isolated, so no weight is added */
  if (m > 0) qsort(L, (size_t)m, sizeof(edge_t), edge_cmp);
  int64_t out = 0;
  for (int64_t i = 0; i < m; ++i) {
    if (out > 0 && L[i].lo == lo_out[out - 1] && L[i].hi == hi_out[out - 1])
      continue;
    lo_out[out] = L[i].lo;
    hi_out[out] = L[i].hi;
    ++out;
  }
  free(L);
  free(has);
  free(nr);
  return out;
}

/* ======================================================================== */
/* The ladder: Steps 0-4 until no candidate merge (Step 1), no edge or one   */
/* component (Alg. A-2 early exits); level l+1 runs on level l's result.     */
/* ======================================================================== */

static int grow_edges(int64_t need, size_t *cap, int32_t **a, int32_t **b,
                      int64_t **c, int32_t **a2, int32_t **b2, int64_t **c2,
                      double **dl) {
  if ((size_t)need <= *cap) return OR_OK;
  size_t nc = (size_t)need * 2;
  void *p[7] = {realloc(*a, nc * sizeof(int32_t)), NULL, NULL, NULL, NULL,
                NULL, NULL};
  if (p[0]) *a = (int32_t *)p[0];
  p[1] = realloc(*b, nc * sizeof(int32_t));
  if (p[1]) *b = (int32_t *)p[1];
  p[2] = realloc(*c, nc * sizeof(int64_t));
  if (p[2]) *c = (int64_t *)p[2];
  p[3] = realloc(*a2, nc * sizeof(int32_t));
  if (p[3]) *a2 = (int32_t *)p[3];
  p[4] = realloc(*b2, nc * sizeof(int32_t));
  if (p[4]) *b2 = (int32_t *)p[4];
  p[5] = realloc(*c2, nc * sizeof(int64_t));
  if (p[5]) *c2 = (int64_t *)p[5];
  p[6] = realloc(*dl, nc * sizeof(double));
  if (p[6]) *dl = (double *)p[6];
  for (int i = 0; i < 7; ++i)
    if (!p[i]) return OR_ENOMEM;
  *cap = nc;
  return OR_OK;
}

static int partition_impl(const float *emb, const float *xyz, int64_t n,
                          int32_t d, int64_t ne, const int32_t *lo,
                          const int32_t *hi, const int64_t *w, int32_t L,
                          const double *lambdas, const int64_t *min_size,
                          int32_t link_k, int32_t max_rounds, int32_t *labels,
                          int64_t *n_comp, double *energy, or_round_log *log,
                          int64_t log_cap, int64_t *log_len) {
  if (!emb || n < 1 || n > INT32_MAX || d < 1 || d > 64 || ne < 0 ||
      L < 1 || !lambdas || !labels || !n_comp || (ne > 0 && (!lo || !hi || !w)))
    return OR_EINVAL;
  if (link_k < 0 || (link_k > 0 && !xyz)) return OR_EINVAL;
  for (int32_t l = 0; l < L; ++l)
    if (!isfinite(lambdas[l]) || lambdas[l] < 0.0) return OR_EINVAL;
  for (int64_t e = 0; e < ne; ++e)
    if (lo[e] < 0 || hi[e] < 0 || lo[e] >= n || hi[e] >= n || lo[e] == hi[e] ||
        w[e] <= 0)
      return OR_EINVAL;
  if (max_rounds <= 0) max_rounds = 256;
  int32_t F = or_fixed_shift(emb, n, d);
  if (F < 0) return F;
  int32_t G = 0; /* fixed-point shift of the positions (linking only) */
  if (link_k > 0) {
    G = or_fixed_shift(xyz, n, 3);
    if (G < 0) return G;
  }
  if (log_len) *log_len = 0;

  /* Step 0: every point is its own superpoint, the adjacency is E. */
  int64_t nn = n, me = ne;
  int64_t *size = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  int64_t *S = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n * d));
  int64_t *size2 = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  int64_t *S2 = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n * d));
  size_t ecap = (size_t)(ne > 0 ? ne : 1);
  int32_t *elo = (int32_t *)malloc(sizeof(int32_t) * ecap);
  int32_t *ehi = (int32_t *)malloc(sizeof(int32_t) * ecap);
  int64_t *ew = (int64_t *)malloc(sizeof(int64_t) * ecap);
  int32_t *elo2 = (int32_t *)malloc(sizeof(int32_t) * ecap);
  int32_t *ehi2 = (int32_t *)malloc(sizeof(int32_t) * ecap);
  int64_t *ew2 = (int64_t *)malloc(sizeof(int64_t) * ecap);
  double *delta = (double *)malloc(sizeof(double) * ecap);
  int32_t *target = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  int32_t *label = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  int32_t *plabel = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  int64_t *Sx = NULL;
  int32_t *llo = NULL, *lhi = NULL;
  char *has = NULL;
  if (link_k > 0) {
    Sx = (int64_t *)malloc(sizeof(int64_t) * (size_t)(3 * n));
    llo = (int32_t *)malloc(sizeof(int32_t) * (size_t)n * (size_t)link_k);
    lhi = (int32_t *)malloc(sizeof(int32_t) * (size_t)n * (size_t)link_k);
    has = (char *)malloc((size_t)n);
  }
  int rc = OR_OK;
  if (!size || !S || !size2 || !S2 || !elo || !ehi || !ew || !elo2 || !ehi2 ||
      !ew2 || !delta || !target || !label || !plabel ||
      (link_k > 0 && (!Sx || !llo || !lhi || !has))) {
    rc = OR_ENOMEM;
    goto done;
  }
  for (int64_t p = 0; p < n; ++p) {
    size[p] = 1;
    plabel[p] = (int32_t)p;
  }
  or_quantize(emb, n, d, F, S);
  memcpy(elo, lo, sizeof(int32_t) * (size_t)ne);
  memcpy(ehi, hi, sizeof(int32_t) * (size_t)ne);
  memcpy(ew, w, sizeof(int64_t) * (size_t)ne);
  double scale = ldexp(1.0, -F);

  for (int32_t l = 0; l < L; ++l) {
    double lambda = lambdas[l];
    int64_t smin = min_size ? min_size[l] : 0;
    for (int32_t round = 0;; ++round) {
      if (link_k > 0 && nn > 1) {
        /* prepare_graph: link the nodes that have no edge (reading R7) */
        memset(has, 0, (size_t)nn);
        for (int64_t e = 0; e < me; ++e) has[elo[e]] = has[ehi[e]] = 1;
        int64_t iso = 0;
        for (int64_t v = 0; v < nn; ++v) iso += !has[v];
        if (iso > 0) {
          memset(Sx, 0, sizeof(int64_t) * (size_t)(3 * nn));
          for (int64_t p = 0; p < n; ++p)
            for (int a = 0; a < 3; ++a)
              Sx[3 * (int64_t)plabel[p] + a] +=
                  (int64_t)llrint(ldexp((double)xyz[3 * p + a], G));
          int64_t nl = or_link_isolated(nn, me, elo, ehi, size, Sx, link_k,
                                        llo, lhi);
          if (nl < 0) {
            rc = (int)nl;
            goto done;
          }
          rc = grow_edges(me + nl, &ecap, &elo, &ehi, &ew, &elo2, &ehi2, &ew2,
                          &delta);
          if (rc) goto done;
          for (int64_t i = 0; i < nl; ++i) {
            elo[me + i] = llo[i];
            ehi[me + i] = lhi[i];
            ew[me + i] = 1;
          }
          me += nl;
        }
      }
      if (me == 0) break; /* no edge left: nothing can merge */
      if (round >= max_rounds) {
        rc = OR_ENOTCONV;
        goto done;
      }
      or_gains(me, elo, ehi, ew, size, S, d, F, lambda, delta);
      or_select(nn, me, elo, ehi, delta, size, smin, target);
      int64_t choosing = 0;
      for (int64_t v = 0; v < nn; ++v) choosing += (target[v] >= 0);

      if (log && log_len && *log_len < log_cap) {
        /* decision margins over every choosing node: best vs second-best
         * candidate, and |Delta_best| relative to the magnitude of its two
         * terms.  One pass over the edges keeps each node's two best. */
        int64_t *b1 = (int64_t *)malloc(sizeof(int64_t) * (size_t)nn);
        int64_t *b2 = (int64_t *)malloc(sizeof(int64_t) * (size_t)nn);
        if (!b1 || !b2) {
          free(b1);
          free(b2);
          rc = OR_ENOMEM;
          goto done;
        }
        for (int64_t v = 0; v < nn; ++v) b1[v] = b2[v] = -1;
        for (int64_t e = 0; e < me; ++e) {
          int32_t ends[2] = {elo[e], ehi[e]};
          for (int s2 = 0; s2 < 2; ++s2) {
            int32_t v = ends[s2];
            if (!is_candidate(delta[e], size[v], smin)) continue;
            if (b1[v] < 0 || edge_better(e, b1[v], elo, ehi, delta)) {
              b2[v] = b1[v];
              b1[v] = e;
            } else if (b2[v] < 0 || edge_better(e, b2[v], elo, ehi, delta)) {
              b2[v] = e;
            }
          }
        }
        double min_gap = 1.0, min_sign = 1.0;
        for (int64_t v = 0; v < nn; ++v) {
          if (b1[v] < 0) continue;
          double f, ss;
          double g = edge_gain(elo[b1[v]], ehi[b1[v]], ew[b1[v]], size, S, d,
                               scale, lambda, &f, &ss);
          double mag = f * ss + lambda * (double)ew[b1[v]];
          if (mag > 0.0 && fabs(g) / mag < min_sign) min_sign = fabs(g) / mag;
          if (b2[v] >= 0) {
            double g2 = delta[b2[v]];
            double den = fmax(fabs(g), fabs(g2));
            if (den > 0.0 && (g - g2) / den < min_gap) min_gap = (g - g2) / den;
          }
        }
        free(b1);
        free(b2);
        or_round_log *r = &log[(*log_len)++];
        r->level = l;
        r->round = round;
        r->n_nodes = nn;
        r->n_edges = me;
        r->n_choosing = choosing;
        r->n_comp = nn;
        r->min_gap = min_gap;
        r->min_sign = min_sign;
      }
      if (choosing == 0) break; /* Step 1: no candidate merge */

      int64_t nc = or_components(nn, target, label);
      int64_t m2 = or_contract(nn, me, elo, ehi, ew, size, S, d, label, nc,
                               size2, S2, elo2, ehi2, ew2);
      for (int64_t p = 0; p < n; ++p) plabel[p] = label[plabel[p]];
      if (log && log_len && *log_len > 0 && log[*log_len - 1].level == l &&
          log[*log_len - 1].round == round)
        log[*log_len - 1].n_comp = nc;
      { int64_t *t = size; size = size2; size2 = t; }
      { int64_t *t = S; S = S2; S2 = t; }
      { int32_t *t = elo; elo = elo2; elo2 = t; }
      { int32_t *t = ehi; ehi = ehi2; ehi2 = t; }
      { int64_t *t = ew; ew = ew2; ew2 = t; }
      nn = nc;
      me = m2;
      if (nn == 1) break; /* a single component is left */
    }
    memcpy(labels + (int64_t)l * n, plabel, sizeof(int32_t) * (size_t)n);
    n_comp[l] = nn;
    if (energy)
      energy[l] = or_energy(emb, n, d, F, plabel, nn, ne, lo, hi, w, lambda);
  }
done:
  free(size);
  free(S);
  free(size2);
  free(S2);
  free(elo);
  free(ehi);
  free(ew);
  free(elo2);
  free(ehi2);
  free(ew2);
  free(delta);
  free(target);
  free(label);
  free(plabel);
  free(Sx);
  free(llo);
  free(lhi);
  free(has);
  return rc;
}

int or_partition(const float *emb, int64_t n, int32_t d, int64_t ne,
                 const int32_t *lo, const int32_t *hi, const int64_t *w,
                 int32_t L, const double *lambdas, const int64_t *min_size,
                 int32_t max_rounds, int32_t *labels, int64_t *n_comp,
                 double *energy, or_round_log *log, int64_t log_cap,
                 int64_t *log_len) {
  return partition_impl(emb, NULL, n, d, ne, lo, hi, w, L, lambdas, min_size,
                        0, max_rounds, labels, n_comp, energy, log, log_cap,
                        log_len);
}

int or_partition_linked(const float *emb, const float *xyz, int64_t n,
                        int32_t d, int64_t ne, const int32_t *lo,
                        const int32_t *hi, const int64_t *w, int32_t L,
                        const double *lambdas, const int64_t *min_size,
                        int32_t link_k, int32_t max_rounds, int32_t *labels,
                        int64_t *n_comp, double *energy, or_round_log *log,
                        int64_t log_cap, int64_t *log_len) {
  if (!xyz || link_k < 1) return OR_EINVAL;
  return partition_impl(emb, xyz, n, d, ne, lo, hi, w, L, lambdas, min_size,
                        link_k, max_rounds, labels, n_comp, energy, log,
                        log_cap, log_len);
}

/* ======================================================================== */
/* Per-component statistics for a labelling (component_attributes in        */
/* Alg. A-2; means as in Sec. 3.2).                                          */
/* ======================================================================== */

static int fixed_means(const int32_t *label, int64_t n, int64_t nc,
                       const float *v, int32_t d, const int64_t *size,
                       float *out) {
  int32_t F = or_fixed_shift(v, n, d);
  if (F < 0) return F;
  int64_t *S = (int64_t *)calloc((size_t)(nc * d), sizeof(int64_t));
  if (!S) return OR_ENOMEM;
  for (int64_t p = 0; p < n; ++p)
    for (int32_t i = 0; i < d; ++i)
      S[label[p] * d + i] += (int64_t)llrint(ldexp((double)v[p * d + i], F));
  double scale = ldexp(1.0, -F);
  for (int64_t c = 0; c < nc; ++c)
    for (int32_t i = 0; i < d; ++i) {
      double q = (size[c] > 0) ? (double)S[c * d + i] / (double)size[c] : 0.0;
      out[c * d + i] = (float)(q * scale);
    }
  free(S);
  return OR_OK;
}

int or_component_stats(const int32_t *label, int64_t n, int64_t nc,
                       const float *emb, int32_t d, const float *xyz,
                       int64_t *size, float *mean, float *centroid) {
  if (!label || n < 1 || nc < 1 || !emb || d < 1 || d > 64 || !size || !mean)
    return OR_EINVAL;
  for (int64_t p = 0; p < n; ++p)
    if (label[p] < 0 || label[p] >= nc) return OR_EINVAL;
  memset(size, 0, sizeof(int64_t) * (size_t)nc);
  for (int64_t p = 0; p < n; ++p) size[label[p]] += 1;
  int rc = fixed_means(label, n, nc, emb, d, size, mean);
  if (rc) return rc;
  if (xyz && centroid) rc = fixed_means(label, n, nc, xyz, 3, size, centroid);
  return rc;
}

/* ======================================================================== */
/* Grid subsampling (Sec. 4.1 subsamples every cloud on a regular grid      */
/* before partitioning).  Reading R13: the cell of a point is               */
/* floor((x_i - o_i) / h) per axis in IEEE fp32, o the coordinate-wise      */
/* minimum of the cloud; the point kept for a cell is its smallest index;   */
/* kept indices are returned in increasing order.                           */
/* ======================================================================== */

typedef struct {
  int64_t cell; /* cx * 2^42 + cy * 2^21 + cz */
  int32_t idx;
} cell_rec;

static int cell_rec_cmp(const void *a, const void *b) {
  const cell_rec *x = (const cell_rec *)a, *y = (const cell_rec *)b;
  if (x->cell != y->cell) return (x->cell < y->cell) ? -1 : 1;
  return (x->idx < y->idx) ? -1 : (x->idx > y->idx);
}

static int int32_cmp(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x < y) ? -1 : (x > y);
}

int64_t or_grid_subsample(const float *xyz, int64_t n, float h,
                          int32_t *keep) {
  if (!xyz || !keep || n < 1 || n > INT32_MAX || !(h > 0.0f) || !isfinite(h))
    return OR_EINVAL;
  float o[3];
  for (int a = 0; a < 3; ++a) o[a] = xyz[a];
  for (int64_t p = 0; p < n; ++p)
    for (int a = 0; a < 3; ++a) {
      float v = xyz[3 * p + a];
      if (!isfinite(v)) return OR_ENONFINITE;
      if (v < o[a]) o[a] = v;
    }
  cell_rec *r = (cell_rec *)malloc(sizeof(cell_rec) * (size_t)n);
  if (!r) return OR_ENOMEM;
  for (int64_t p = 0; p < n; ++p) {
    int64_t c[3];
    for (int a = 0; a < 3; ++a) {
      float off = xyz[3 * p + a] - o[a];
      float q = off / h;
      float f = floorf(q);
      if (!(f < 2097152.0f)) { /* 2^21 cells per axis */
        free(r);
        return OR_ERANGE;
      }
      c[a] = (int64_t)f;
    }
    r[p].cell = (c[0] << 42) | (c[1] << 21) | c[2];
    r[p].idx = (int32_t)p;
  }
  qsort(r, (size_t)n, sizeof(cell_rec), cell_rec_cmp);
  int64_t m = 0;
  for (int64_t i = 0; i < n; ++i)
    if (i == 0 || r[i].cell != r[i - 1].cell) keep[m++] = r[i].idx;
  free(r);
  qsort(keep, (size_t)m, sizeof(int32_t), int32_cmp);
  return m;
}

/* ======================================================================== */
/* Affinity and contrastive edge loss (Sec. 3.1, Eq. softmax and Eq. loss). */
/* Readings R14-R17:                                                        */
/*   R14 the edges are the unordered pairs of the kNN relation (as R2); an  */
/*       edge belongs to the smallest slot p*k + j that lists it, and that  */
/*       slot's random word draws it.                                        */
/*   R15 with rho < 1 the sample keeps m = min(n_intra,                      */
/*       floor(rho * n_inter / (1 - rho))) intra edges, those with the       */
/*       smallest (word, slot); rho = 1 keeps them all.  Every inter edge is */
/*       kept.                                                               */
/*   R16 -log(a) = d / tau and -log(1 - a) = -log(-expm1(-d / tau)); the     */
/*       loss is the plain sum over the sampled edges.                       */
/*   R17 the gradient of |e_p - e_q| at e_p = e_q is taken as 0.             */
/* ======================================================================== */

typedef struct {
  int32_t a, b; /* a < b */
  int64_t slot;
} pair_rec;

static int pair_rec_cmp(const void *x, const void *y) {
  const pair_rec *s = (const pair_rec *)x, *t = (const pair_rec *)y;
  if (s->a != t->a) return (s->a < t->a) ? -1 : 1;
  if (s->b != t->b) return (s->b < t->b) ? -1 : 1;
  return (s->slot < t->slot) ? -1 : (s->slot > t->slot);
}

typedef struct {
  uint32_t word;
  int64_t slot;
  int64_t edge;
} draw_rec;

static int draw_rec_cmp(const void *x, const void *y) {
  const draw_rec *s = (const draw_rec *)x, *t = (const draw_rec *)y;
  if (s->word != t->word) return (s->word < t->word) ? -1 : 1;
  return (s->slot < t->slot) ? -1 : (s->slot > t->slot);
}

/* |e_p - e_q| in fp64, squares summed in dimension order. */
static double emb_dist(const float *emb, int32_t d, int64_t p, int64_t q) {
  double s = 0.0;
  for (int32_t i = 0; i < d; ++i) {
    double t = (double)emb[p * d + i] - (double)emb[q * d + i];
    double t2 = t * t;
    s = s + t2;
  }
  return sqrt(s);
}

int or_edge_loss(const float *emb, int64_t n, int32_t d, const int32_t *nbr,
                 int32_t k, const int32_t *cls, const uint32_t *word,
                 double tau, double rho, double *affinity, double *grad,
                 uint8_t *sampled, or_loss_out *out) {
  if (!emb || !nbr || !cls || !word || !out || n < 1 || n > INT32_MAX ||
      d < 1 || d > 1024 || k < 1 || !(tau > 0.0) || !isfinite(tau) ||
      !(rho >= 0.0 && rho <= 1.0))
    return OR_EINVAL;
  int64_t ns = n * k;
  for (int64_t s = 0; s < ns; ++s)
    if (nbr[s] < -1 || nbr[s] >= n) return OR_EINVAL;
  for (int64_t v = 0; v < n * d; ++v)
    if (!isfinite(emb[v])) return OR_ENONFINITE;

  /* Eq. softmax for every slot; an empty slot has affinity 0. */
  if (affinity)
    for (int64_t s = 0; s < ns; ++s) {
      int32_t q = nbr[s];
      affinity[s] = (q < 0) ? 0.0 : exp(-emb_dist(emb, d, s / k, q) / tau);
    }

  /* the unordered pairs and the slot each one belongs to */
  pair_rec *pr = (pair_rec *)malloc(sizeof(pair_rec) * (size_t)(ns > 0 ? ns : 1));
  if (!pr) return OR_ENOMEM;
  int64_t m = 0;
  for (int64_t s = 0; s < ns; ++s) {
    int32_t p = (int32_t)(s / k), q = nbr[s];
    if (q < 0 || q == p) continue;
    pr[m].a = (p < q) ? p : q;
    pr[m].b = (p < q) ? q : p;
    pr[m].slot = s;
    ++m;
  }
  qsort(pr, (size_t)m, sizeof(pair_rec), pair_rec_cmp);
  int64_t ne = 0;
  for (int64_t i = 0; i < m; ++i)
    if (i == 0 || pr[i].a != pr[i - 1].a || pr[i].b != pr[i - 1].b)
      pr[ne++] = pr[i];

  /* R15: the intra-edge sample */
  int64_t n_intra = 0, n_inter = 0;
  for (int64_t e = 0; e < ne; ++e) {
    if (cls[pr[e].a] == cls[pr[e].b]) ++n_intra;
    else ++n_inter;
  }
  int64_t keep_intra = n_intra;
  if (rho < 1.0) {
    double cap = floor(rho * (double)n_inter / (1.0 - rho));
    if (cap < (double)keep_intra) keep_intra = (int64_t)cap;
  }
  char *kept = (char *)calloc((size_t)(ne > 0 ? ne : 1), 1);
  draw_rec *dr = (draw_rec *)malloc(sizeof(draw_rec) * (size_t)(n_intra > 0 ? n_intra : 1));
  if (!kept || !dr) {
    free(pr);
    free(kept);
    free(dr);
    return OR_ENOMEM;
  }
  int64_t ni = 0;
  for (int64_t e = 0; e < ne; ++e) {
    if (cls[pr[e].a] != cls[pr[e].b]) {
      kept[e] = 1;
      continue;
    }
    dr[ni].word = word[pr[e].slot];
    dr[ni].slot = pr[e].slot;
    dr[ni].edge = e;
    ++ni;
  }
  qsort(dr, (size_t)ni, sizeof(draw_rec), draw_rec_cmp);
  for (int64_t i = 0; i < keep_intra; ++i) kept[dr[i].edge] = 1;
  if (sampled) {
    memset(sampled, 0, (size_t)ns);
    for (int64_t e = 0; e < ne; ++e)
      if (kept[e]) sampled[pr[e].slot] = 1;
  }

  /* Eq. loss over the sample, and its gradient */
  if (grad)
    for (int64_t v = 0; v < n * d; ++v) grad[v] = 0.0;
  double loss = 0.0;
  for (int64_t e = 0; e < ne; ++e) {
    if (!kept[e]) continue;
    int32_t p = (int32_t)(pr[e].slot / k), q = nbr[pr[e].slot];
    double dist = emb_dist(emb, d, p, q);
    int intra = cls[p] == cls[q];
    double term, coef;
    if (intra) {
      term = dist / tau;
      coef = (dist > 0.0) ? 1.0 / (tau * dist) : 0.0;
    } else {
      double em = expm1(-dist / tau); /* a - 1 */
      term = -log(-em);
      /* d/d(dist) of -log(1 - exp(-dist/tau)) = -1 / (tau * expm1(dist/tau)) */
      coef = (dist > 0.0) ? -1.0 / (tau * expm1(dist / tau) * dist) : 0.0;
    }
    loss = loss + term;
    if (grad)
      for (int32_t i = 0; i < d; ++i) {
        double diff = (double)emb[(int64_t)p * d + i] - (double)emb[(int64_t)q * d + i];
        double g = coef * diff;
        grad[(int64_t)p * d + i] += g;
        grad[(int64_t)q * d + i] -= g;
      }
  }
  out->loss = loss;
  out->n_edges = ne;
  out->n_intra = n_intra;
  out->n_inter = n_inter;
  out->n_intra_kept = keep_intra;
  free(pr);
  free(kept);
  free(dr);
  return OR_OK;
}

/* ======================================================================== */
/* Partition purity and oracle mIoU (Sec. 4.2 "Metrics": each superpoint    */
/* takes its majority ground-truth label).  Reading R18: a majority tie     */
/* goes to the smallest class; IoU_c = TP / (|gt = c| + |pred = c| - TP)    */
/* over the classes present in the ground truth, averaged in class order;   */
/* purity = sum TP / n.                                                     */
/* ======================================================================== */

typedef struct {
  int32_t comp, cls;
} cc_rec;

static int cc_rec_cmp(const void *x, const void *y) {
  const cc_rec *s = (const cc_rec *)x, *t = (const cc_rec *)y;
  if (s->comp != t->comp) return (s->comp < t->comp) ? -1 : 1;
  return (s->cls < t->cls) ? -1 : (s->cls > t->cls);
}

int or_purity(const int32_t *label, int64_t n, int64_t nc, const int32_t *cls,
              int32_t n_cls, int32_t *majority, double *iou,
              or_purity_out *out) {
  if (!label || !cls || !out || n < 1 || n > INT32_MAX || nc < 1 ||
      nc > INT32_MAX || n_cls < 1)
    return OR_EINVAL;
  for (int64_t p = 0; p < n; ++p)
    if (label[p] < 0 || label[p] >= nc || cls[p] < 0 || cls[p] >= n_cls)
      return OR_EINVAL;
  cc_rec *r = (cc_rec *)malloc(sizeof(cc_rec) * (size_t)n);
  int32_t *maj = (int32_t *)malloc(sizeof(int32_t) * (size_t)nc);
  int64_t *best = (int64_t *)calloc((size_t)nc, sizeof(int64_t));
  int64_t *tp = (int64_t *)calloc((size_t)n_cls, sizeof(int64_t));
  int64_t *ngt = (int64_t *)calloc((size_t)n_cls, sizeof(int64_t));
  int64_t *npred = (int64_t *)calloc((size_t)n_cls, sizeof(int64_t));
  if (!r || !maj || !best || !tp || !ngt || !npred) {
    free(r); free(maj); free(best); free(tp); free(ngt); free(npred);
    return OR_ENOMEM;
  }
  for (int64_t p = 0; p < n; ++p) {
    r[p].comp = label[p];
    r[p].cls = cls[p];
  }
  qsort(r, (size_t)n, sizeof(cc_rec), cc_rec_cmp);
  for (int64_t c = 0; c < nc; ++c) maj[c] = -1;
  /* runs of equal (comp, cls), classes ascending inside a component: a
   * strictly larger count replaces the majority, so ties keep the smaller */
  for (int64_t i = 0; i < n;) {
    int64_t j = i;
    while (j < n && r[j].comp == r[i].comp && r[j].cls == r[i].cls) ++j;
    int64_t cnt = j - i;
    if (cnt > best[r[i].comp]) {
      best[r[i].comp] = cnt;
      maj[r[i].comp] = r[i].cls;
    }
    i = j;
  }
  for (int64_t p = 0; p < n; ++p) {
    int32_t g = cls[p], y = maj[label[p]];
    ngt[g] += 1;
    npred[y] += 1;
    if (g == y) tp[g] += 1;
  }
  double sum = 0.0;
  int64_t present = 0, tp_all = 0;
  for (int32_t c = 0; c < n_cls; ++c) {
    tp_all += tp[c];
    double v = NAN;
    if (ngt[c] > 0) {
      v = (double)tp[c] / (double)(ngt[c] + npred[c] - tp[c]);
      sum = sum + v;
      ++present;
    }
    if (iou) iou[c] = v;
  }
  out->miou = sum / (double)present;
  out->purity = (double)tp_all / (double)n;
  out->n_present = present;
  if (majority) memcpy(majority, maj, sizeof(int32_t) * (size_t)nc);
  free(r); free(maj); free(best); free(tp); free(ngt); free(npred);
  return OR_OK;
}

/* ======================================================================== */
/* Point-embedding MLP, a random-weight stand-in for the point embedding     */
/* network of Sec. 3.1 on the LiDAR-sweep workload.  Reading R20: inputs,    */
/* weights and hidden activations are bfloat16 (round to nearest even);     */
/* each layer is an exact dot product plus an fp32 bias, ReLU after the two  */
/* hidden layers, the hidden values rounded to bfloat16 before the next     */
/* layer; the output is the last layer's sum rounded to fp32.               */
/* ======================================================================== */

/* Round to the nearest value with 8 significant bits, ties to even. */
double or_round_bf16(double v) {
  if (v == 0.0 || !isfinite(v)) return v;
  int e;
  double m = frexp(v, &e); /* v = m * 2^e, 0.5 <= |m| < 1 */
  double r = nearbyint(ldexp(m, 8)); /* default mode: ties to even */
  return ldexp(r, e - 8);
}

static double bf16_bits_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

int or_embed_mlp(const uint16_t *x, int64_t n, int32_t d_in, int32_t d_hid,
                 int32_t d_out, const uint16_t *w1, const float *b1,
                 const uint16_t *w2, const float *b2, const uint16_t *w3,
                 const float *b3, double *out) {
  if (!x || !w1 || !b1 || !w2 || !b2 || !w3 || !b3 || !out || n < 1 ||
      d_in < 1 || d_hid < 1 || d_out < 1)
    return OR_EINVAL;
  double *h1 = (double *)malloc(sizeof(double) * (size_t)d_hid);
  double *h2 = (double *)malloc(sizeof(double) * (size_t)d_hid);
  if (!h1 || !h2) {
    free(h1);
    free(h2);
    return OR_ENOMEM;
  }
  for (int64_t p = 0; p < n; ++p) {
    /* layer 1: W1 is d_in x d_hid, row k = input k */
    for (int32_t j = 0; j < d_hid; ++j) {
      double s = 0.0;
      for (int32_t k = 0; k < d_in; ++k)
        s += bf16_bits_to_double(x[p * d_in + k]) *
             bf16_bits_to_double(w1[(int64_t)k * d_hid + j]);
      s += (double)b1[j];
      h1[j] = or_round_bf16(s > 0.0 ? s : 0.0);
    }
    for (int32_t j = 0; j < d_hid; ++j) {
      double s = 0.0;
      for (int32_t k = 0; k < d_hid; ++k)
        s += h1[k] * bf16_bits_to_double(w2[(int64_t)k * d_hid + j]);
      s += (double)b2[j];
      h2[j] = or_round_bf16(s > 0.0 ? s : 0.0);
    }
    for (int32_t j = 0; j < d_out; ++j) {
      double s = 0.0;
      for (int32_t k = 0; k < d_hid; ++k)
        s += h2[k] * bf16_bits_to_double(w3[(int64_t)k * d_out + j]);
      s += (double)b3[j];
      out[p * d_out + j] = s;
    }
  }
  free(h1);
  free(h2);
  return OR_OK;
}
