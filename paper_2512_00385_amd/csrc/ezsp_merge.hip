// ezsp_merge.hip -- the merge ladder of EZ-SP (arXiv 2512.00385, Sec. 3.2):
// kNN graph build, then rounds of Steps 1-4 on the superpoint adjacency
// until no candidate merge is left, for every regularisation strength of the
// ladder (hierarchical partition).
//
// Representation.  Nodes of round r are the superpoints of round r, stored
// in an internal order (Morton order of their first point when the graph came
// from xyz) that keeps neighbours close in memory.  The adjacency is a CSR
// holding every undirected edge in both directions: row v lists (u, w_vu).
// Each node keeps its size |P|, the exact int64 fixed-point sum of its
// embeddings, its mean in fp64 and `minpt`, the smallest original point
// index of its points; ordering nodes by minpt is the same as ordering them
// by their canonical number, so ties and output labels use minpt and the
// internal order never shows in the results.
//
// One round (all on the device, one host readback at the end):
//   select   Steps 1-2: every node scans its row, evaluates Prop. 1's gain,
//            keeps the best candidate (largest gain, ties to smaller minpt)
//   hook     merge graph of chosen edges; every cycle of it is a mutual pair
//            (each choice is at least as good as the choice it follows), the
//            lower id becomes the root
//   jump     pointer jumping to the roots = weakly connected components
//            (Step 3, what App. Alg. A-1 computes)
//   relabel  roots numbered by a scan
//   stats    Step 4: sizes, int64 sums, minpt, row capacity per component
//   contract Step 4: per-component open-addressing tables collect the
//            relabelled edges and add up the weights of parallel edges; a
//            scan compacts them into the next CSR
#include <math.h>

#include "ezsp_internal.h"

namespace ezsp {

constexpr uint64_t kEmpty = ~0ull;
constexpr int kJumpCap = 1 << 16;
constexpr int kLongRow = 64;  // rows longer than this go to k_select_long
constexpr int kLongGrid = 1024;

// ---------------------------------------------------------------------------
// small kernels
// ---------------------------------------------------------------------------
__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ __launch_bounds__(256) void k_gather_rows(const float *emb,
                                                     const int32_t *perm,
                                                     int32_t n, int32_t d,
                                                     float *out) {
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t >= (int64_t)n * d) return;
  const int64_t i = t / d;
  const int32_t c = (int32_t)(t - i * d);
  out[t] = emb[(int64_t)perm[i] * d + c];
}

// ---------------------------------------------------------------------------
// graph build: the union of the kNN relations, one undirected edge of weight
// 1 per pair (Sec. 3.1, Sec. 4.1; duplicates and self loops removed as in
// App. Alg. A-2, prepare_graph), stored in both directions
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool row_has(const int32_t *nbr, int32_t k,
                                        int32_t j, int32_t x) {
  const int32_t *r = nbr + (int64_t)j * k;
  for (int32_t s = 0; s < k; ++s)
    if (r[s] == x) return true;
  return false;
}

// Entry t of row i is a forward edge when it is a valid id, not i itself and
// not a repeat of an earlier entry of the row.
__device__ __forceinline__ bool fwd_entry(const int32_t *row, int32_t t,
                                          int32_t i, int32_t n, Ctl *ctl) {
  const int32_t j = row[t];
  if (j == -1 || j == i) return false;
  if (j < -1 || j >= n) {
    raise_err(ctl, kErrBadIndex);
    return false;
  }
  for (int32_t s = 0; s < t; ++s)
    if (row[s] == j) return false;
  return true;
}

__global__ __launch_bounds__(256) void k_graph_count(const int32_t *nbr,
                                                     int32_t n, int32_t k,
                                                     int32_t *fwd, int32_t *rev,
                                                     Ctl *ctl) {
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const int32_t *row = nbr + (int64_t)i * k;
  int32_t c = 0;
  for (int32_t t = 0; t < k; ++t) {
    if (!fwd_entry(row, t, i, n, ctl)) continue;
    const int32_t j = row[t];
    ++c;
    if (!row_has(nbr, k, j, i)) atomicAdd(&rev[j], 1);
  }
  fwd[i] = c;
}

struct ScanDeg {
  const int32_t *fwd, *rev;
  int32_t *out;
  int32_t n;
  __device__ int32_t value(int32_t i) const {
    return i < n ? fwd[i] + rev[i] : 0;
  }
  __device__ void emit(int32_t i, int32_t excl, int32_t) const {
    if (i <= n) out[i] = excl;
  }
};

__global__ __launch_bounds__(256) void k_graph_fill(
    const int32_t *nbr, int32_t n, int32_t k, const int32_t *fwd,
    const int32_t *rp, int32_t *cursor, int32_t *col, int32_t *w, int32_t *src,
    Ctl *ctl) {
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const int32_t *row = nbr + (int64_t)i * k;
  const int32_t base = rp[i];
  int32_t c = 0;
  for (int32_t t = 0; t < k; ++t) {
    if (!fwd_entry(row, t, i, n, ctl)) continue;
    const int32_t j = row[t];
    col[base + c] = j;
    w[base + c] = 1;
    src[base + c] = i;
    ++c;
    if (!row_has(nbr, k, j, i)) {
      const int32_t pos = rp[j] + fwd[j] + atomicAdd(&cursor[j], 1);
      if (pos < rp[j + 1]) {
        col[pos] = i;
        w[pos] = 1;
        src[pos] = j;
      } else {
        raise_err(ctl, kErrInternal);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// node state of a round
// ---------------------------------------------------------------------------
struct NodeIn {
  const int32_t *size;   // |P|            (null in the first round)
  const int64_t *S;      // fixed-point sums (null in the first round)
  const double *mu;      // fp64 means      (null in the first round)
  const int32_t *minpt;  // smallest point  (null in the first round)
  const float *emb;      // point embeddings, internal order (first round)
  const int32_t *perm;   // internal -> original point, nullable (identity)
};

// Mean of node v along dimension i: ((double)S / |P|) * 2^-F.  In the first
// round every node is one point, S = rint(e * 2^F) and |P| = 1, which is the
// same value as rint(e * 2^F) * 2^-F computed in double.
template <bool FIRST>
__device__ __forceinline__ double node_mu(const NodeIn &s, int32_t v,
                                          int32_t i, int32_t d, double sF,
                                          double sIF) {
  if (FIRST) {
    const double q = rint((double)s.emb[(int64_t)v * d + i] * sF);
    return q * sIF;
  }
  return s.mu[(int64_t)v * d + i];
}

template <bool FIRST>
__device__ __forceinline__ int32_t node_size(const NodeIn &s, int32_t v) {
  return FIRST ? 1 : s.size[v];
}

template <bool FIRST>
__device__ __forceinline__ int32_t node_minpt(const NodeIn &s, int32_t v) {
  if (FIRST) return s.perm ? s.perm[v] : v;
  return s.minpt[v];
}

__global__ void k_round_init(Ctl *ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctl->any_choice = 0;
    ctl->n_next = 0;
    ctl->e_next = 0;
    ctl->slots = 0;
    ctl->n_long = 0;
  }
}

// Steps 1-2.  Prop. 1 (Eq. delta):
//   Delta(P,Q) = lambda * w_PQ - |P||Q| / (|P|+|Q|) * |Y_P - Y_Q|^2,
// evaluated in fp64 in a fixed order (no contraction): f = (sP*sQ)/(sP+sQ),
// ss = sum_i (mu_P,i - mu_Q,i)^2 left to right, Delta = lambda*w - f*ss.
// A directed edge P -> Q is a candidate when Delta > 0 or |P| < s_min; P
// keeps its largest candidate, ties to the neighbour with smaller minpt.
template <bool FIRST>
__global__ __launch_bounds__(256) void k_select(
    int32_t nn, const int32_t *__restrict__ rp, const int32_t *__restrict__ col,
    const int32_t *__restrict__ w, NodeIn s, int32_t d, double lambda,
    int64_t smin, int32_t *__restrict__ target, int32_t *__restrict__ long_rows,
    Ctl *ctl) {
  const int32_t v = xcd_tid();
  if (v >= nn) return;
  const int32_t e0 = rp[v], e1 = rp[v + 1];
  if (e1 - e0 > kLongRow) {  // a whole block takes this row later
    const int32_t slot = atomicAdd(&ctl->n_long, 1);
    long_rows[slot] = v;
    return;
  }
  const int F = ctl->F;
  const double sF = ldexp(1.0, F), sIF = ldexp(1.0, -F);
  const int32_t sv = node_size<FIRST>(s, v);
  const double dsv = (double)sv;
  const bool small = (int64_t)sv < smin;
  bool has = false;
  double bD = 0.0;
  int32_t bMP = 0, bU = -1;
  for (int32_t e = e0; e < e1; ++e) {
    const int32_t u = col[e];
    if ((uint32_t)u >= (uint32_t)nn) {
      raise_err(ctl, kErrInternal);
      continue;
    }
    const double dsu = (double)node_size<FIRST>(s, u);
    const double num = dsv * dsu;
    const double den = dsv + dsu;
    const double f = num / den;
    double ss = 0.0;
    for (int32_t i = 0; i < d; ++i) {
      const double diff = node_mu<FIRST>(s, v, i, d, sF, sIF) -
                          node_mu<FIRST>(s, u, i, d, sF, sIF);
      const double sq = diff * diff;
      ss = ss + sq;
    }
    const double cut = lambda * (double)w[e];
    const double fit = f * ss;
    const double g = cut - fit;
    if (g > 0.0 || small) {
      const int32_t mp = node_minpt<FIRST>(s, u);
      if (!has || g > bD || (g == bD && mp < bMP)) {
        has = true;
        bD = g;
        bMP = mp;
        bU = u;
      }
    }
  }
  target[v] = has ? bU : -1;
  if (__ballot(has) && (threadIdx.x & (kWave - 1)) == 0) ctl->any_choice = 1;
}

// Steps 1-2 for rows longer than kLongRow: one block per row, threads stride
// over the row and the best candidate is found by a block reduction under
// the same order (larger gain, then smaller minpt).
struct Best {
  double g;
  int32_t mp, u;  // u < 0: no candidate
};

__device__ __forceinline__ bool best_before(const Best &a, const Best &b) {
  if (a.u < 0) return false;
  if (b.u < 0) return true;
  return a.g > b.g || (a.g == b.g && a.mp < b.mp);
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_select_long(
    const int32_t *__restrict__ rp, const int32_t *__restrict__ col,
    const int32_t *__restrict__ w, NodeIn s, int32_t d, double lambda,
    int64_t smin, int32_t nn, int32_t *__restrict__ target,
    const int32_t *__restrict__ long_rows, Ctl *ctl) {
  __shared__ double sg[256 / kWave];
  __shared__ int32_t smp[256 / kWave], su[256 / kWave];
  const int32_t n_long = ctl->n_long;
  const int F = ctl->F;
  const double sF = ldexp(1.0, F), sIF = ldexp(1.0, -F);
  for (int32_t li = blockIdx.x; li < n_long; li += gridDim.x) {
    const int32_t v = long_rows[li];
    if ((uint32_t)v >= (uint32_t)nn) {
      raise_err(ctl, kErrInternal);
      continue;
    }
    const int32_t sv = node_size<FIRST>(s, v);
    const double dsv = (double)sv;
    const bool small = (int64_t)sv < smin;
    Best b{0.0, 0, -1};
    for (int32_t e = rp[v] + threadIdx.x; e < rp[v + 1]; e += blockDim.x) {
      const int32_t u = col[e];
      if ((uint32_t)u >= (uint32_t)nn) {
        raise_err(ctl, kErrInternal);
        continue;
      }
      const double dsu = (double)node_size<FIRST>(s, u);
      const double num = dsv * dsu;
      const double den = dsv + dsu;
      const double f = num / den;
      double ss = 0.0;
      for (int32_t i = 0; i < d; ++i) {
        const double diff = node_mu<FIRST>(s, v, i, d, sF, sIF) -
                            node_mu<FIRST>(s, u, i, d, sF, sIF);
        const double sq = diff * diff;
        ss = ss + sq;
      }
      const double cut = lambda * (double)w[e];
      const double fit = f * ss;
      const double g = cut - fit;
      if (g > 0.0 || small) {
        const Best c{g, node_minpt<FIRST>(s, u), u};
        if (best_before(c, b)) b = c;
      }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      Best o;
      o.g = __shfl_xor(b.g, off, kWave);
      o.mp = __shfl_xor(b.mp, off, kWave);
      o.u = __shfl_xor(b.u, off, kWave);
      if (best_before(o, b)) b = o;
    }
    const int wid = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
      sg[wid] = b.g;
      smp[wid] = b.mp;
      su[wid] = b.u;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      Best r{sg[0], smp[0], su[0]};
      for (int q = 1; q < 256 / kWave; ++q) {
        const Best o{sg[q], smp[q], su[q]};
        if (best_before(o, r)) r = o;
      }
      target[v] = r.u;
      if (r.u >= 0) ctl->any_choice = 1;
    }
    __syncthreads();
  }
}

// Merge graph -> forest: a node points to its choice, except the lower end
// of a mutual pair, which becomes a root.  Always writes every parent.
__global__ __launch_bounds__(256) void k_hook(int32_t nn, const int32_t *target,
                                              int32_t *parent, Ctl *ctl) {
  const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= nn) return;
  const int32_t t = target[v];
  int32_t p = v;
  if (t >= 0) {
    if (t >= nn) {
      raise_err(ctl, kErrInternal);
    } else {
      const int32_t tt = target[t];
      p = (tt == v && v < t) ? v : t;
    }
  }
  parent[v] = p;
}

// Pointer jumping: every step moves strictly up the forest, so the loop ends
// at the root; concurrent updates by other threads only shorten it.
__global__ __launch_bounds__(256) void k_jump(int32_t nn, int32_t *parent,
                                              Ctl *ctl) {
  const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= nn) return;
  int32_t p = parent[v];
  int it = 0;
  for (; it < kJumpCap; ++it) {
    if ((uint32_t)p >= (uint32_t)nn) {
      raise_err(ctl, kErrInternal);
      p = v;
      break;
    }
    const int32_t pp = __atomic_load_n(&parent[p], __ATOMIC_RELAXED);
    if (pp == p) break;
    p = pp;
  }
  if (it == kJumpCap) raise_err(ctl, kErrJump);
  __atomic_store_n(&parent[v], p, __ATOMIC_RELAXED);
}

struct ScanRoots {
  const int32_t *parent;
  int32_t *newid;
  int32_t nn;
  __device__ int32_t value(int32_t v) const {
    return (v < nn && parent[v] == v) ? 1 : 0;
  }
  __device__ void emit(int32_t v, int32_t excl, int32_t val) const {
    if (val) newid[v] = excl;
  }
};

__global__ __launch_bounds__(256) void k_assign(int32_t nn,
                                                const int32_t *parent,
                                                const int32_t *newid,
                                                int32_t *L, Ctl *ctl) {
  const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= nn) return;
  const int32_t r = parent[v];
  int32_t c = 0;
  if ((uint32_t)r < (uint32_t)nn) {
    c = newid[r];
  } else {
    raise_err(ctl, kErrInternal);
  }
  L[v] = c;
}

// Step 4 statistics.  acc arrays are the next round's node state.
__global__ __launch_bounds__(256) void k_zero_acc(int32_t bound, int32_t d,
                                                  const Ctl *ctl, int32_t *size,
                                                  int64_t *S, int32_t *minpt,
                                                  int32_t *cap, int32_t *ndeg) {
  if (!ctl->any_choice) return;
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= bound || c >= ctl->n_next) return;
  size[c] = 0;
  minpt[c] = INT32_MAX;
  cap[c] = 0;
  ndeg[c] = 0;
  for (int32_t i = 0; i < d; ++i) S[(int64_t)c * d + i] = 0;
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_stats_add(
    int32_t nn, const int32_t *__restrict__ L, const int32_t *__restrict__ rp,
    NodeIn s, int32_t d, Ctl *ctl, int32_t *size, int64_t *S, int32_t *minpt,
    int32_t *cap) {
  if (!ctl->any_choice) return;
  const int32_t v = xcd_tid();
  if (v >= nn) return;
  const int32_t c = L[v];
  if ((uint32_t)c >= (uint32_t)ctl->n_next) {
    raise_err(ctl, kErrInternal);
    return;
  }
  atomicAdd(&size[c], node_size<FIRST>(s, v));
  atomicMin(&minpt[c], node_minpt<FIRST>(s, v));
  atomicAdd(&cap[c], rp[v + 1] - rp[v]);
  const double sF = ldexp(1.0, ctl->F);
  for (int32_t i = 0; i < d; ++i) {
    int64_t q;
    if (FIRST)
      q = (int64_t)rint((double)s.emb[(int64_t)v * d + i] * sF);
    else
      q = s.S[(int64_t)v * d + i];
    atomicAdd(reinterpret_cast<unsigned long long *>(&S[(int64_t)c * d + i]),
              (unsigned long long)q);
  }
}

__global__ __launch_bounds__(256) void k_stats_final(int32_t bound, int32_t d,
                                                     const Ctl *ctl,
                                                     const int32_t *size,
                                                     const int64_t *S,
                                                     double *mu) {
  if (!ctl->any_choice) return;
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t c = t / d;
  if (c >= bound || c >= ctl->n_next) return;
  const double sIF = ldexp(1.0, -ctl->F);
  const double q = (double)S[t] / (double)size[c];
  mu[t] = q * sIF;
}

// Contraction into per-component open-addressing tables.  Component A owns
// slots [toff[A], toff[A] + cap[A]) where cap[A] is the summed degree of its
// members, an upper bound on its distinct neighbours.
__global__ __launch_bounds__(256) void k_table_clear(int32_t bound,
                                                     const Ctl *ctl,
                                                     uint64_t *keys,
                                                     int32_t *tw) {
  if (!ctl->any_choice) return;
  const int32_t s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= bound || s >= ctl->slots) return;
  keys[s] = kEmpty;
  tw[s] = 0;
}

__global__ __launch_bounds__(256) void k_insert(
    int32_t ed, const int32_t *__restrict__ src, const int32_t *__restrict__ col,
    const int32_t *__restrict__ w, const int32_t *__restrict__ L,
    const int32_t *__restrict__ toff, const int32_t *__restrict__ cap,
    uint64_t *keys, int32_t *tw, int32_t *ndeg, int32_t nn, int32_t table_cap,
    Ctl *ctl) {
  if (!ctl->any_choice) return;
  const int32_t e = xcd_tid();
  if (e >= ed) return;
  const int32_t a = src[e], b = col[e];
  if ((uint32_t)a >= (uint32_t)nn || (uint32_t)b >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
  const int32_t A = L[a];
  const int32_t B = L[b];
  if (A == B) return;  // edge inside a merged component
  const int32_t nc = ctl->n_next;
  if ((uint32_t)A >= (uint32_t)nc || (uint32_t)B >= (uint32_t)nc) {
    raise_err(ctl, kErrInternal);
    return;
  }
  const int32_t c = cap[A];
  const int32_t base = toff[A];
  if (c <= 0 || base < 0 || base + c > ctl->slots || base + c > table_cap) {
    raise_err(ctl, kErrInternal);
    return;
  }
  const uint64_t key = ((uint64_t)(uint32_t)A << 32) | (uint32_t)B;
  uint32_t h = ((uint32_t)B * 2654435761u) % (uint32_t)c;
  for (int32_t probe = 0; probe < c; ++probe) {
    unsigned long long *slot =
        reinterpret_cast<unsigned long long *>(&keys[base + h]);
    const unsigned long long old = atomicCAS(slot, kEmpty, key);
    if (old == kEmpty) {
      atomicAdd(&ndeg[A], 1);
      atomicAdd(&tw[base + h], w[e]);
      return;
    }
    if (old == key) {
      atomicAdd(&tw[base + h], w[e]);
      return;
    }
    h = (h + 1 == (uint32_t)c) ? 0u : h + 1;
  }
  raise_err(ctl, kErrInternal);
}

struct ScanCompact {
  const uint64_t *keys;
  const int32_t *tw;
  const int32_t *slots;
  int32_t *col, *w, *src;
  int32_t cap;  // capacity of col/w/src
  __device__ int32_t value(int32_t s) const {
    return (s < *slots && keys[s] != kEmpty) ? 1 : 0;
  }
  __device__ void emit(int32_t s, int32_t excl, int32_t val) const {
    if (!val || excl >= cap) return;
    const uint64_t k = keys[s];
    col[excl] = (int32_t)(uint32_t)(k & 0xffffffffull);
    src[excl] = (int32_t)(k >> 32);
    w[excl] = tw[s];
  }
};

// point -> current node map, composed every merging round
template <bool FIRST>
__global__ __launch_bounds__(256) void k_compose(int32_t n, int32_t nn,
                                                 int32_t *M, const int32_t *L,
                                                 Ctl *ctl) {
  if (!ctl->any_choice) return;
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const int32_t c = FIRST ? i : M[i];
  if ((uint32_t)c >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
  M[i] = L[c];
}

// ---------------------------------------------------------------------------
// level output: canonical labels (numbered by smallest point index) and the
// energy of Eq. gmpp
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_mark(int32_t nc, const int32_t *minpt,
                                              int32_t *mark, int32_t n,
                                              Ctl *ctl) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nc) return;
  const int32_t m = minpt[c];
  if ((uint32_t)m >= (uint32_t)n) {
    raise_err(ctl, kErrInternal);
    return;
  }
  mark[m] = 1;
}

__global__ __launch_bounds__(256) void k_labels(int32_t n, int32_t nc,
                                                const int32_t *inv,
                                                const int32_t *M,
                                                const int32_t *minpt,
                                                const int32_t *rank,
                                                int32_t *out, Ctl *ctl) {
  const int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t i = inv ? inv[p] : p;
  const int32_t c = ((uint32_t)i < (uint32_t)n) ? M[i] : -1;
  if ((uint32_t)c >= (uint32_t)nc) {
    raise_err(ctl, kErrInternal);
    out[p] = -1;
    return;
  }
  const int32_t m = minpt[c];
  if ((uint32_t)m >= (uint32_t)n) {
    raise_err(ctl, kErrInternal);
    out[p] = -1;
    return;
  }
  out[p] = rank[m];
}

__global__ __launch_bounds__(256) void k_iota(int32_t n, int32_t *out) {
  const int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < n) out[p] = p;
}

constexpr int kEnergyBlocks = 1024;

// Fidelity term sum_p |e_p - Y_P(p)|^2 in the direct form; per-block partial
// sums in a fixed order, so the result is reproducible.
template <bool FIRST>
__global__ __launch_bounds__(256) void k_energy_fid(int32_t n, int32_t d,
                                                    int32_t nc,
                                                    const float *emb,
                                                    const int32_t *M,
                                                    const double *mu,
                                                    const Ctl *ctl,
                                                    double *partial) {
  __shared__ double ws[256 / kWave];
  const double sF = ldexp(1.0, ctl->F), sIF = ldexp(1.0, -ctl->F);
  double acc = 0.0;
  const int64_t total = (int64_t)n * d;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / d;
    const int32_t j = (int32_t)(t - i * d);
    const double e = (double)emb[t];
    double m;
    if (FIRST) {
      m = rint(e * sF) * sIF;
    } else {
      const int32_t c = M[i];
      m = ((uint32_t)c < (uint32_t)nc) ? mu[(int64_t)c * d + j] : 0.0;
    }
    const double r = e - m;
    const double sq = r * r;
    acc = acc + sq;
  }
  for (int off = kWave / 2; off > 0; off >>= 1)
    acc += __shfl_xor(acc, off, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0) ws[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double b = 0.0;
    for (int q = 0; q < 256 / kWave; ++q) b += ws[q];
    partial[blockIdx.x] = b;
  }
}

__global__ void k_energy_sum(const double *partial, int32_t nb, Ctl *ctl) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  for (int32_t b = 0; b < nb; ++b) s += partial[b];
  ctl->fid_total = s;
}

__global__ __launch_bounds__(256) void k_weight_sum(int32_t ed,
                                                    const int32_t *w,
                                                    Ctl *ctl) {
  long long acc = 0;
  for (int32_t e = blockIdx.x * blockDim.x + threadIdx.x; e < ed;
       e += gridDim.x * blockDim.x)
    acc += w[e];
  for (int off = kWave / 2; off > 0; off >>= 1)
    acc += __shfl_xor(acc, off, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0 && acc)
    atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->cut_w2),
              (unsigned long long)acc);
}

__global__ void k_energy_reset(Ctl *ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctl->cut_w2 = 0;
    ctl->fid_total = 0.0;
  }
}

// ---------------------------------------------------------------------------
// host driver
// ---------------------------------------------------------------------------
namespace {

struct Bufs {
  float *emb_int;
  int32_t *fwd, *rev, *cursor;
  int32_t *rp[2], *col[2], *w[2], *src[2];
  int32_t *size[2], *minpt[2];
  int64_t *S[2];
  double *mu;
  int32_t *target, *parent, *newid, *L, *cap, *toff, *ndeg, *long_rows;
  uint64_t *keys;
  int32_t *tw;
  int32_t *M, *mark, *rank;
  int32_t *bsum, *tmp;
  double *partial;
};

int64_t edge_bound(int32_t n, int32_t k) { return 2 * (int64_t)n * k; }

void carve(Arena &a, int32_t n, int32_t d, int32_t k, bool need_emb,
           Bufs *b) {
  const int64_t ed = edge_bound(n, k);
  const size_t n1 = (size_t)n + 1;
  b->emb_int = need_emb ? a.take<float>((size_t)n * d) : nullptr;
  b->fwd = a.take<int32_t>(n1);
  b->rev = a.take<int32_t>(n1);
  b->cursor = a.take<int32_t>(n1);
  for (int j = 0; j < 2; ++j) {
    b->rp[j] = a.take<int32_t>(n1);
    b->col[j] = a.take<int32_t>(ed);
    b->w[j] = a.take<int32_t>(ed);
    b->src[j] = a.take<int32_t>(ed);
    b->size[j] = a.take<int32_t>(n1);
    b->minpt[j] = a.take<int32_t>(n1);
    b->S[j] = a.take<int64_t>((size_t)n * d);
  }
  b->mu = a.take<double>((size_t)n * d);
  b->target = a.take<int32_t>(n1);
  b->parent = a.take<int32_t>(n1);
  b->newid = a.take<int32_t>(n1);
  b->L = a.take<int32_t>(n1);
  b->cap = a.take<int32_t>(n1);
  b->toff = a.take<int32_t>(n1);
  b->ndeg = a.take<int32_t>(n1);
  b->long_rows = a.take<int32_t>(n1);
  b->keys = a.take<uint64_t>(ed);
  b->tw = a.take<int32_t>(ed);
  b->M = a.take<int32_t>(n1);
  b->mark = a.take<int32_t>(n1);
  b->rank = a.take<int32_t>(n1);
  b->bsum = a.take<int32_t>(scan_blocks(ed + n1) + 2);
  b->tmp = a.take<int32_t>(8);
  b->partial = a.take<double>(kEnergyBlocks);
}

inline dim3 blocks_for(int64_t n, int nt = 256) {
  int64_t b = (n + nt - 1) / nt;
  if (b < 1) b = 1;
  return dim3((unsigned)b);
}

int status_from_err(uint32_t err) {
  if (err & kErrNonFinite) {
    set_error("non-finite value in the input");
    return -2;
  }
  if (err & kErrRange) {
    set_error("embeddings too large for exact fixed-point sums (F < 16)");
    return -3;
  }
  if (err & kErrBadIndex) {
    set_error("neighbour index or label out of range");
    return -1;
  }
  if (err & kErrJump) {
    set_error("pointer jumping did not reach the roots");
    return -5;
  }
  set_error("internal consistency check failed on the device (0x%x)", err);
  return -5;
}

template <bool FIRST>
void launch_round(const Bufs &b, int cur, int32_t n, int32_t k, int32_t nn,
                  int32_t ed, int32_t d, const NodeIn &s, double lambda, int64_t smin,
                  Ctl *ctl, hipStream_t st) {
  const int nxt = 1 - cur;
  const int32_t tcap = (int32_t)edge_bound(n, k);
  hipLaunchKernelGGL(k_round_init, dim3(1), dim3(64), 0, st, ctl);
  prof_begin("select", st);
  hipLaunchKernelGGL(k_select<FIRST>, xcd_grid(blocks_for(nn).x), dim3(256), 0,
                     st, nn, b.rp[cur], b.col[cur], b.w[cur], s, d, lambda,
                     smin, b.target, b.long_rows, ctl);
  hipLaunchKernelGGL(k_select_long<FIRST>, dim3(kLongGrid), dim3(256), 0, st,
                     b.rp[cur], b.col[cur], b.w[cur], s, d, lambda, smin, nn,
                     b.target, b.long_rows, ctl);
  prof_end(st);
  prof_begin("union", st);
  hipLaunchKernelGGL(k_hook, blocks_for(nn), dim3(256), 0, st, nn, b.target,
                     b.parent, ctl);
  hipLaunchKernelGGL(k_jump, blocks_for(nn), dim3(256), 0, st, nn, b.parent,
                     ctl);
  device_scan(ScanRoots{b.parent, b.newid, nn}, nn, b.bsum, &ctl->n_next, st);
  prof_end(st);
  hipLaunchKernelGGL(k_assign, blocks_for(nn), dim3(256), 0, st, nn, b.parent,
                     b.newid, b.L, ctl);
  prof_begin("stats", st);
  hipLaunchKernelGGL(k_zero_acc, blocks_for(nn), dim3(256), 0, st, nn, d, ctl,
                     b.size[nxt], b.S[nxt], b.minpt[nxt], b.cap, b.ndeg);
  hipLaunchKernelGGL(k_stats_add<FIRST>, xcd_grid(blocks_for(nn).x), dim3(256),
                     0, st, nn,
                     b.L, b.rp[cur], s, d, ctl, b.size[nxt], b.S[nxt],
                     b.minpt[nxt], b.cap);
  hipLaunchKernelGGL(k_stats_final, blocks_for((int64_t)nn * d), dim3(256), 0,
                     st, nn, d, ctl, b.size[nxt], b.S[nxt], b.mu);
  prof_end(st);
  prof_begin("contract", st);
  device_scan(ScanArray{b.cap, b.toff, nn, &ctl->n_next}, nn + 1, b.bsum,
              &ctl->slots, st);
  hipLaunchKernelGGL(k_table_clear, blocks_for(ed), dim3(256), 0, st, ed, ctl,
                     b.keys, b.tw);
  hipLaunchKernelGGL(k_insert, xcd_grid(blocks_for(ed).x), dim3(256), 0, st,
                     ed,
                     b.src[cur], b.col[cur], b.w[cur], b.L, b.toff, b.cap,
                     b.keys, b.tw, b.ndeg, nn, tcap, ctl);
  device_scan(ScanArray{b.ndeg, b.rp[nxt], nn, &ctl->n_next}, nn + 1, b.bsum,
              &ctl->e_next, st);
  device_scan(ScanCompact{b.keys, b.tw, &ctl->slots, b.col[nxt], b.w[nxt],
                          b.src[nxt], ed},
              ed, b.bsum, b.tmp, st);
  prof_end(st);
  prof_begin("compose", st);
  hipLaunchKernelGGL(k_compose<FIRST>, xcd_grid(blocks_for(n).x), dim3(256), 0,
                     st, n, nn,
                     b.M, b.L, ctl);
  prof_end(st);
}

}  // namespace

void ladder_reserve(Arena &a, int32_t n, int32_t d, int32_t k) {
  Bufs b;
  carve(a, n, d, k, true, &b);
}

int ladder_run(const LadderArgs &g, Ctl *ctl, Arena &a, hipStream_t st) {
  Bufs b;
  carve(a, g.n, g.d, g.k, true, &b);
  Ctl *h = pinned_ctl();
  if (!h) {
    set_error("hipHostMalloc of the control block failed");
    return -5;
  }
  const int32_t n = g.n, d = g.d, k = g.k;
  int rc;

  // embeddings in internal order, fixed-point shift (Step 0)
  const float *emb = g.emb;
  if (g.perm) {
    hipLaunchKernelGGL(k_gather_rows, blocks_for((int64_t)n * d), dim3(256),
                       0, st, g.emb, g.perm, n, d, b.emb_int);
    emb = b.emb_int;
  }
  hipLaunchKernelGGL(k_maxabs, dim3(256), dim3(256), 0, st, emb,
                     (int64_t)n * d, ctl);
  hipLaunchKernelGGL(k_fixshift, dim3(1), dim3(64), 0, st, ctl, n);

  // graph (Step 0: the superpoint adjacency starts as the kNN graph)
  hipLaunchKernelGGL(k_fill_i32, blocks_for(n), dim3(256), 0, st, b.rev,
                     (int64_t)n, 0);
  hipLaunchKernelGGL(k_fill_i32, blocks_for(n), dim3(256), 0, st, b.cursor,
                     (int64_t)n, 0);
  prof_begin("graph_build", st);
  hipLaunchKernelGGL(k_graph_count, xcd_grid(blocks_for(n).x), dim3(256), 0,
                     st, g.nbr, n,
                     k, b.fwd, b.rev, ctl);
  device_scan(ScanDeg{b.fwd, b.rev, b.rp[0], n}, n + 1, b.bsum, &ctl->e_next,
              st);
  hipLaunchKernelGGL(k_graph_fill, xcd_grid(blocks_for(n).x), dim3(256), 0,
                     st, g.nbr, n,
                     k, b.fwd, b.rp[0], b.cursor, b.col[0], b.w[0], b.src[0],
                     ctl);
  prof_end(st);
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  int32_t ed = h->e_next;
  if ((int64_t)ed > edge_bound(n, k) || ed < 0) {
    set_error("graph larger than its bound");
    return -5;
  }
  // algorithmic bytes: read the n*k table, write 12 bytes per undirected edge
  prof_bytes("graph_build", 4.0 * n * k + 12.0 * (ed / 2));

  int cur = 0;
  bool first = true;
  int32_t nn = n;
  const int32_t max_rounds = g.max_rounds > 0 ? g.max_rounds : 256;
  for (int32_t l = 0; l < g.n_levels; ++l) {
    const double lambda = g.lambdas[l];
    const int64_t smin = g.min_size ? g.min_size[l] : 0;
    for (int32_t round = 0;; ++round) {
      if (ed == 0) break;  // no edge left: nothing can merge
      if (round >= max_rounds) {
        set_error("level %d reached max_rounds = %d", l, max_rounds);
        return -6;
      }
      NodeIn s;
      s.emb = emb;
      s.perm = g.perm;
      if (first) {
        s.size = nullptr;
        s.S = nullptr;
        s.mu = nullptr;
        s.minpt = nullptr;
        launch_round<true>(b, cur, n, k, nn, ed, d, s, lambda, smin, ctl, st);
      } else {
        s.size = b.size[cur];
        s.S = b.S[cur];
        s.mu = b.mu;
        s.minpt = b.minpt[cur];
        launch_round<false>(b, cur, n, k, nn, ed, d, s, lambda, smin, ctl, st);
      }
      if ((rc = read_ctl(ctl, h, st))) return rc;
      if (h->err) return status_from_err(h->err);
      if (prof_on()) {
        // algorithmic bytes of the round (undirected edges of 12 bytes,
        // node statistics of S bytes: 4d fp32 in the first round, then
        // 8d int64 sums + 8 bytes of size and smallest point)
        const double E0 = ed / 2, S0 = first ? 4.0 * d : 8.0 * d + 8.0;
        prof_bytes("select", 12.0 * E0 + S0 * nn + 4.0 * nn);
        if (h->any_choice) {
          const double E1 = h->e_next / 2, S1 = 8.0 * d + 8.0;
          prof_bytes("union", 8.0 * nn);
          prof_bytes("stats", S0 * nn + S1 * h->n_next);
          prof_bytes("contract", 12.0 * E0 + 4.0 * nn + 12.0 * E1);
          prof_bytes("compose", 8.0 * n);
        }
      }
      if (!h->any_choice) break;  // Step 1: no candidate merge
      if (h->n_next < 1 || h->n_next >= nn || h->e_next < 0 || h->e_next > ed) {
        set_error("round sizes out of range (%d nodes, %d edges)", h->n_next,
                  h->e_next);
        return -5;
      }
      cur = 1 - cur;
      first = false;
      nn = h->n_next;
      ed = h->e_next;
      if (nn == 1) break;  // a single component is left
    }

    // level output
    int32_t *out = g.labels + (int64_t)l * n;
    if (first) {
      hipLaunchKernelGGL(k_iota, blocks_for(n), dim3(256), 0, st, n, out);
    } else {
      hipLaunchKernelGGL(k_fill_i32, blocks_for(n), dim3(256), 0, st, b.mark,
                         (int64_t)n, 0);
      hipLaunchKernelGGL(k_mark, blocks_for(nn), dim3(256), 0, st, nn,
                         b.minpt[cur], b.mark, n, ctl);
      device_scan(ScanArray{b.mark, b.rank, n, nullptr}, n, b.bsum, b.tmp, st);
      hipLaunchKernelGGL(k_labels, blocks_for(n), dim3(256), 0, st, n, nn,
                         g.inv, b.M, b.minpt[cur], b.rank, out, ctl);
    }
    g.n_comp[l] = nn;
    if (g.want_energy && g.energy) {
      hipLaunchKernelGGL(k_energy_reset, dim3(1), dim3(64), 0, st, ctl);
      if (first)
        hipLaunchKernelGGL(k_energy_fid<true>, dim3(kEnergyBlocks), dim3(256),
                           0, st, n, d, nn, emb, b.M, b.mu, ctl, b.partial);
      else
        hipLaunchKernelGGL(k_energy_fid<false>, dim3(kEnergyBlocks), dim3(256),
                           0, st, n, d, nn, emb, b.M, b.mu, ctl, b.partial);
      hipLaunchKernelGGL(k_energy_sum, dim3(1), dim3(64), 0, st, b.partial,
                         kEnergyBlocks, ctl);
      hipLaunchKernelGGL(k_weight_sum, dim3(256), dim3(256), 0, st, ed,
                         b.w[cur], ctl);
      if ((rc = read_ctl(ctl, h, st))) return rc;
      if (h->err) return status_from_err(h->err);
      const double cut = (double)(h->cut_w2 / 2);
      const double reg = lambda * cut;
      g.energy[l] = h->fid_total + reg;
    }
  }
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  return 0;
}

}  // namespace ezsp
