// ezsp_merge.hip -- the merge ladder of EZ-SP (arXiv 2512.00385, Sec. 3.2):
// kNN graph, then rounds of Steps 1-4 on the superpoint adjacency until no
// candidate merge is left, for every regularisation strength of the ladder
// (hierarchical partition).
//
// Representation.  Nodes of a round are its superpoints, stored in an
// internal order (Morton order of the points when the graph came from xyz)
// that keeps neighbours close in memory.  Each node keeps its size |P|, the
// exact int64 fixed-point sum of its embeddings, its fp64 mean and `minpt`,
// the smallest original point index of its points.  Ordering nodes by minpt
// is ordering them by their canonical number, so the tie rule and the output
// labels use minpt and the internal order never shows in the results.
//
// Adjacency, both directions of every undirected edge:
//   first round  row v = the valid entries of the kNN row v (weight 1) plus
//                a short reverse list of the u that have v in their kNN row
//                while v does not have u;
//   later rounds row v = a window [ws[v], ws[v] + wl[v]) of a table of
//                packed (neighbour << 32 | weight) slots, empty slots = ~0.
//
// One round (host reads the control block back once at the end):
//   select    Steps 1-2: each node scans its row, evaluates Prop. 1's gain
//             and keeps the best candidate (largest gain, ties to the
//             smaller minpt); rows longer than kLongRow take a whole wave
//   hook      merge graph -> forest: every cycle of the merge graph is a
//             mutual pair (each choice is at least as good as the choice it
//             follows), the lower id of a pair becomes a root
//   jump      pointer jumping to the roots: weakly connected components
//             (Step 3, the partition App. Alg. A-1 computes)
//   relabel   roots numbered by a scan
//   members   counting sort of the nodes by component (one atomic per node)
//   stats     Step 4: size, int64 sums, fp64 mean, minpt, summed degree per
//             component, gathered from its members (no atomics)
//   contract  Step 4: one thread per directed entry relabels it into its
//             component's window of the next table (capacity = summed
//             degree); parallel edges add their weights in the same slot,
//             edges inside a component are dropped; the window is the next
//             round's row and every occupied slot records its owner
#include <math.h>
#include <stdlib.h>

#include <algorithm>

#include "ezsp_internal.h"

namespace ezsp {

constexpr uint64_t kEmpty = ~0ull;
constexpr int kJumpWalk = 64;  // steps of a pointer-jumping walk
constexpr int kLongRow = 128;    // longer rows go in entry chunks ...
constexpr int kLongChunk = 1024; // ... of this many entries, a wave each
constexpr int kLongGrid = 2048;  // blocks of 4 waves for the chunks
constexpr int kBigComp = 128;   // components with more members: one block
constexpr int kSelLanesFirst = 2;  // lanes per row in the first round's select
constexpr int kSelLanes = 4;       // ... in later rounds
constexpr int kStatsLanes = 4;     // lanes per component in the statistics
constexpr int kBigGrid = 512;
constexpr int kChunk = 1024;    // table slots contracted by one block in LDS
constexpr int kBatch = 256;     // members taken at a time by a block
constexpr int kPreSlots = 4096; // LDS pre-aggregation table of a big tile

// ---------------------------------------------------------------------------
// small kernels
// ---------------------------------------------------------------------------
__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Rows of 4k floats: 16-byte moves, and the max |e| of Step 0's fixed-point
// shift (with the non-finite check) taken on the way, striped per block.
__global__ __launch_bounds__(256) void k_gather_rows4(const float4 *emb,
                                                      const int32_t *perm,
                                                      int32_t n, int32_t d4,
                                                      float4 *out, Ctl *ctl) {
  uint32_t m = 0;
  bool bad = false;
  const int64_t total = (int64_t)n * d4;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / d4;
    const float4 x = emb[(int64_t)perm[i] * d4 + (t - i * d4)];
    out[t] = x;
    const float v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (!isfinite(v[j])) bad = true;
      else m = max(m, __float_as_uint(fabsf(v[j])));
    }
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1)
    m = max(m, (uint32_t)__shfl_xor((int)m, off, kWave));
  __shared__ uint32_t sm[256 / kWave];
  __shared__ int sbad;
  if (threadIdx.x == 0) sbad = 0;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) sm[threadIdx.x / kWave] = m;
  if (__ballot(bad) && (threadIdx.x & (kWave - 1)) == 0) sbad = 1;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = sm[0];
    for (int q = 1; q < 256 / kWave; ++q) r = max(r, sm[q]);
    stripe_max(ctl->maxabs_s, (int32_t)r);  // |e| bits < 2^31
    if (sbad) raise_err(ctl, kErrNonFinite);
  }
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
// first-round graph: the union of the kNN relations, one undirected edge of
// weight 1 per pair (Sec. 3.1, Sec. 4.1; self loops and repeats removed as
// App. Alg. A-2's prepare_graph does)
// ---------------------------------------------------------------------------

// A caller's neighbour table (stride k) into the internal one (stride
// pad4(k)): entries outside [-1, n) are an error; -1, the point itself and
// repeats of an earlier entry become -1, and so does the padding.
__global__ __launch_bounds__(256) void k_sanitize(const int32_t *nbr,
                                                  int32_t n, int32_t k,
                                                  int32_t *out, Ctl *ctl) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t kp = pad4(k);
  const int32_t *r = nbr + (int64_t)i * k;
  int32_t *o = out + (int64_t)i * kp;
  for (int32_t t = 0; t < k; ++t) {
    int32_t j = r[t];
    if (j < -1 || j >= n) {
      raise_err(ctl, kErrBadIndex);
      j = -1;
    }
    if (j == i) j = -1;
    for (int32_t s = 0; s < t && j >= 0; ++s)
      if (r[s] == j) j = -1;
    o[t] = j;
  }
  for (int32_t t = k; t < kp; ++t) o[t] = -1;
}

// Row j of the internal table (stride kp, a multiple of 4) contains x?
__device__ __forceinline__ bool row_has(const int32_t *nbr, int32_t kp,
                                        int32_t j, int32_t x) {
  const int4 *r = reinterpret_cast<const int4 *>(nbr + (int64_t)j * kp);
  bool hit = false;
  for (int32_t q = 0; q < kp / 4; ++q) {
    const int4 v = r[q];
    hit |= (v.x == x) | (v.y == x) | (v.z == x) | (v.w == x);
  }
  return hit;
}

// Reverse entries: i lists u, u does not list i -> u's row gets i.  The
// count pass keeps, per point, the bit mask of its entries that are not
// mutual (k <= 64), so the fill pass does not look at the rows again.  All
// row checks of a point are made before its atomics.
__global__ __launch_bounds__(256) void k_rev_count(const int32_t *nbr,
                                                   int32_t n, int32_t k,
                                                   int32_t *rev,
                                                   uint64_t *nmask, Ctl *ctl) {
  const int32_t i = xcd_tid();
  const int32_t kp = pad4(k);
  int32_t fwd = 0;
  if (i < n) {
    const int32_t *r = nbr + (int64_t)i * kp;
    uint64_t mask = 0;
#pragma unroll 4
    for (int32_t t = 0; t < k; ++t) {
      const int32_t u = r[t];
      if (u < 0) continue;
      ++fwd;
      if (!row_has(nbr, kp, u, i)) mask |= 1ull << t;
    }
    nmask[i] = mask;
    for (uint64_t m = mask; m; m &= m - 1)
      atomicAdd(&rev[r[__builtin_ctzll(m)]], 1);
  }
  fwd = wave_sum(fwd);
  if ((threadIdx.x & (kWave - 1)) == 0 && fwd) stripe_add(ctl->e_fwd_s, fwd);
}

__global__ __launch_bounds__(256) void k_rev_fill(const int32_t *nbr,
                                                  int32_t n, int32_t k,
                                                  const uint64_t *nmask,
                                                  const int32_t *rrp,
                                                  int32_t *cursor,
                                                  int32_t *rcol, Ctl *ctl) {
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const int32_t *r = nbr + (int64_t)i * pad4(k);
  // four entries at a time: their cursor increments (atomics that return a
  // position) and list bounds are issued before any is used
  constexpr int kQ = 4;
  for (uint64_t m = nmask[i]; m;) {
    int32_t u[kQ], pos[kQ], lo[kQ], hi[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      u[q] = -1;
      if (m) {
        u[q] = r[__builtin_ctzll(m)];
        m &= m - 1;
      }
    }
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      pos[q] = 0;
      lo[q] = hi[q] = 0;
      if (u[q] >= 0) {
        pos[q] = atomicAdd(&cursor[u[q]], 1);
        lo[q] = rrp[u[q]];
        hi[q] = rrp[u[q] + 1];
      }
    }
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      if (u[q] < 0) continue;
      const int32_t p = lo[q] + pos[q];
      if (p < hi[q]) {
        rcol[p] = i;
      } else {
        raise_err(ctl, kErrInternal);
      }
    }
  }
}

// The reverse count and fill of a kNN graph from this library, a block per
// kRevR consecutive points.  Internal order is Morton order, so most
// neighbours of a point lie in its own block (86 % of the driving tile's
// kNN entries for blocks of 512): their points and k-th keys are read from
// LDS, and the reverse entries they receive are counted with LDS atomics,
// one global add per point at the end.  In the fill, the entries from
// inside the block take the top of u's list (LDS cursors, counting down
// from rrp[u+1]) and those from other blocks the bottom (global cursors
// from rrp[u]); both kernels split the entries the same way, so the two
// parts fill the list exactly.  u lists i exactly when i's key as seen from
// u, (d2 bits, original index) with d2 in the kNN's own operation order,
// does not exceed u's k-th key: the test needs u's point and k-th key
// instead of u's whole row.  Same lists as k_rev_count and k_rev_fill, up
// to the order inside a list.
constexpr int kRevR = 512;
constexpr int kRevNT = 256;  // threads per block: two passes over its points
                             // (faster than four, or one of 1024 threads)
__global__ __launch_bounds__(kRevNT) void k_rev_count_blk(
    const int32_t *nbr, int32_t n, int32_t k, const float4 *__restrict__ pts,
    const uint64_t *__restrict__ kth, int32_t *rev, uint64_t *nmask,
    Ctl *ctl) {
  __shared__ float4 sp[kRevR];
  __shared__ uint64_t sk[kRevR];
  __shared__ int32_t sc[kRevR];
  const int32_t lo = xcd_block() * kRevR;
  if (lo >= n) return;  // the whole block
  const int32_t nr = min(kRevR, n - lo);
  for (int32_t q = threadIdx.x; q < nr; q += blockDim.x) {
    sp[q] = pts[lo + q];
    sk[q] = kth[lo + q];
    sc[q] = 0;
  }
  __syncthreads();
  constexpr int kCh = 3;  // row chunks of four entries taken at once
  const int32_t kp = pad4(k);
  const int32_t nch = kp / 4;
  int32_t fwd = 0;
  for (int32_t r = threadIdx.x; r < nr; r += blockDim.x) {
    const int32_t i = lo + r;
    const int4 *r4 = reinterpret_cast<const int4 *>(nbr + (int64_t)i * kp);
    const float4 pi = sp[r];
    uint64_t mask = 0;
    for (int32_t c0 = 0; c0 < nch; c0 += kCh) {
      int32_t u[4 * kCh];
#pragma unroll
      for (int j = 0; j < kCh; ++j) {
        const int4 c = r4[min(c0 + j, nch - 1)];
        const bool in = c0 + j < nch;
        u[4 * j + 0] = in ? c.x : -1;
        u[4 * j + 1] = in ? c.y : -1;
        u[4 * j + 2] = in ? c.z : -1;
        u[4 * j + 3] = in ? c.w : -1;
      }
      float4 pu[4 * kCh];
      uint64_t ku[4 * kCh];
#pragma unroll
      for (int t = 0; t < 4 * kCh; ++t) {
        // empty entries read the point itself; entries out of range are
        // caught by the sanitizer or the kNN, never reach here
        const int32_t uc = (uint32_t)u[t] < (uint32_t)n ? u[t] : i;
        const uint32_t ru = (uint32_t)(uc - lo);
        // one generic pointer for LDS and global memory: a flat load each,
        // with no branch (two branches writing the same registers make the
        // LDS one wait for every global load in flight)
        const bool inb = ru < (uint32_t)nr;
        const float4 *ps = inb ? &sp[ru] : &pts[uc];
        const uint64_t *ks = inb ? &sk[ru] : &kth[uc];
        pu[t] = *ps;
        ku[t] = *ks;
      }
#pragma unroll
      for (int t = 0; t < 4 * kCh; ++t) {
        const int32_t slot = 4 * c0 + t;  // entries past k hold -1
        if (u[t] < 0) continue;
        ++fwd;
        const float dx = pi.x - pu[t].x, dy = pi.y - pu[t].y,
                    dz = pi.z - pu[t].z;
        const float d2 = fmaf(dz, dz, fmaf(dy, dy, dx * dx));
        const uint64_t key = ((uint64_t)__float_as_uint(d2) << 32) |
                             (uint32_t)__float_as_int(pi.w);
        if (key > ku[t]) mask |= 1ull << slot;
      }
    }
    nmask[i] = mask;
    const int32_t *row = nbr + (int64_t)i * kp;
    for (uint64_t m = mask; m; m &= m - 1) {
      const int32_t u = row[__builtin_ctzll(m)];
      const uint32_t ru = (uint32_t)(u - lo);
      if (ru < (uint32_t)nr)
        atomicAdd(&sc[ru], 1);
      else if ((uint32_t)u < (uint32_t)n)
        atomicAdd(&rev[u], 1);
      else
        raise_err(ctl, kErrInternal);
    }
  }
  __syncthreads();
  for (int32_t q = threadIdx.x; q < nr; q += blockDim.x)
    if (sc[q]) atomicAdd(&rev[lo + q], sc[q]);
  fwd = wave_sum(fwd);
  if ((threadIdx.x & (kWave - 1)) == 0 && fwd) stripe_add(ctl->e_fwd_s, fwd);
}

__global__ __launch_bounds__(kRevNT) void k_rev_fill_blk(
    const int32_t *nbr, int32_t n, int32_t k, const uint64_t *nmask,
    const int32_t *rrp, int32_t *cursor, int32_t *rcol, Ctl *ctl) {
  __shared__ int32_t srp[kRevR + 1];
  __shared__ int32_t sc[kRevR];
  const int32_t lo = xcd_block() * kRevR;
  if (lo >= n) return;  // the whole block
  const int32_t nr = min(kRevR, n - lo);
  for (int32_t q = threadIdx.x; q <= nr; q += blockDim.x) {
    srp[q] = rrp[lo + q];
    if (q < nr) sc[q] = 0;
  }
  __syncthreads();
  const int32_t kp = pad4(k);
  for (int32_t r = threadIdx.x; r < nr; r += blockDim.x) {
    const int32_t i = lo + r;
    const int32_t *row = nbr + (int64_t)i * kp;
    // four entries at a time: their positions (atomics that return one)
    // and list bounds are issued before any is used
    constexpr int kQ = 4;
    for (uint64_t m = nmask[i]; m;) {
      int32_t u[kQ], p[kQ], lim[kQ];
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        u[q] = -1;
        if (m) {
          u[q] = row[__builtin_ctzll(m)];
          m &= m - 1;
        }
      }
      // each entry's position and list bounds through one generic pointer
      // (flat atomics and loads, no branch): the top of the list from the
      // LDS cursors, counting down, or the bottom from the global ones
      int32_t pos[kQ], b0[kQ], b1[kQ];
      bool inb[kQ];
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        if ((uint32_t)u[q] >= (uint32_t)n) u[q] = -1;
        const int32_t uq = u[q] < 0 ? lo : u[q];
        const uint32_t ru = (uint32_t)(uq - lo);
        inb[q] = ru < (uint32_t)nr;
        int32_t *cur = inb[q] ? &sc[ru] : &cursor[uq];
        const int32_t *bnd = inb[q] ? &srp[ru] : &rrp[uq];
        pos[q] = u[q] >= 0 ? atomicAdd(cur, 1) : 0;
        b0[q] = bnd[0];
        b1[q] = bnd[1];
      }
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        p[q] = inb[q] ? b1[q] - 1 - pos[q] : b0[q] + pos[q];
        lim[q] = inb[q] ? b0[q] : b1[q];
      }
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        if (u[q] < 0) continue;
        const bool ok = inb[q] ? p[q] >= lim[q] : p[q] < lim[q];
        if (ok)
          rcol[p[q]] = i;
        else
          raise_err(ctl, kErrInternal);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// node state and adjacency of a round
// ---------------------------------------------------------------------------
struct NodeIn {
  const int32_t *size;   // |P|              (null in the first round)
  const int64_t *S;      // fixed-point sums (null in the first round)
  const double *mu;      // fp64 means       (null in the first round)
  const int32_t *minpt;  // smallest point   (null in the first round)
  const float *emb;      // point embeddings, internal order (first round)
  const int32_t *perm;   // internal -> original point, nullable (identity)
  const uint8_t *merged; // 1 for a node formed by a merge in the last round;
                         // null: every node is evaluated (a level's first
                         // round)
};

struct Adj {
  // first round
  const int32_t *nbr;  // n rows of stride kp, -1 = no entry
  int32_t k, kp;
  const int32_t *rrp, *rcol;  // reverse lists
  int32_t n_rev;
  // later rounds
  const int32_t *ws, *wl;
  const uint64_t *tbl;
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
__device__ __forceinline__ int64_t node_S(const NodeIn &s, int32_t v,
                                          int32_t i, int32_t d, double sF) {
  if (FIRST) return (int64_t)rint((double)s.emb[(int64_t)v * d + i] * sF);
  return s.S[(int64_t)v * d + i];
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

// Slots of v's row (including empty ones).
template <bool FIRST>
__device__ __forceinline__ int32_t row_span(const Adj &a, int32_t v) {
  if (FIRST) return a.k + (a.rrp[v + 1] - a.rrp[v]);
  return a.wl[v];
}

// Calls f(u, w) for the entries j = begin, begin + stride, ... of v's row.
template <bool FIRST, class Fn>
__device__ __forceinline__ void for_row(const Adj &a, int32_t v, int32_t begin,
                                        int32_t stride, Fn &&f) {
  if (FIRST) {
    const int32_t *r = a.nbr + (int64_t)v * a.kp;
    const int32_t r0 = a.rrp[v];
    const int32_t len = a.k + (a.rrp[v + 1] - r0);
    for (int32_t j = begin; j < len; j += stride) {
      const int32_t u = (j < a.k) ? r[j] : a.rcol[r0 + (j - a.k)];
      if (u >= 0) f(u, 1);
    }
  } else {
    const uint64_t *t = a.tbl + a.ws[v];
    const int32_t len = a.wl[v];
    for (int32_t j = begin; j < len; j += stride) {
      const uint64_t e = t[j];
      if (e != kEmpty) f((int32_t)(e >> 32), (int32_t)(uint32_t)e);
    }
  }
}

// Entry j of v's row (0 <= j < row_span); false for an empty entry.
template <bool FIRST>
__device__ __forceinline__ bool row_entry(const Adj &a, int32_t v, int32_t j,
                                          int32_t &u, int32_t &w) {
  if (FIRST) {
    u = (j < a.k) ? a.nbr[(int64_t)v * a.kp + j]
                  : a.rcol[a.rrp[v] + (j - a.k)];
    w = 1;
    return u >= 0;
  }
  const uint64_t e = a.tbl[a.ws[v] + j];
  u = (int32_t)(e >> 32);
  w = (int32_t)(uint32_t)e;
  return e != kEmpty;
}

// Row base of v for row_entry_at: the start of v's reverse list (first
// round) or of its table window (later rounds).
template <bool FIRST>
__device__ __forceinline__ int32_t row_base(const Adj &a, int32_t v) {
  return FIRST ? a.rrp[v] : a.ws[v];
}

// row_entry with v's row base already known.
template <bool FIRST>
__device__ __forceinline__ bool row_entry_at(const Adj &a, int32_t v,
                                             int32_t base, int32_t j,
                                             int32_t &u, int32_t &w) {
  if (FIRST) {
    u = (j < a.k) ? a.nbr[(int64_t)v * a.kp + j] : a.rcol[base + (j - a.k)];
    w = 1;
    return u >= 0;
  }
  const uint64_t e = a.tbl[base + j];
  u = (int32_t)(e >> 32);
  w = (int32_t)(uint32_t)e;
  return e != kEmpty;
}

__global__ void k_round_init(Ctl *ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctl->any_choice = 0;
    ctl->n_next = 0;
    ctl->e_next = 0;
    ctl->slots = 0;
    ctl->n_long = 0;
    ctl->n_lchunk = 0;
    ctl->n_big = 0;
    ctl->n_cbig = 0;
    ctl->n_tiles = 0;
    ctl->n_iso = 0;
    ctl->n_link = 0;
  }
  if (blockIdx.x == 0) stripe_zero(ctl->e_next_s);
}

// ---------------------------------------------------------------------------
// Steps 1-2.  Prop. 1 (Eq. delta):
//   Delta(P,Q) = lambda * w_PQ - |P||Q| / (|P|+|Q|) * |Y_P - Y_Q|^2,
// evaluated in fp64 in a fixed order (no contraction): f = (sP*sQ)/(sP+sQ),
// ss = sum_i (mu_P,i - mu_Q,i)^2 left to right, Delta = lambda*w - f*ss.
// The formula is symmetric bit for bit, so P and Q see the same value.
// A directed edge P -> Q is a candidate when Delta > 0 or |P| < s_min; P
// keeps its largest candidate, ties to the neighbour with smaller minpt.
// ---------------------------------------------------------------------------
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
__device__ __forceinline__ double edge_gain(const NodeIn &s, int32_t v,
                                            double dsv, int32_t u, int32_t w,
                                            int32_t d, double lambda,
                                            double sF, double sIF) {
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
  const double cut = lambda * (double)w;
  const double fit = f * ss;
  return cut - fit;
}

// Mean row of a node held in registers when D is a compile-time size DT
// (a multiple of 4): one vector load per 16 bytes instead of one scalar load
// per dimension.  Same values as node_mu.
template <bool FIRST, int DT>
struct MeanRow {
  double m[DT > 0 ? DT : 1];
  __device__ __forceinline__ void load(const NodeIn &s, int32_t v, double sF,
                                       double sIF) {
    if constexpr (DT > 0) {
      if (FIRST) {
        const float4 *p =
            reinterpret_cast<const float4 *>(s.emb + (int64_t)v * DT);
#pragma unroll
        for (int q = 0; q < DT / 4; ++q) {
          const float4 x = p[q];
          m[4 * q + 0] = rint((double)x.x * sF) * sIF;
          m[4 * q + 1] = rint((double)x.y * sF) * sIF;
          m[4 * q + 2] = rint((double)x.z * sF) * sIF;
          m[4 * q + 3] = rint((double)x.w * sF) * sIF;
        }
      } else {
        const double2 *p =
            reinterpret_cast<const double2 *>(s.mu + (int64_t)v * DT);
#pragma unroll
        for (int q = 0; q < DT / 2; ++q) {
          const double2 x = p[q];
          m[2 * q + 0] = x.x;
          m[2 * q + 1] = x.y;
        }
      }
    }
  }
};

// Prop. 1 for the edge (v, u) with v's mean row already loaded; the same
// operations in the same order as edge_gain.
template <bool FIRST, int DT>
__device__ __forceinline__ double edge_gain_t(const NodeIn &s,
                                              const MeanRow<FIRST, DT> &mv,
                                              int32_t v, double dsv,
                                              int32_t u, int32_t w, int32_t d,
                                              double lambda, double sF,
                                              double sIF) {
  if constexpr (DT == 0) {
    return edge_gain<FIRST>(s, v, dsv, u, w, d, lambda, sF, sIF);
  } else {
    MeanRow<FIRST, DT> mu;
    mu.load(s, u, sF, sIF);
    const double dsu = (double)node_size<FIRST>(s, u);
    const double num = dsv * dsu;
    const double den = dsv + dsu;
    const double f = num / den;
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < DT; ++i) {
      const double diff = mv.m[i] - mu.m[i];
      const double sq = diff * diff;
      ss = ss + sq;
    }
    const double cut = lambda * (double)w;
    const double fit = f * ss;
    return cut - fit;
  }
}

// Long rows: every row longer than kLongRow is split into chunks of
// kLongChunk entries; chunk item i belongs to long row item[i], which starts
// at chunk base[slot] and has nch[slot] chunks.  Per chunk: the best
// candidate (g, mp, u) and the count of valid entries.
struct LongWork {
  int32_t *rows, *base, *nch, *item;
  double *g;
  int32_t *mp, *u, *cnt;
  int32_t cap;  // chunk items available
};

// Steps 1-2 for rows of up to kLongRow entries, G lanes per row: the lanes
// take every G-th entry of the row (shorter dependent chains per lane than
// a thread per row, and a wave waits for its longest rows only G-fold
// shortened), then the group combines its candidates.
// With a worklist (WL, incremental rounds), group i takes node work[i] of
// the first n_work; otherwise group v takes node v of the nn.
template <bool FIRST, int DT, int G, bool WL = false>
__global__ __launch_bounds__(256) void k_select(
    int32_t nn, Adj a, NodeIn s, int32_t d, double lambda, int64_t smin,
    int32_t *__restrict__ target, int32_t *__restrict__ deg, LongWork lw,
    const int32_t *__restrict__ work, int32_t n_work, Ctl *ctl) {
  const int32_t tid = xcd_tid();
  const int32_t item = tid / G;
  const int lg = tid & (G - 1);
  const int32_t n_items = WL ? n_work : nn;
  const int32_t v = item < n_items ? (WL ? work[item] : item) : nn;
  const bool in = v < nn;
  const int32_t span = in ? row_span<FIRST>(a, v) : 0;
  const bool live = in && span <= kLongRow;
  if (in && !live && lg == 0) {  // listed with its chunks
    const int32_t nch = (span + kLongChunk - 1) / kLongChunk;
    const int32_t slot = atomicAdd(&ctl->n_long, 1);
    const int32_t base = atomicAdd(&ctl->n_lchunk, nch);
    if (slot < nn && base + nch <= lw.cap) {
      lw.rows[slot] = v;
      lw.base[slot] = base;
      lw.nch[slot] = nch;
      for (int32_t c = 0; c < nch; ++c) lw.item[base + c] = slot;
    } else {
      raise_err(ctl, kErrInternal);
    }
  }
  Best b{0.0, -1, -1};  // mp < 0: not loaded yet
  int32_t cnt = 0;
  bool skip = false;
  if constexpr (!FIRST) {
    // A node that did not merge, with no neighbour that merged, has the
    // gains of the last round, which gave it no candidate: no candidate now.
    if (s.merged) {
      int32_t any = 0, c0 = 0;
      if (live) {
        any = s.merged[v];
        if (!any)  // a merged node is evaluated anyway: no scan for it
          for_row<false>(a, v, lg, G, [&](int32_t u, int32_t) {
            ++c0;
            if ((uint32_t)u < (uint32_t)nn) any |= s.merged[u];
          });
      }
#pragma unroll
      for (int off = G / 2; off > 0; off >>= 1)
        any |= __shfl_xor(any, off, kWave);
      if (!any) {
        skip = true;
        cnt = c0;
      }
    }
  }
  if (live && !skip) {
    const int F = ctl->F;
    const double sF = ldexp(1.0, F), sIF = ldexp(1.0, -F);
    const int32_t sv = node_size<FIRST>(s, v);
    const double dsv = (double)sv;
    const bool small = (int64_t)sv < smin;
    MeanRow<FIRST, DT> mv;
    mv.load(s, v, sF, sIF);
    for_row<FIRST>(a, v, lg, G, [&](int32_t u, int32_t w) {
      ++cnt;
      if ((uint32_t)u >= (uint32_t)nn) {
        raise_err(ctl, kErrInternal);
        return;
      }
      const double g =
          edge_gain_t<FIRST, DT>(s, mv, v, dsv, u, w, d, lambda, sF, sIF);
      // the smallest point only breaks a tie of equal gains: loaded for a
      // tie and for the lane's final choice, not for every candidate
      if (g > 0.0 || small) {
        if (b.u < 0 || g > b.g) {
          b = Best{g, -1, u};
        } else if (g == b.g) {
          if (b.mp < 0) b.mp = node_minpt<FIRST>(s, b.u);
          const int32_t mp = node_minpt<FIRST>(s, u);
          if (mp < b.mp) b = Best{g, mp, u};
        }
      }
    });
    if (b.u >= 0 && b.mp < 0) b.mp = node_minpt<FIRST>(s, b.u);
  }
  if constexpr (G > 1) {
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) {
      Best o;
      o.g = __shfl_xor(b.g, off, kWave);
      o.mp = __shfl_xor(b.mp, off, kWave);
      o.u = __shfl_xor(b.u, off, kWave);
      if (best_before(o, b)) b = o;
      cnt += __shfl_xor(cnt, off, kWave);
    }
  }
  if (live && lg == 0) {
    target[v] = b.u;
    deg[v] = cnt;
  }
  if (__ballot(live && lg == 0 && b.u >= 0) && (threadIdx.x & (kWave - 1)) == 0)
    ctl->any_choice = 1;
}

// Steps 1-2 of the first round for D = DT (a multiple of 4): a block takes
// kSelFirstBytes / (4 DT) consecutive nodes and stages their embedding rows
// in LDS.  Internal order is Morton order, so most neighbours of a node lie
// in its own block (on the driving tile, 86 % of the kNN entries for blocks
// of 512 nodes) and are read from LDS, the others from global memory.
// Every node is one point (|P| = 1), so the smallest point of a neighbour,
// which only breaks ties of equal gains, is loaded only for a tie and for
// each lane's final choice.  The same choice as k_select<true>.
// The rows are staged as the fp32 integers a = rint(e * 2^F): e * 2^F is
// exact in fp32 (16 <= F <= 40, |e| * 2^F < 2^62) and so is its rounding,
// and mu = a * 2^-F.  Scaling by a power of two commutes with rounding in
// the normal range, so the sum of the squared differences of the a's
// times 2^-2F is, bit for bit, the sum over the mu's: the conversion is
// done once per staged row, and a gain costs four operations a dimension.
constexpr int kSelFirstBytes = 32768;
// 512 threads take a block's nodes in two passes: measured faster than
// four passes (256 threads), one (1024 threads, fewer blocks resident), and
// blocks of 256 or 1024 nodes
constexpr int kSelFirstNT = 512;
template <int DT, int G>
__global__ __launch_bounds__(kSelFirstNT) void k_select_first(
    int32_t nn, Adj a, NodeIn s, double lambda, int64_t smin,
    int32_t *__restrict__ target, int32_t *__restrict__ deg, LongWork lw,
    Ctl *ctl) {
  static_assert(DT > 0 && DT % 4 == 0, "float4 rows");
  constexpr int Q = DT / 4;                          // float4 per row
  constexpr int32_t R = kSelFirstBytes / (16 * Q);   // nodes per block
  __shared__ float4 sE[R * Q];
  const int32_t lo = xcd_block() * R;
  if (lo >= nn) return;  // the whole block
  const int32_t nr = min(R, nn - lo);
  const float4 *gE = reinterpret_cast<const float4 *>(s.emb);
  const int F = ctl->F;
  const float sFf = ldexpf(1.0f, F);
  const double sIF2 = ldexp(1.0, -2 * F);
  auto quant = [&](float4 x) {
    return make_float4(rintf(x.x * sFf), rintf(x.y * sFf), rintf(x.z * sFf),
                       rintf(x.w * sFf));
  };
  for (int32_t q = threadIdx.x; q < nr * Q; q += blockDim.x)
    sE[q] = quant(gE[(int64_t)lo * Q + q]);
  __syncthreads();
  const bool small = (int64_t)1 < smin;
  const int lg = threadIdx.x & (G - 1);
  bool chose = false;
  for (int32_t r0 = 0; r0 < nr; r0 += (int32_t)blockDim.x / G) {
    const int32_t r = r0 + (int32_t)threadIdx.x / G;
    const int32_t v = lo + r;
    const bool in = r < nr;
    const int32_t span = in ? row_span<true>(a, v) : 0;
    const bool live = in && span <= kLongRow;
    if (in && !live && lg == 0) {  // listed with its chunks
      const int32_t nch = (span + kLongChunk - 1) / kLongChunk;
      const int32_t slot = atomicAdd(&ctl->n_long, 1);
      const int32_t base = atomicAdd(&ctl->n_lchunk, nch);
      if (slot < nn && base + nch <= lw.cap) {
        lw.rows[slot] = v;
        lw.base[slot] = base;
        lw.nch[slot] = nch;
        for (int32_t c = 0; c < nch; ++c) lw.item[base + c] = slot;
      } else {
        raise_err(ctl, kErrInternal);
      }
    }
    Best b{0.0, -1, -1};  // mp < 0: not loaded yet
    int32_t cnt = 0;
    if (live) {
      double mv[DT];  // the a's of v's row
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const float4 x = sE[r * Q + q];
        mv[4 * q + 0] = (double)x.x;
        mv[4 * q + 1] = (double)x.y;
        mv[4 * q + 2] = (double)x.z;
        mv[4 * q + 3] = (double)x.w;
      }
      for_row<true>(a, v, lg, G, [&](int32_t u, int32_t w) {
        ++cnt;
        if ((uint32_t)u >= (uint32_t)nn) {
          raise_err(ctl, kErrInternal);
          return;
        }
        float4 x[Q];
        const uint32_t ru = (uint32_t)(u - lo);
        if (ru < (uint32_t)nr) {
#pragma unroll
          for (int q = 0; q < Q; ++q) x[q] = sE[ru * Q + q];
        } else {
#pragma unroll
          for (int q = 0; q < Q; ++q) x[q] = quant(gE[(int64_t)u * Q + q]);
        }
        // edge_gain_t's operations in its order, with |P| = |Q| = 1
        const double dsv = 1.0, dsu = 1.0;
        const double num = dsv * dsu;
        const double den = dsv + dsu;
        const double f = num / den;
        double ss = 0.0;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const float e4[4] = {x[q].x, x[q].y, x[q].z, x[q].w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const double diff = mv[4 * q + c] - (double)e4[c];
            const double sq = diff * diff;
            ss = ss + sq;
          }
        }
        ss = ss * sIF2;  // exact: a power of two
        const double cut = lambda * (double)w;
        const double fit = f * ss;
        const double g = cut - fit;
        if (g > 0.0 || small) {
          if (b.u < 0 || g > b.g) {
            b = Best{g, -1, u};
          } else if (g == b.g) {
            if (b.mp < 0) b.mp = node_minpt<true>(s, b.u);
            const int32_t mp = node_minpt<true>(s, u);
            if (mp < b.mp) b = Best{g, mp, u};
          }
        }
      });
      if (b.u >= 0 && b.mp < 0) b.mp = node_minpt<true>(s, b.u);
    }
    if constexpr (G > 1) {
#pragma unroll
      for (int off = G / 2; off > 0; off >>= 1) {
        Best o;
        o.g = __shfl_xor(b.g, off, kWave);
        o.mp = __shfl_xor(b.mp, off, kWave);
        o.u = __shfl_xor(b.u, off, kWave);
        if (best_before(o, b)) b = o;
        cnt += __shfl_xor(cnt, off, kWave);
      }
    }
    if (live && lg == 0) {
      target[v] = b.u;
      deg[v] = cnt;
      chose |= b.u >= 0;
    }
  }
  if (__ballot(chose) && (threadIdx.x & (kWave - 1)) == 0) ctl->any_choice = 1;
}

// Steps 1-2 over the chunks of the long rows, a wave per chunk.
template <bool FIRST, int DT>
__global__ __launch_bounds__(256) void k_select_long(
    int32_t nn, Adj a, NodeIn s, int32_t d, double lambda, int64_t smin,
    LongWork lw, Ctl *ctl) {
  const int32_t n_items = ctl->n_lchunk;
  const int F = ctl->F;
  const double sF = ldexp(1.0, F), sIF = ldexp(1.0, -F);
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t wave0 = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                                  threadIdx.x / kWave);
  const int32_t nwaves = (int32_t)(gridDim.x * (blockDim.x / kWave));
  for (int32_t it = wave0; it < n_items; it += nwaves) {
    const int32_t slot = lw.item[it];
    const int32_t v = lw.rows[slot];
    if ((uint32_t)v >= (uint32_t)nn) {
      raise_err(ctl, kErrInternal);
      continue;
    }
    const int32_t j0 = (it - lw.base[slot]) * kLongChunk;
    const int32_t j1 = min(row_span<FIRST>(a, v), j0 + kLongChunk);
    const int32_t rb = row_base<FIRST>(a, v);
    const int32_t sv = node_size<FIRST>(s, v);
    const double dsv = (double)sv;
    const bool small = (int64_t)sv < smin;
    MeanRow<FIRST, DT> mv;
    mv.load(s, v, sF, sIF);
    Best b{0.0, 0, -1};
    int32_t cnt = 0;
    for (int32_t j = j0 + lane; j < j1; j += kWave) {
      int32_t u, w;
      if (!row_entry_at<FIRST>(a, v, rb, j, u, w)) continue;
      ++cnt;
      if ((uint32_t)u >= (uint32_t)nn) {
        raise_err(ctl, kErrInternal);
        continue;
      }
      const double g =
          edge_gain_t<FIRST, DT>(s, mv, v, dsv, u, w, d, lambda, sF, sIF);
      if (g > 0.0 || small) {
        const Best c{g, node_minpt<FIRST>(s, u), u};
        if (best_before(c, b)) b = c;
      }
    }
    cnt = wave_sum(cnt);
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      Best o;
      o.g = __shfl_xor(b.g, off, kWave);
      o.mp = __shfl_xor(b.mp, off, kWave);
      o.u = __shfl_xor(b.u, off, kWave);
      if (best_before(o, b)) b = o;
    }
    if (lane == 0) {
      lw.g[it] = b.g;
      lw.mp[it] = b.mp;
      lw.u[it] = b.u;
      lw.cnt[it] = cnt;
    }
  }
}

// The long rows' choices from their chunks (same order as best_before).
// A wave per long row: the lanes take every 64th chunk, then the wave
// reduces (a giant component's row has hundreds of chunks).
__global__ __launch_bounds__(256) void k_select_combine(
    LongWork lw, int32_t *__restrict__ target, int32_t *__restrict__ deg,
    Ctl *ctl) {
  const int32_t n_long = ctl->n_long;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t wave0 = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                                  threadIdx.x / kWave);
  const int32_t nwaves = (int32_t)(gridDim.x * (blockDim.x / kWave));
  for (int32_t slot = wave0; slot < n_long; slot += nwaves) {
    const int32_t b0 = lw.base[slot], nch = lw.nch[slot];
    Best b{0.0, 0, -1};
    int32_t cnt = 0;
    for (int32_t c = b0 + lane; c < b0 + nch; c += kWave) {
      const Best o{lw.g[c], lw.mp[c], lw.u[c]};
      if (best_before(o, b)) b = o;
      cnt += lw.cnt[c];
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      Best o;
      o.g = __shfl_xor(b.g, off, kWave);
      o.mp = __shfl_xor(b.mp, off, kWave);
      o.u = __shfl_xor(b.u, off, kWave);
      if (best_before(o, b)) b = o;
      cnt += __shfl_xor(cnt, off, kWave);
    }
    if (lane == 0) {
      const int32_t v = lw.rows[slot];
      target[v] = b.u;
      deg[v] = cnt;
      if (b.u >= 0) ctl->any_choice = 1;
    }
  }
}

// ---------------------------------------------------------------------------
// Step 3: merge graph -> forest -> components
// ---------------------------------------------------------------------------

// A node points to its choice, except the lower end of a mutual pair, which
// becomes a root.  Always writes every parent.
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

// Pointer jumping, first pass: each thread walks from its node towards the
// root, reading parents that other threads may already have moved closer to
// their roots (every value read is an ancestor, so the walk only shortens).
// A walk stops after kJumpWalk steps: a long chain (a line of points in
// index order with tied gains makes one of length n) would otherwise cost
// n dependent loads per thread.  A stopped walk keeps the ancestor it
// reached and marks the round unfinished (any_choice = -1), so that the
// round's later kernels wait; the host then completes the forest with
// pointer-doubling passes (k_double) and launches them again.
// A block stages the parents of its kJumpR consecutive nodes in LDS: a
// node's choice is a neighbour, mostly in the same block of Morton order,
// so most steps read LDS, and only a step out of the block reads global
// memory.  The staged values and the block's own updates are ancestors
// too, and a root's entry is itself in both copies.
constexpr int kJumpR = 512;  // (two passes: faster than blocks of 1024)
__global__ __launch_bounds__(256) void k_jump(int32_t nn, int32_t *parent,
                                              Ctl *ctl) {
  __shared__ int32_t sp[kJumpR];
  const int32_t lo = xcd_block() * kJumpR;
  if (lo >= nn) return;  // the whole block
  const int32_t nr = min(kJumpR, nn - lo);
  for (int32_t q = threadIdx.x; q < nr; q += blockDim.x) sp[q] = parent[lo + q];
  __syncthreads();
  bool deep = false;
  for (int32_t r = threadIdx.x; r < nr; r += blockDim.x) {
    const int32_t v = lo + r;
    int32_t p = sp[r];
    int it = 0;
    for (; it < kJumpWalk; ++it) {
      if ((uint32_t)p >= (uint32_t)nn) {
        raise_err(ctl, kErrInternal);
        p = v;
        break;
      }
      const uint32_t rp = (uint32_t)(p - lo);
      const int32_t pp = rp < (uint32_t)nr
                             ? __atomic_load_n(&sp[rp], __ATOMIC_RELAXED)
                             : __atomic_load_n(&parent[p], __ATOMIC_RELAXED);
      if (pp == p) break;
      p = pp;
    }
    __atomic_store_n(&sp[r], p, __ATOMIC_RELAXED);
    __atomic_store_n(&parent[v], p, __ATOMIC_RELAXED);
    deep |= it == kJumpWalk;
  }
  if (deep) __atomic_store_n(&ctl->any_choice, -1, __ATOMIC_RELAXED);
}

// One pointer-doubling pass: parent[v] = parent[parent[v]].  Values read
// concurrently are ancestors at least as high as the pass would see in
// lockstep, so every pass at least halves the remaining depth, and
// ceil(log2 depth) passes reach the roots.  jump_changed records whether
// any parent moved.
__global__ __launch_bounds__(256) void k_double(int32_t nn, int32_t *parent,
                                                Ctl *ctl) {
  const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= nn) return;
  const int32_t p = parent[v];
  if ((uint32_t)p >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
  const int32_t pp = __atomic_load_n(&parent[p], __ATOMIC_RELAXED);
  if (pp != p) {
    __atomic_store_n(&parent[v], pp, __ATOMIC_RELAXED);
    ctl->jump_changed = 1;
  }
}

// Starts a round of doubling passes (jump_changed = 0); with done set, marks
// the forest complete so the round's later kernels run (any_choice = 1).
__global__ void k_jump_state(Ctl *ctl, int done) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    if (done) ctl->any_choice = 1;
    else ctl->jump_changed = 0;
  }
}

// Roots numbered in node order; the pass also clears the member counters
// of the next components (c < n_next <= nn).
struct ScanRoots {
  const int32_t *parent;
  int32_t *newid;
  int32_t *cnt;
  int32_t nn;
  __device__ int32_t value(int32_t v) const {
    return (v < nn && parent[v] == v) ? 1 : 0;
  }
  __device__ void emit(int32_t v, int32_t excl, int32_t val) const {
    if (val) newid[v] = excl;
    if (v < nn) cnt[v] = 0;
  }
};

// Window offsets of the next table (exclusive scan of the capacities, the
// total at [len]) and the first component of every contraction chunk:
// cstart[q] = the first c with toff[c] >= q * chunk, for q = 0 ..
// ceil(slots / chunk).  Component i takes the q with q * chunk in
// (toff[i], toff[i + 1]] (they start at component i + 1); q = 0 starts at 0
// and a last partial chunk at len.
struct ScanWindows {
  const int32_t *cap;
  int32_t *toff;
  const int32_t *n_dev;
  int32_t *cstart;
  int32_t chunk, qcap;
  Ctl *ctl;
  __device__ int32_t value(int32_t i) const {
    return (i < *n_dev) ? cap[i] : 0;
  }
  __device__ void put(int32_t q, int32_t c) const {
    if ((uint32_t)q < (uint32_t)qcap) cstart[q] = c;
    else raise_err(ctl, kErrInternal);
  }
  __device__ void emit(int32_t i, int32_t excl, int32_t v) const {
    if (!round_live(ctl)) return;  // nothing merged: capacities are stale
    const int32_t len = *n_dev;
    if (i > len) return;
    toff[i] = excl;
    if (i == 0) put(0, 0);
    if (i < len) {
      for (int32_t q = excl / chunk + 1; q <= (excl + v) / chunk; ++q)
        put(q, i + 1);
    } else if (excl % chunk != 0) {
      put(excl / chunk + 1, len);
    }
  }
};

// Component of every node and its place among the component's members.
// Nodes of one component mostly sit together in node order, so the lanes
// of a wave are grouped by component (ballot per distinct value) and each
// group takes its places with one atomic, made by its lowest lane.
__global__ __launch_bounds__(256) void k_assign(int32_t nn,
                                                const int32_t *parent,
                                                const int32_t *newid,
                                                int32_t *L, int32_t *cnt,
                                                int32_t *rank, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t v = xcd_tid();
  const bool act = v < nn;
  int32_t c = -1;
  if (act) {
    const int32_t r = parent[v];
    c = 0;
    if ((uint32_t)r < (uint32_t)nn) {
      c = newid[r];
    } else {
      raise_err(ctl, kErrInternal);
    }
    if ((uint32_t)c >= (uint32_t)ctl->n_next) {
      raise_err(ctl, kErrInternal);
      c = 0;
    }
    L[v] = c;
  }
  const int lane = threadIdx.x & (kWave - 1);
  uint64_t todo = __ballot(act);
  uint64_t mine = 0;
  int leader = 0;
  while (todo) {
    const int l = __builtin_ctzll(todo);
    const int32_t cl = __shfl(c, l, kWave);
    const uint64_t m = __ballot(c == cl) & todo;
    if ((m >> lane) & 1) {
      mine = m;
      leader = l;
    }
    todo &= ~m;
  }
  int32_t base = 0;
  if (act && lane == leader) base = atomicAdd(&cnt[c], __popcll(mine));
  base = __shfl(base, leader, kWave);
  if (act) rank[v] = base + __popcll(mine & ((1ull << lane) - 1));
}

// Members in component order; the first member of each component also
// writes the next round's merged flag (a component of more than one
// member), so every component's flag is written once.
__global__ __launch_bounds__(256) void k_place(int32_t nn, const int32_t *L,
                                               const int32_t *moff,
                                               const int32_t *rank,
                                               int32_t *mem, uint8_t *merged,
                                               Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t v = xcd_tid();
  if (v >= nn) return;
  const int32_t c = L[v];
  const int32_t r = rank[v];
  const int32_t m0 = moff[c];
  const int32_t pos = m0 + r;
  if ((uint32_t)pos < (uint32_t)nn) {
    mem[pos] = v;
    if (r == 0) merged[c] = (moff[c + 1] - m0 > 1) ? 1 : 0;
  } else {
    raise_err(ctl, kErrInternal);
  }
}

// ---------------------------------------------------------------------------
// Step 4 statistics, gathered from the members of each component
// ---------------------------------------------------------------------------
struct NodeOut {
  int32_t *size;
  int64_t *S;
  double *mu;
  int32_t *minpt;
  int32_t *cap;   // summed member degree = window of the next table
  int32_t *wl;    // row length (the window until a chunk compacts it)
  int32_t *cbig;  // components whose window exceeds one chunk
  int32_t chunk;  // slots per contraction chunk (at most kChunk)
  int32_t big_members;  // components with more members take a block
  int32_t *tile_c, *tile_i;  // member tiles of the large windows
};

// Records the window of component c; a window larger than a chunk goes to
// the global path, split into tiles of kBatch members.
// A window larger than an LDS chunk is filled with global atomics: it gets
// twice its summed degree, so open addressing stays at load factor <= 1/2.
__device__ __forceinline__ void note_window(const NodeOut &o, int32_t c,
                                            int32_t cap, int32_t members,
                                            Ctl *ctl) {
  if (cap > o.chunk) cap *= 2;
  o.cap[c] = cap;
  o.wl[c] = cap;
  if (cap > o.chunk) {
    o.cbig[atomicAdd(&ctl->n_cbig, 1)] = c;
    const int32_t tiles = (members + kBatch - 1) / kBatch;
    const int32_t t0 = atomicAdd(&ctl->n_tiles, tiles);
    for (int32_t t = 0; t < tiles; ++t) {
      o.tile_c[t0 + t] = c;
      o.tile_i[t0 + t] = t;
    }
  }
}

constexpr int kDimChunk = 8;

template <bool FIRST, int DT>
__global__ __launch_bounds__(256) void k_stats(
    int32_t bound, const int32_t *__restrict__ mem,
    const int32_t *__restrict__ moff, NodeIn s,
    const int32_t *__restrict__ deg, int32_t d, NodeOut o,
    int32_t *__restrict__ big, Ctl *ctl) {
  if (!round_live(ctl)) return;
  int32_t c;
  if (!xcd_item(min(bound, ctl->n_next), c)) return;
  const int32_t m0 = moff[c], m1 = moff[c + 1];
  if (m1 - m0 > o.big_members) {
    big[atomicAdd(&ctl->n_big, 1)] = c;
    return;
  }
  const double sF = ldexp(1.0, ctl->F), sIF = ldexp(1.0, -ctl->F);
  int32_t size = 0, mp = INT32_MAX, cap = 0;
  for (int32_t j = m0; j < m1; ++j) {
    const int32_t m = mem[j];
    size += node_size<FIRST>(s, m);
    mp = min(mp, node_minpt<FIRST>(s, m));
    cap += deg[m];
  }
  o.size[c] = size;
  o.minpt[c] = mp;
  note_window(o, c, cap, m1 - m0, ctl);
  const double dsz = (double)size;
  if constexpr (DT > 0) {
    int64_t acc[DT];
#pragma unroll
    for (int q = 0; q < DT; ++q) acc[q] = 0;
    for (int32_t j = m0; j < m1; ++j) {
      const int32_t m = mem[j];
      if (FIRST) {
        const float4 *p =
            reinterpret_cast<const float4 *>(s.emb + (int64_t)m * DT);
#pragma unroll
        for (int q = 0; q < DT / 4; ++q) {
          const float4 x = p[q];
          acc[4 * q + 0] += (int64_t)rint((double)x.x * sF);
          acc[4 * q + 1] += (int64_t)rint((double)x.y * sF);
          acc[4 * q + 2] += (int64_t)rint((double)x.z * sF);
          acc[4 * q + 3] += (int64_t)rint((double)x.w * sF);
        }
      } else {
        const longlong2 *p =
            reinterpret_cast<const longlong2 *>(s.S + (int64_t)m * DT);
#pragma unroll
        for (int q = 0; q < DT / 2; ++q) {
          const longlong2 x = p[q];
          acc[2 * q + 0] += x.x;
          acc[2 * q + 1] += x.y;
        }
      }
    }
    longlong2 *So = reinterpret_cast<longlong2 *>(o.S + (int64_t)c * DT);
    double2 *Mo = reinterpret_cast<double2 *>(o.mu + (int64_t)c * DT);
#pragma unroll
    for (int q = 0; q < DT / 2; ++q) {
      So[q] = make_longlong2(acc[2 * q], acc[2 * q + 1]);
      const double q0 = (double)acc[2 * q] / dsz;
      const double q1 = (double)acc[2 * q + 1] / dsz;
      Mo[q] = make_double2(q0 * sIF, q1 * sIF);
    }
    return;
  }
  for (int32_t i0 = 0; i0 < d; i0 += kDimChunk) {
    int64_t acc[kDimChunk];
#pragma unroll
    for (int q = 0; q < kDimChunk; ++q) acc[q] = 0;
    for (int32_t j = m0; j < m1; ++j) {
      const int32_t m = mem[j];
#pragma unroll
      for (int q = 0; q < kDimChunk; ++q)
        if (i0 + q < d) acc[q] += node_S<FIRST>(s, m, i0 + q, d, sF);
    }
#pragma unroll
    for (int q = 0; q < kDimChunk; ++q) {
      if (i0 + q < d) {
        const int64_t t = (int64_t)c * d + i0 + q;
        o.S[t] = acc[q];
        const double qv = (double)acc[q] / dsz;
        o.mu[t] = qv * sIF;
      }
    }
  }
}

// Components with many members: one block each, threads stride over the
// members and the sums are combined in shared memory (integer, so the
// order does not matter).
// Step 4 statistics with G lanes per component (rows of DT values) and the
// row's dimensions split among them: lane lg sums dimensions
// [lg*DT/G, (lg+1)*DT/G) of every member, four members a step, so a
// component of one member, most of them in a level with few merges, keeps
// all G lanes loading, and the loads of a member's row are side by side;
// sizes, smallest points and degrees are summed over every G-th member and
// combined in the group (exact int64, so the order does not matter).
// Components are laid out over the XCDs like xcd_item, in whole groups.
// FIRST: the members are points, their sums rint(e * 2^F) of the fp32
// embedding; later: the members' int64 sums.
template <bool FIRST, int DT, int G>
__global__ __launch_bounds__(256) void k_stats_s(
    int32_t bound, const int32_t *__restrict__ mem,
    const int32_t *__restrict__ moff, NodeIn s,
    const int32_t *__restrict__ deg, NodeOut o,
    int32_t *__restrict__ big, Ctl *ctl) {
  constexpr int kPer = DT / G;  // dimensions per lane
  static_assert(DT % G == 0 && kPer % 2 == 0, "dims per lane");
  constexpr int kU = 4;  // members a step, their loads in flight together
  if (!round_live(ctl)) return;
  const int32_t total = min(bound, ctl->n_next) * G;
  const int32_t per = ((total + kXcd - 1) / kXcd + G - 1) / G * G;
  const int32_t j =
      (int32_t)(blockIdx.x / kXcd) * (int32_t)blockDim.x + (int32_t)threadIdx.x;
  const int32_t sub = (int32_t)(blockIdx.x % kXcd) * per + j;
  if (j >= per || sub >= total) return;  // whole groups
  const int32_t c = sub / G;
  const int lg = sub & (G - 1);
  const int32_t m0 = moff[c], m1 = moff[c + 1];
  if (m1 - m0 > o.big_members) {
    if (lg == 0) big[atomicAdd(&ctl->n_big, 1)] = c;
    return;
  }
  const double sF = ldexp(1.0, ctl->F), sIF = ldexp(1.0, -ctl->F);
  int32_t size = 0, mp = INT32_MAX, cap = 0;
  int64_t acc[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) acc[q] = 0;
  for (int32_t t0 = m0; t0 < m1; t0 += kU) {
    int32_t mm[kU];
#pragma unroll
    for (int e = 0; e < kU; ++e) mm[e] = mem[min(t0 + e, m1 - 1)];
    if constexpr (FIRST) {
      float2 x[kU][kPer / 2];
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const float2 *p = reinterpret_cast<const float2 *>(
            s.emb + (int64_t)mm[e] * DT + lg * kPer);
#pragma unroll
        for (int q = 0; q < kPer / 2; ++q) x[e][q] = p[q];
      }
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const int32_t t = t0 + e;
        if (t >= m1) break;
#pragma unroll
        for (int q = 0; q < kPer / 2; ++q) {
          acc[2 * q + 0] += (int64_t)rint((double)x[e][q].x * sF);
          acc[2 * q + 1] += (int64_t)rint((double)x[e][q].y * sF);
        }
        if ((t - m0) % G == lg) {  // this lane's share of the scalars
          size += 1;
          mp = min(mp, node_minpt<true>(s, mm[e]));
          cap += deg[mm[e]];
        }
      }
    } else {
      longlong2 x[kU][kPer / 2];
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const longlong2 *p = reinterpret_cast<const longlong2 *>(
            s.S + (int64_t)mm[e] * DT + lg * kPer);
#pragma unroll
        for (int q = 0; q < kPer / 2; ++q) x[e][q] = p[q];
      }
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        const int32_t t = t0 + e;
        if (t >= m1) break;
#pragma unroll
        for (int q = 0; q < kPer / 2; ++q) {
          acc[2 * q + 0] += x[e][q].x;
          acc[2 * q + 1] += x[e][q].y;
        }
        if ((t - m0) % G == lg) {  // this lane's share of the scalars
          size += s.size[mm[e]];
          mp = min(mp, s.minpt[mm[e]]);
          cap += deg[mm[e]];
        }
      }
    }
  }
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) {
    size += __shfl_xor(size, off, kWave);
    cap += __shfl_xor(cap, off, kWave);
    mp = min(mp, __shfl_xor(mp, off, kWave));
  }
  if (lg == 0) {
    o.size[c] = size;
    o.minpt[c] = mp;
    note_window(o, c, cap, m1 - m0, ctl);
  }
  const double dsz = (double)size;
  longlong2 *So = reinterpret_cast<longlong2 *>(o.S + (int64_t)c * DT + lg * kPer);
  double2 *Mo = reinterpret_cast<double2 *>(o.mu + (int64_t)c * DT + lg * kPer);
#pragma unroll
  for (int q = 0; q < kPer / 2; ++q) {
    So[q] = make_longlong2(acc[2 * q], acc[2 * q + 1]);
    const double q0 = (double)acc[2 * q] / dsz;
    const double q1 = (double)acc[2 * q + 1] / dsz;
    Mo[q] = make_double2(q0 * sIF, q1 * sIF);
  }
}

// k_stats_big for D = DT: one pass over the members, each thread summing
// whole rows (16-byte loads, two members in flight), then a block
// reduction (exact int64, so the order does not matter).
template <bool FIRST, int DT>
__global__ __launch_bounds__(256) void k_stats_big_t(
    const int32_t *__restrict__ mem, const int32_t *__restrict__ moff,
    NodeIn s, const int32_t *__restrict__ deg, NodeOut o,
    const int32_t *__restrict__ big, Ctl *ctl) {
  static_assert(DT > 0 && DT % 4 == 0, "vector rows");
  constexpr int kU = 2;
  constexpr int NW = 256 / kWave;
  __shared__ long long sS[NW][DT];
  __shared__ int32_t ssize[NW], smp[NW], scap[NW];
  if (!round_live(ctl)) return;
  const double sF = ldexp(1.0, ctl->F), sIF = ldexp(1.0, -ctl->F);
  const int32_t n_big = ctl->n_big;
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  for (int32_t bi = blockIdx.x; bi < n_big; bi += gridDim.x) {
    const int32_t c = big[bi];
    const int32_t m0 = moff[c], m1 = moff[c + 1];
    int64_t acc[DT];
#pragma unroll
    for (int q = 0; q < DT; ++q) acc[q] = 0;
    int32_t size = 0, mp = INT32_MAX, cap = 0;
    for (int32_t j0 = m0 + (int32_t)threadIdx.x; j0 < m1; j0 += kU * 256) {
      int32_t mm[kU];
#pragma unroll
      for (int e = 0; e < kU; ++e) mm[e] = mem[min(j0 + e * 256, m1 - 1)];
      if constexpr (FIRST) {
        float4 x[kU][DT / 4];
#pragma unroll
        for (int e = 0; e < kU; ++e) {
          const float4 *p =
              reinterpret_cast<const float4 *>(s.emb + (int64_t)mm[e] * DT);
#pragma unroll
          for (int q = 0; q < DT / 4; ++q) x[e][q] = p[q];
        }
#pragma unroll
        for (int e = 0; e < kU; ++e) {
          if (j0 + e * 256 >= m1) break;
#pragma unroll
          for (int q = 0; q < DT / 4; ++q) {
            acc[4 * q + 0] += (int64_t)rint((double)x[e][q].x * sF);
            acc[4 * q + 1] += (int64_t)rint((double)x[e][q].y * sF);
            acc[4 * q + 2] += (int64_t)rint((double)x[e][q].z * sF);
            acc[4 * q + 3] += (int64_t)rint((double)x[e][q].w * sF);
          }
          size += 1;
          mp = min(mp, node_minpt<true>(s, mm[e]));
          cap += deg[mm[e]];
        }
      } else {
        longlong2 x[kU][DT / 2];
#pragma unroll
        for (int e = 0; e < kU; ++e) {
          const longlong2 *p =
              reinterpret_cast<const longlong2 *>(s.S + (int64_t)mm[e] * DT);
#pragma unroll
          for (int q = 0; q < DT / 2; ++q) x[e][q] = p[q];
        }
#pragma unroll
        for (int e = 0; e < kU; ++e) {
          if (j0 + e * 256 >= m1) break;
#pragma unroll
          for (int q = 0; q < DT / 2; ++q) {
            acc[2 * q + 0] += x[e][q].x;
            acc[2 * q + 1] += x[e][q].y;
          }
          size += s.size[mm[e]];
          mp = min(mp, s.minpt[mm[e]]);
          cap += deg[mm[e]];
        }
      }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
#pragma unroll
      for (int q = 0; q < DT; ++q)
        acc[q] += (int64_t)__shfl_xor((long long)acc[q], off, kWave);
      size += __shfl_xor(size, off, kWave);
      cap += __shfl_xor(cap, off, kWave);
      mp = min(mp, __shfl_xor(mp, off, kWave));
    }
    if (lane == 0) {
#pragma unroll
      for (int q = 0; q < DT; ++q) sS[wv][q] = (long long)acc[q];
      ssize[wv] = size;
      smp[wv] = mp;
      scap[wv] = cap;
    }
    __syncthreads();
    int32_t tsize = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) tsize += ssize[w];
    if (threadIdx.x == 0) {
      int32_t tmp = INT32_MAX, tcap = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        tmp = min(tmp, smp[w]);
        tcap += scap[w];
      }
      o.size[c] = tsize;
      o.minpt[c] = tmp;
      note_window(o, c, tcap, m1 - m0, ctl);
    }
    if (threadIdx.x < DT) {
      long long v = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += sS[w][threadIdx.x];
      const int64_t t = (int64_t)c * DT + threadIdx.x;
      o.S[t] = v;
      const double qv = (double)v / (double)tsize;
      o.mu[t] = qv * sIF;
    }
    __syncthreads();  // the shared sums are reused by the next component
  }
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_stats_big(
    const int32_t *__restrict__ mem, const int32_t *__restrict__ moff,
    NodeIn s, const int32_t *__restrict__ deg, int32_t d, NodeOut o,
    const int32_t *__restrict__ big, Ctl *ctl) {
  __shared__ unsigned long long sS[64];
  __shared__ int32_t ssize, smp, scap;
  if (!round_live(ctl)) return;
  const double sF = ldexp(1.0, ctl->F), sIF = ldexp(1.0, -ctl->F);
  const int32_t n_big = ctl->n_big;
  for (int32_t bi = blockIdx.x; bi < n_big; bi += gridDim.x) {
    const int32_t c = big[bi];
    const int32_t m0 = moff[c], m1 = moff[c + 1];
    for (int t = threadIdx.x; t < 64; t += blockDim.x) sS[t] = 0ull;
    if (threadIdx.x == 0) {
      ssize = 0;
      smp = INT32_MAX;
      scap = 0;
    }
    __syncthreads();
    int32_t size = 0, mp = INT32_MAX, cap = 0;
    for (int32_t j = m0 + threadIdx.x; j < m1; j += blockDim.x) {
      const int32_t m = mem[j];
      size += node_size<FIRST>(s, m);
      mp = min(mp, node_minpt<FIRST>(s, m));
      cap += deg[m];
    }
    atomicAdd(&ssize, size);
    atomicMin(&smp, mp);
    atomicAdd(&scap, cap);
    for (int32_t i0 = 0; i0 < d; i0 += kDimChunk) {
      int64_t acc[kDimChunk];
#pragma unroll
      for (int q = 0; q < kDimChunk; ++q) acc[q] = 0;
      for (int32_t j = m0 + threadIdx.x; j < m1; j += blockDim.x) {
        const int32_t m = mem[j];
#pragma unroll
        for (int q = 0; q < kDimChunk; ++q)
          if (i0 + q < d) acc[q] += node_S<FIRST>(s, m, i0 + q, d, sF);
      }
#pragma unroll
      for (int q = 0; q < kDimChunk; ++q) {
        if (i0 + q < d) {
          const long long r = wave_sum((long long)acc[q]);
          if ((threadIdx.x & (kWave - 1)) == 0)
            atomicAdd(&sS[i0 + q], (unsigned long long)r);
        }
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      o.size[c] = ssize;
      o.minpt[c] = smp;
      note_window(o, c, scap, m1 - m0, ctl);
    }
    for (int32_t i = threadIdx.x; i < d; i += blockDim.x) {
      const int64_t t = (int64_t)c * d + i;
      const int64_t v = (int64_t)sS[i];
      o.S[t] = v;
      const double qv = (double)v / (double)ssize;
      o.mu[t] = qv * sIF;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Step 4 contraction into the next table.  Component A owns the slots
// [toff[A], toff[A] + cap[A]); cap[A], the summed degree of its members,
// bounds its distinct neighbours, so open addressing always finds a slot.
//
// Chunks: block j takes the components whose window starts in
// [j*kChunk, (j+1)*kChunk) and whose window is at most kChunk slots; their
// windows lie inside 2*kChunk slots from j*kChunk, which the block keeps in
// LDS.  It walks their members' rows in batches of 256 members (the entries
// of a batch are spread over all threads), adds every relabelled edge to
// the LDS window of its component (parallel edges add their weights,
// edges inside a component are dropped), then writes each row compacted to
// the start of its window.  Larger windows go through the global path.
// ---------------------------------------------------------------------------
// Loads a batch of members into LDS with the exclusive prefix of their row
// spans (members of skipped components count 0); returns the entry total.
template <bool FIRST, class Keep>
__device__ __forceinline__ int32_t load_batch(const Adj &a,
                                              const int32_t *__restrict__ mem,
                                              int32_t idx0, int32_t idx1,
                                              int32_t *pre, int32_t *bm,
                                              int32_t *wsum, Keep &&keep) {
  const int32_t idx = idx0 + (int32_t)threadIdx.x;
  int32_t m = -1, span = 0;
  if (idx < idx1) {
    m = mem[idx];
    if (keep(m)) span = row_span<FIRST>(a, m);
  }
  int32_t total;
  const int32_t excl = block_excl_scan<256>(span, wsum, &total);
  pre[threadIdx.x] = excl;
  bm[threadIdx.x] = m;
  if (threadIdx.x == 0) pre[kBatch] = total;
  __syncthreads();
  return total;
}

// Members and entries of U flat indices f[e] of the batch: the U searches
// over pre[0..kBatch) take their (fixed) steps together, so each step's LDS
// reads are issued back to back.
template <int U>
__device__ __forceinline__ void batch_find_n(const int32_t *pre,
                                             const int32_t (&f)[U],
                                             int32_t (&slot)[U],
                                             int32_t (&j)[U]) {
#pragma unroll
  for (int e = 0; e < U; ++e) slot[e] = 0;
#pragma unroll
  for (int32_t len = kBatch; len > 1;) {
    const int32_t half = len >> 1;
#pragma unroll
    for (int e = 0; e < U; ++e)
      slot[e] = pre[slot[e] + half] <= f[e] ? slot[e] + half : slot[e];
    len -= half;
  }
#pragma unroll
  for (int e = 0; e < U; ++e) j[e] = f[e] - pre[slot[e]];
}


// Start slot of key B in a window of cap slots: the multiplicative hash
// scaled into [0, cap) by the high half of a 32x32 product (one
// instruction, where a remainder by a variable takes a dozen).
__device__ __forceinline__ uint32_t window_slot(int32_t B, int32_t cap) {
  return __umulhi((uint32_t)B * 2654435761u, (uint32_t)cap);
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_contract_chunk(
    int32_t nn, Adj a, const int32_t *__restrict__ L,
    const int32_t *__restrict__ mem, const int32_t *__restrict__ moff,
    const int32_t *__restrict__ toff, const int32_t *__restrict__ cap,
    const int32_t *__restrict__ cstart, uint64_t *__restrict__ tbl,
    int32_t *__restrict__ wl, int32_t chunk, Ctl *ctl) {
  __shared__ int32_t kb[2 * kChunk];
  __shared__ int32_t kw[2 * kChunk];
  __shared__ int32_t pre[kBatch + 1];
  // members of the batch: node, component, window start in the chunk,
  // window capacity, row base
  __shared__ int32_t bm[kBatch], bA[kBatch], blb[kBatch], bcp[kBatch];
  __shared__ int32_t bbase[kBatch];
  __shared__ int32_t wsum[256 / kWave];
  if (!round_live(ctl)) return;
  // chunks q = this block's, then every gridDim.x-th: the grid is sized for
  // the entries, the windows may span up to twice as many slots
  const int32_t slots = ctl->slots;
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t below = (1ull << lane) - 1;
  int32_t uniq = 0;
  for (int32_t q = xcd_block(); (int64_t)q * chunk < slots; q += gridDim.x) {
    const int32_t j0 = q * chunk;
    // components whose windows start in [j0, j0 + chunk)
    const int32_t c_lo = cstart[q], c_hi = cstart[q + 1];
    for (int t = threadIdx.x; t < 2 * chunk; t += blockDim.x) {
      kb[t] = -1;
      kw[t] = 0;
    }
    __syncthreads();
    const int32_t m_lo = moff[c_lo];
    // a window larger than a chunk can only be the last one starting here
    // (the next window starts past the chunk); its members are not walked
    const int32_t m_hi =
        (c_hi > c_lo && cap[c_hi - 1] > chunk) ? moff[c_hi - 1] : moff[c_hi];
    constexpr int kUnroll = 4;  // entries per thread with their loads in flight
    // entry (slot, u, w) of the batch into its component's LDS window
    auto insert = [&](bool ok, int32_t sl, int32_t B, int32_t w) {
      const int32_t A = ok ? bA[sl] : -1;
      if (!ok || A == B) return;  // edge inside a merged component
      const int32_t lb = blb[sl], cp = bcp[sl];
      uint32_t h = window_slot(B, cp);
      int32_t probe = 0;
      for (; probe < cp; ++probe) {
        const int32_t old = atomicCAS(&kb[lb + h], -1, B);
        if (old == -1 || old == B) {
          atomicAdd(&kw[lb + h], w);
          break;
        }
        h = (h + 1 == (uint32_t)cp) ? 0u : h + 1;
      }
      if (probe == cp) raise_err(ctl, kErrInternal);
    };
    for (int32_t b0 = m_lo; b0 < m_hi; b0 += kBatch) {
      const int32_t idx = b0 + (int32_t)threadIdx.x;
      int32_t span = 0;
      bool take = false;
      if (idx < m_hi) {
        const int32_t m = mem[idx];
        // the row's span and base depend on m only: loaded with L[m]
        const int32_t sp = row_span<FIRST>(a, m);
        const int32_t rb = row_base<FIRST>(a, m);
        const int32_t A = L[m];
        const int32_t cp = cap[A];
        const int32_t lb = toff[A] - j0;
        if (cp > 0 && cp <= chunk) {
          if (lb < 0 || lb + cp > 2 * chunk) {
            raise_err(ctl, kErrInternal);
          } else {
            take = true;
            // first round: the k forward entries go by position (slot =
            // entry / k), only the reverse lists by search
            span = FIRST ? sp - a.k : sp;
            bm[threadIdx.x] = m;
            bA[threadIdx.x] = A;
            blb[threadIdx.x] = lb;
            bcp[threadIdx.x] = cp;
            bbase[threadIdx.x] = rb;
          }
        }
      }
      if (FIRST && !take) bA[threadIdx.x] = -1;  // no forward entries
      int32_t total;
      pre[threadIdx.x] = block_excl_scan<256>(span, wsum, &total);
      if (threadIdx.x == 0) pre[kBatch] = total;
      __syncthreads();
      if constexpr (FIRST) {
        const int32_t nsl = min(kBatch, m_hi - b0);
        const int32_t kf = a.k, totf = nsl * kf;
        // f / k as a multiply-high: ceil(2^32 / k) is exact for f * k < 2^32
        const uint32_t kmag = 0xffffffffu / (uint32_t)kf + 1u;
        for (int32_t f0 = threadIdx.x; f0 < totf; f0 += kUnroll * 256) {
          int32_t sl[kUnroll], u[kUnroll], B[kUnroll];
          bool ok[kUnroll];
#pragma unroll
          for (int e = 0; e < kUnroll; ++e) {
            const int32_t f = min(f0 + e * 256, totf - 1);
            sl[e] = kf == 1 ? f : (int32_t)__umulhi((uint32_t)f, kmag);
            const int32_t j = f - sl[e] * kf;
            ok[e] = f0 + e * 256 < totf && bA[sl[e]] >= 0;
            u[e] = ok[e] ? a.nbr[(int64_t)bm[sl[e]] * a.kp + j] : -1;
          }
#pragma unroll
          for (int e = 0; e < kUnroll; ++e) {
            ok[e] = ok[e] && u[e] >= 0;
            if (ok[e] && (uint32_t)u[e] >= (uint32_t)nn) {
              raise_err(ctl, kErrInternal);
              ok[e] = false;
            }
            B[e] = ok[e] ? L[u[e]] : -1;
          }
#pragma unroll
          for (int e = 0; e < kUnroll; ++e) insert(ok[e], sl[e], B[e], 1);
        }
      }
      for (int32_t f0 = threadIdx.x; f0 < total; f0 += kUnroll * 256) {
        int32_t slot[kUnroll], u[kUnroll], w[kUnroll], B[kUnroll];
        int32_t fe[kUnroll], je[kUnroll];
        bool ok[kUnroll];
  #pragma unroll
        for (int e = 0; e < kUnroll; ++e) fe[e] = min(f0 + e * 256, total - 1);
        batch_find_n<kUnroll>(pre, fe, slot, je);
  #pragma unroll
        for (int e = 0; e < kUnroll; ++e) {
          ok[e] = false;
          if (f0 + e * 256 < total)  // (first round: reverse entry je)
            ok[e] = row_entry_at<FIRST>(a, bm[slot[e]], bbase[slot[e]],
                                        FIRST ? a.k + je[e] : je[e], u[e],
                                        w[e]);
        }
  #pragma unroll
        for (int e = 0; e < kUnroll; ++e) {
          if (ok[e] && (uint32_t)u[e] >= (uint32_t)nn) {
            raise_err(ctl, kErrInternal);
            ok[e] = false;
          }
          B[e] = ok[e] ? L[u[e]] : -1;
        }
  #pragma unroll
        for (int e = 0; e < kUnroll; ++e) insert(ok[e], slot[e], B[e], w[e]);
      }
      __syncthreads();
    }
    // rows compacted to the start of their windows, a wave per window:
    // occupied slots ranked by ballot, written in slot order
    for (int32_t c = c_lo + (int32_t)threadIdx.x / kWave; c < c_hi;
         c += blockDim.x / kWave) {
      const int32_t cp = cap[c];
      if (cp <= 0 || cp > chunk) continue;
      const int32_t base = toff[c], lb = base - j0;
      int32_t out = 0;
      for (int32_t t0 = 0; t0 < cp; t0 += kWave) {
        const int32_t t = t0 + lane;
        const int32_t B = t < cp ? kb[lb + t] : -1;
        const uint64_t occ = __ballot(B >= 0);
        if (B >= 0)
          tbl[base + out + __popcll(occ & below)] =
              ((uint64_t)(uint32_t)B << 32) | (uint32_t)kw[lb + t];
        out += __popcll(occ);
      }
      if (lane == 0) {
        wl[c] = out;
        uniq += out;
      }
    }
    __syncthreads();  // the LDS table is reused by the next chunk
  }
  int32_t tot;
  block_excl_scan<256>(uniq, wsum, &tot);
  if (threadIdx.x == 0 && tot) stripe_add(ctl->e_next_s, tot);
}

// Global path for windows larger than a chunk: the window is cleared, then
// tiles of 256 members are pre-aggregated in an LDS table (one component per
// tile, keyed by neighbour) and flushed into the window with atomics.  Rows
// keep their empty slots.
__global__ __launch_bounds__(256) void k_clear_big(
    const int32_t *__restrict__ cbig, const int32_t *__restrict__ toff,
    const int32_t *__restrict__ cap, uint64_t *tbl, int32_t tcap, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t nb = ctl->n_cbig;
  for (int32_t bi = blockIdx.x; bi < nb; bi += gridDim.x) {
    const int32_t c = cbig[bi];
    const int32_t base = toff[c], cp = cap[c];
    if (base < 0 || base + cp > tcap) {
      raise_err(ctl, kErrInternal);
      continue;
    }
    for (int32_t t = threadIdx.x; t < cp; t += blockDim.x)
      tbl[base + t] = kEmpty;
  }
}

// Adds weight w of the edge A -> B to A's window (slots base + base64 ..
// + cap); true for a new slot.
__device__ __forceinline__ bool table_add(uint64_t *tbl, int32_t base,
                                          int32_t cap, int32_t B, int32_t w,
                                          Ctl *ctl, int64_t base64 = 0) {
  uint32_t h = window_slot(B, cap);
  const unsigned long long mine =
      ((unsigned long long)(uint32_t)B << 32) | (uint32_t)w;
  for (int32_t probe = 0; probe < cap; ++probe) {
    unsigned long long *slot =
        reinterpret_cast<unsigned long long *>(tbl + base64 + base + h);
    unsigned long long cur = __atomic_load_n(slot, __ATOMIC_RELAXED);
    if (cur == kEmpty) {
      cur = atomicCAS(slot, kEmpty, mine);
      if (cur == kEmpty) return true;
    }
    if ((int32_t)(cur >> 32) == B) {
      atomicAdd(slot, (unsigned long long)(uint32_t)w);
      return false;
    }
    h = (h + 1 == (uint32_t)cap) ? 0u : h + 1;
  }
  raise_err(ctl, kErrInternal);
  return false;
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_contract_big(
    int32_t nn, Adj a, const int32_t *__restrict__ L,
    const int32_t *__restrict__ mem, const int32_t *__restrict__ moff,
    const int32_t *__restrict__ toff, const int32_t *__restrict__ cap,
    const int32_t *__restrict__ tile_c, const int32_t *__restrict__ tile_i,
    uint64_t *tbl, int32_t tcap, Ctl *ctl) {
  __shared__ int32_t pk[kPreSlots];
  __shared__ int32_t pw[kPreSlots];
  __shared__ int32_t pre[kBatch + 1];
  __shared__ int32_t bm[kBatch];
  __shared__ int32_t wsum[256 / kWave];
  if (!round_live(ctl)) return;
  const int32_t n_tiles = ctl->n_tiles;
  int32_t added = 0;
  for (int32_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
    const int32_t A = tile_c[t];
    for (int q = threadIdx.x; q < kPreSlots; q += blockDim.x) {
      pk[q] = -1;
      pw[q] = 0;
    }
    __syncthreads();
    const int32_t base = toff[A], cp = cap[A];
    if (base < 0 || cp <= 0 || base + cp > tcap) {
      raise_err(ctl, kErrInternal);
      __syncthreads();
      continue;
    }
    const int32_t i0 = moff[A] + tile_i[t] * kBatch;
    const int32_t i1 = min(moff[A + 1], i0 + kBatch);
    // long rows (listed with their chunks in the select) are contracted
    // chunk by chunk by k_contract_long
    const int32_t total = load_batch<FIRST>(
        a, mem, i0, i1, pre, bm, wsum,
        [&](int32_t m) { return row_span<FIRST>(a, m) <= kLongRow; });
    constexpr int kU = 4;  // entries per thread with their loads in flight
    for (int32_t f0 = threadIdx.x; f0 < total; f0 += kU * 256) {
      int32_t fe[kU], slot[kU], je[kU], u[kU], w[kU], B[kU];
      bool ok[kU];
#pragma unroll
      for (int e = 0; e < kU; ++e) fe[e] = min(f0 + e * 256, total - 1);
      batch_find_n<kU>(pre, fe, slot, je);
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        ok[e] = f0 + e * 256 < total &&
                row_entry<FIRST>(a, bm[slot[e]], je[e], u[e], w[e]);
        if (ok[e] && (uint32_t)u[e] >= (uint32_t)nn) {
          raise_err(ctl, kErrInternal);
          ok[e] = false;
        }
      }
#pragma unroll
      for (int e = 0; e < kU; ++e) B[e] = ok[e] ? L[u[e]] : A;
#pragma unroll
      for (int e = 0; e < kU; ++e) {
        if (B[e] == A) continue;  // no entry, or inside the component
        uint32_t h = ((uint32_t)B[e] * 2654435761u) & (kPreSlots - 1);
        bool done = false;
        for (int32_t probe = 0; probe < 32 && !done; ++probe) {
          const int32_t old = atomicCAS(&pk[h], -1, B[e]);
          if (old == -1 || old == B[e]) {
            atomicAdd(&pw[h], w[e]);
            done = true;
          }
          h = (h + 1) & (kPreSlots - 1);
        }
        if (!done) added += table_add(tbl, base, cp, B[e], w[e], ctl) ? 1 : 0;
      }
    }
    __syncthreads();
    for (int q = threadIdx.x; q < kPreSlots; q += blockDim.x)
      if (pk[q] >= 0) added += table_add(tbl, base, cp, pk[q], pw[q], ctl);
    __syncthreads();
  }
  added = wave_sum(added);
  if ((threadIdx.x & (kWave - 1)) == 0 && added)
    stripe_add(ctl->e_next_s, added);
}

// The chunks of long rows whose component has a window larger than an LDS
// chunk: a block per chunk item, pre-aggregated in LDS (a chunk has fewer
// entries than the LDS table has slots), then added to the window.
template <bool FIRST>
__global__ __launch_bounds__(256) void k_contract_long(
    int32_t nn, Adj a, const int32_t *__restrict__ L,
    const int32_t *__restrict__ toff, const int32_t *__restrict__ cap,
    int32_t chunk, LongWork lw, uint64_t *tbl, int32_t tcap, Ctl *ctl) {
  static_assert(kLongChunk <= kPreSlots / 2, "a chunk fits the LDS table");
  __shared__ int32_t pk[kPreSlots];
  __shared__ int32_t pw[kPreSlots];
  if (!round_live(ctl)) return;
  const int32_t n_items = ctl->n_lchunk;
  int32_t added = 0;
  for (int32_t it = blockIdx.x; it < n_items; it += gridDim.x) {
    const int32_t slot = lw.item[it];
    const int32_t v = lw.rows[slot];
    const int32_t A = L[v];
    const int32_t cp = cap[A];
    if (cp <= chunk) continue;  // block-uniform: the LDS path has this row
    const int32_t base = toff[A];
    if (base < 0 || base + cp > tcap) {
      if (threadIdx.x == 0) raise_err(ctl, kErrInternal);
      continue;
    }
    for (int q = threadIdx.x; q < kPreSlots; q += blockDim.x) {
      pk[q] = -1;
      pw[q] = 0;
    }
    __syncthreads();
    const int32_t j0 = (it - lw.base[slot]) * kLongChunk;
    const int32_t j1 = min(row_span<FIRST>(a, v), j0 + kLongChunk);
    const int32_t rb = row_base<FIRST>(a, v);
    for (int32_t j = j0 + (int32_t)threadIdx.x; j < j1; j += blockDim.x) {
      int32_t u, w;
      if (!row_entry_at<FIRST>(a, v, rb, j, u, w)) continue;
      if ((uint32_t)u >= (uint32_t)nn) {
        raise_err(ctl, kErrInternal);
        continue;
      }
      const int32_t B = L[u];
      if (B == A) continue;
      uint32_t h = ((uint32_t)B * 2654435761u) & (kPreSlots - 1);
      for (int32_t probe = 0; probe < kPreSlots; ++probe) {
        const int32_t old = atomicCAS(&pk[h], -1, B);
        if (old == -1 || old == B) {
          atomicAdd(&pw[h], w);
          break;
        }
        h = (h + 1) & (kPreSlots - 1);
      }
    }
    __syncthreads();
    for (int q = threadIdx.x; q < kPreSlots; q += blockDim.x)
      if (pk[q] >= 0) added += table_add(tbl, base, cp, pk[q], pw[q], ctl);
    __syncthreads();
  }
  added = wave_sum(added);
  if ((threadIdx.x & (kWave - 1)) == 0 && added)
    stripe_add(ctl->e_next_s, added);
}

// point -> node map after the first round (internal point i -> node L[i])
__global__ __launch_bounds__(256) void k_compose_first(int32_t n, int32_t *M,
                                                       const int32_t *L,
                                                       Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t i = xcd_tid();
  if (i >= n) return;
  M[i] = L[i];
}

// Later rounds compose a node map instead, over the m nodes the point map
// last pointed to (a fifth of the points after the first round on the
// driving tile): Mn[v] = L[v] in the first such round (INIT), then
// Mn[v] = L[Mn[v]]; nn is the round's node count.
template <bool INIT>
__global__ __launch_bounds__(256) void k_compose_nodes(int32_t m, int32_t nn,
                                                       int32_t *Mn,
                                                       const int32_t *L,
                                                       Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t v = xcd_tid();
  if (v >= m) return;
  const int32_t c = INIT ? v : Mn[v];
  if ((uint32_t)c >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
  Mn[v] = L[c];
}

// The point map brought up to date where it is read (level outputs, the
// tail, the incremental rounds): M[i] = Mn[M[i]].
__global__ __launch_bounds__(256) void k_sync_map(int32_t n, int32_t m,
                                                  int32_t *M,
                                                  const int32_t *Mn,
                                                  Ctl *ctl) {
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const int32_t c = M[i];
  if ((uint32_t)c >= (uint32_t)m) {
    raise_err(ctl, kErrInternal);
    return;
  }
  M[i] = Mn[c];
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

// Point p's superpoint at a level: its node M[inv[p]], through Mt when the
// level ended in the tail (Mt over the nt nodes the tail started from).
__global__ __launch_bounds__(256) void k_labels(int32_t n, int32_t nc,
                                                const int32_t *inv,
                                                const int32_t *M,
                                                const int32_t *Mt, int32_t nt,
                                                const int32_t *minpt,
                                                const int32_t *rank,
                                                int32_t *out, Ctl *ctl) {
  const int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t i = inv ? inv[p] : p;
  int32_t c = ((uint32_t)i < (uint32_t)n) ? M[i] : -1;
  if (Mt) c = ((uint32_t)c < (uint32_t)nt) ? Mt[c] : -1;
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
                                                    const int32_t *Mt,
                                                    int32_t nt,
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
      int32_t c = M[i];
      if (Mt) c = ((uint32_t)c < (uint32_t)nt) ? Mt[c] : -1;
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

// Sum of the weights of all rows (both directions of every edge).
__global__ __launch_bounds__(256) void k_weight_sum(int32_t nn, Adj a,
                                                    Ctl *ctl) {
  long long acc = 0;
  for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < nn;
       v += gridDim.x * blockDim.x)
    for_row<false>(a, v, 0, 1, [&](int32_t, int32_t w) { acc += w; });
  acc = wave_sum(acc);
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
// Tail: once the graph is small, every remaining round of every remaining
// level runs inside one block of 1024 threads, with barriers between the
// steps instead of kernel launches and host round trips.  The arithmetic is
// the same as above.  Node ids stay fixed inside the tail: a component
// formed by a merge keeps its root's id, its other members die.  The
// per-node arrays (size, smallest point, row window, parent, the tail-start
// node -> current node map) live in LDS; the fp64 means, the int64 sums and
// the table stay in global memory.  A round:
//   select    the gain of every undirected edge once, from the row of its
//             smaller end (after a level's first round only the edges of
//             nodes formed by a merge in the last round: every other gain
//             is unchanged and gave no candidate), each end's largest
//             candidate gain by a max of an order-preserving key, then
//             among the edges with that gain the neighbour with the
//             smallest minpt, by a 64-bit min of (minpt, neighbour) (Steps
//             1-2, the same choice as best_before)
//   union     hook and pointer jumping on LDS arrays (Step 3)
//   stats     every member adds its size, smallest point and int64 sums
//             into its root; the merged roots' means are recomputed (Step 4)
//   contract  a new window, past the end of the table, for every merged
//             root (its members' rows and its own, relabelled) and for
//             every row that listed a member; the other rows stay as they
//             are, since every node they list keeps its id (Step 4).  When
//             the table is full, every live row is rebuilt into the other
//             buffer instead.
// At a level's end the live nodes are numbered in id order for the
// snapshots that the labels and the energy read.
// ---------------------------------------------------------------------------
constexpr int kTailNT = 1024;
constexpr int kTailNodes = 1536;    // largest graph the tail can take (LDS)
constexpr int kTailWin = 8000;      // slots of new windows built in LDS
constexpr int kTailStart = 1500;    // default switch to the tail
constexpr int kTailEdges = 1 << 16; // ... directed entries at the switch
constexpr int kTailSlots = 1 << 17; // gains: the live windows span at most
                                    // twice the entries at the switch
constexpr int kTailLevels = 16;
static_assert(sizeof(((Ctl *)nullptr)->tail_nc) == kTailLevels * 4,
              "tail level counts travel in the control block");
constexpr int kTailJumps = 64;
// Entries per thread whose loads are issued together in the tail's entry
// loops: the block is alone on one CU, so memory latency, not bandwidth,
// sets the pace of a loop that waits on every entry's loads in turn.
constexpr int kTU = 4;

struct TailState {
  int32_t *ws[2], *wl[2];
  uint64_t *tbl[2];
  const int32_t *size, *minpt;             // node state at the tail's start
  int64_t *S;                              // sums, updated in place
  double *mu;                              // means, updated in place
  double *gain;                            // per listed edge
  uint64_t *elist;                         // edges to evaluate:
                                           // (v | u << 16) << 32 | w
  int32_t *lvl_map, *lvl_minpt, *lvl_nc;  // kTailLevels x nn0 (nc: levels)
  int32_t *lvl_rank;                       // kTailLevels x nn0
  double *lvl_mu;                          // kTailLevels x nn0 x d
  long long *lvl_cut2;                     // kTailLevels
  int32_t nn0, tcur0, d, tcap, gcap, n_levels, level0, round0, max_rounds;
  int32_t want_energy;
  int32_t rebuild_all;  // every round rebuilds every live row (tests)
  double lambda[kTailLevels];
  long long smin[kTailLevels];
};

// The tail is one block, so its global read-modify-writes only need
// workgroup scope: they are performed in this XCD's L2 instead of going out
// to memory as device-scope atomics do.  Kernel end still publishes them.
__device__ __forceinline__ void wg_add64(int64_t *p, int64_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Exclusive scan of value(0..len) into out[0..len], out[len] = total.
template <class V>
__device__ __forceinline__ int32_t tail_scan(int32_t len, V &&value,
                                             int32_t *out, int32_t *wsum) {
  const int32_t per = (len + kTailNT - 1) / kTailNT;
  const int32_t b0 = (int32_t)threadIdx.x * per;
  int32_t sum = 0;
  for (int32_t j = 0; j < per; ++j)
    if (b0 + j < len) sum += value(b0 + j);
  int32_t tot;
  int32_t run = block_excl_scan<kTailNT>(sum, wsum, &tot);
  for (int32_t j = 0; j < per; ++j) {
    const int32_t i = b0 + j;
    if (i < len) {
      const int32_t v = value(i);
      out[i] = run;
      run += v;
    }
  }
  if (threadIdx.x == 0) out[len] = tot;
  __syncthreads();
  return tot;
}

// Rows of U flattened positions p[j]: the last v < nn with pos[v] <= p[j]
// (pos ascending, pos[0] = 0, rows of no span share their successor's
// start).  The U searches take their steps together (the step sizes depend
// on nn only), so each step's LDS reads are issued back to back.
template <int U>
__device__ __forceinline__ void tail_rows(const int32_t *pos, int32_t nn,
                                          const int32_t (&p)[U],
                                          int32_t (&v)[U]) {
#pragma unroll
  for (int j = 0; j < U; ++j) v[j] = 0;
  for (int32_t len = nn; len > 1;) {
    const int32_t half = len >> 1;
#pragma unroll
    for (int j = 0; j < U; ++j)
      v[j] = pos[v[j] + half] <= p[j] ? v[j] + half : v[j];
    len -= half;
  }
}

// Order-preserving key of a finite double; 0 is below every key.
__device__ __forceinline__ unsigned long long gain_key(double g) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(g);
  return (b >> 63) ? ~b : (b | (1ull << 63));
}

// Prop. 1 for the entry (v, u) in the tail: the operations of edge_gain in
// the same order, sizes from LDS and the two mean rows streamed two
// dimensions at a time (few registers: the tail runs 1024 threads).  The
// value is symmetric bit for bit in (v, u).
template <int DT>
__device__ __forceinline__ double tail_gain(const double *__restrict__ mu,
                                            int32_t v, int32_t u, int32_t d,
                                            double dsv, double dsu, int32_t w,
                                            double lambda) {
  const double num = dsv * dsu;
  const double den = dsv + dsu;
  const double f = num / den;
  double ss = 0.0;
  if constexpr (DT > 0) {
    const double2 *a = reinterpret_cast<const double2 *>(mu + (int64_t)v * DT);
    const double2 *b = reinterpret_cast<const double2 *>(mu + (int64_t)u * DT);
#pragma unroll 4
    for (int i = 0; i < DT / 2; ++i) {
      const double2 x = a[i], y = b[i];
      const double d0 = x.x - y.x;
      const double q0 = d0 * d0;
      ss = ss + q0;
      const double d1 = x.y - y.y;
      const double q1 = d1 * d1;
      ss = ss + q1;
    }
  } else {
    for (int32_t i = 0; i < d; ++i) {
      const double diff = mu[(int64_t)v * d + i] - mu[(int64_t)u * d + i];
      const double sq = diff * diff;
      ss = ss + sq;
    }
  }
  const double cut = lambda * (double)w;
  const double fit = f * ss;
  return cut - fit;
}

// Calls f(p, v, e) for every non-empty entry e of the rows whose flattened
// positions pos[] spans (P positions in all): row v, table tb.  The entries
// and rows of kTU positions per thread are loaded before any is used.
template <int U = kTU, class Fn>
__device__ __forceinline__ void tail_entries(const int32_t *pos, int32_t nn,
                                             int32_t P, const int32_t *s_ws,
                                             const uint64_t *tb, Fn &&f) {
  for (int32_t p0 = threadIdx.x; p0 < P; p0 += U * kTailNT) {
    uint64_t ev[U];
    int32_t pp[U], vv[U];
#pragma unroll
    for (int j = 0; j < U; ++j) pp[j] = min(p0 + j * kTailNT, P - 1);
    tail_rows<U>(pos, nn, pp, vv);
#pragma unroll
    for (int j = 0; j < U; ++j) ev[j] = tb[s_ws[vv[j]] + (pp[j] - pos[vv[j]])];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int32_t p = p0 + j * kTailNT;
      if (p >= P || ev[j] == kEmpty) continue;
      f(p, vv[j], ev[j]);
    }
  }
}

template <int DT>
__global__ __launch_bounds__(kTailNT) void k_tail(TailState t, Ctl *ctl) {
  __shared__ int32_t s_size[kTailNodes], s_minpt[kTailNodes];
  __shared__ int32_t s_ws[kTailNodes], s_wl[kTailNodes], s_deg[kTailNodes];
  __shared__ int32_t s_L[kTailNodes], s_sel[kTailNodes], s_Mt[kTailNodes];
  __shared__ int32_t s_pos[kTailNodes + 1], s_nws[kTailNodes + 1];
  __shared__ int32_t s_cap[kTailNodes];
  __shared__ unsigned long long s_key[kTailNodes], s_pick[kTailNodes];
  // node flags: live; formed by a merge in the last round; root with
  // members in this round; row to rebuild in this round
  __shared__ uint8_t s_live[kTailNodes], s_mrg[kTailNodes], s_new[kTailNodes],
      s_touch[kTailNodes];
  // a round's new windows when they fit: built here, then copied out
  __shared__ uint64_t s_win[kTailWin];
  __shared__ int32_t wsum[kTailNT / kWave];
  __shared__ int32_t s_any, s_flag, s_cnt, s_ne;
  __shared__ long long s_cut;
  __shared__ double s_lambda[kTailLevels];
  __shared__ long long s_smin[kTailLevels];
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t d = DT > 0 ? DT : t.d;  // a constant divisor when DT is given
  const int32_t N = t.nn0;
  const double sIF = ldexp(1.0, -ctl->F);
  // the window area is free during selection: it holds the first kLE
  // listed edges and their gains, the rest go to global memory
  constexpr int32_t kLE = kTailWin / 2;
  uint64_t *s_el = s_win;
  double *s_gn = reinterpret_cast<double *>(s_win + kLE);
  // s_key doubles as the new entry counts once the choices are made
  int32_t *s_ndeg = reinterpret_cast<int32_t *>(s_key);
  if (N > kTailNodes || N < 1) {
    if (threadIdx.x == 0) raise_err(ctl, kErrInternal);
    return;
  }
  int32_t tc = t.tcur0;
  if (threadIdx.x < kTailLevels) {
    s_lambda[threadIdx.x] = t.lambda[threadIdx.x];
    s_smin[threadIdx.x] = t.smin[threadIdx.x];
  }
  for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
    s_size[v] = t.size[v];
    s_minpt[v] = t.minpt[v];
    s_ws[v] = t.ws[tc][v];
    s_wl[v] = t.wl[tc][v];
    s_Mt[v] = v;
    s_live[v] = 1;
    s_mrg[v] = 0;
    s_new[v] = 0;
    s_touch[v] = 0;
    s_sel[v] = v;
  }
  if (threadIdx.x == 0) s_cnt = 0;
  __syncthreads();
  // every live row's entries (the incoming windows are packed end to end)
  int32_t top = 0;
  {
    const int32_t P =
        tail_scan(N, [&](int32_t v) { return s_wl[v]; }, s_pos, wsum);
    top = s_ws[N - 1] + s_wl[N - 1];
    for (int32_t v = threadIdx.x; v < N; v += kTailNT) s_deg[v] = 0;
    __syncthreads();
    tail_entries(s_pos, N, P, s_ws, t.tbl[tc],
                 [&](int32_t, int32_t v, uint64_t) { atomicAdd(&s_deg[v], 1); });
    __syncthreads();
  }
  int32_t nn = N;  // live nodes
  int32_t ed = tail_scan(N, [&](int32_t v) { return s_deg[v]; }, s_nws, wsum);
  for (int32_t l = t.level0; l < t.n_levels; ++l) {
    const double lambda = s_lambda[l];
    const long long smin = s_smin[l];
    for (int32_t round = (l == t.level0 ? t.round0 : 0);; ++round) {
      if (ed == 0 || nn == 1) break;  // nothing can merge
      const bool fresh = round == 0 || (l == t.level0 && round == t.round0);
      if (round >= t.max_rounds) {
        if (threadIdx.x == 0) {
          ctl->tail_level = l;
          raise_err(ctl, kErrNotConv);
        }
        return;
      }
      const uint64_t *tb = t.tbl[tc];
      if (threadIdx.x == 0) s_any = 0;
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
        s_key[v] = 0ull;
        s_pick[v] = ~0ull;
      }
      // rows whose entries are evaluated: every live row in a fresh round,
      // else the rows of the nodes formed by a merge in the last round
      auto scanned = [&](int32_t v) {
        return s_live[v] && (fresh || s_mrg[v]);
      };
      if (threadIdx.x == 0) s_ne = 0;
      const int32_t P = tail_scan(
          N, [&](int32_t v) { return scanned(v) ? s_wl[v] : 0; }, s_pos, wsum);
      // the edges to evaluate, each once: from the row of its smaller end
      // when both rows are scanned
      tail_entries<8>(s_pos, N, P, s_ws, tb, [&](int32_t, int32_t v,
                                                 uint64_t e) {
        const int32_t u = (int32_t)(e >> 32);
        if ((uint32_t)u >= (uint32_t)N || !s_live[u]) {
          raise_err(ctl, kErrInternal);
          return;
        }
        if (u < v && scanned(u)) return;
        const int32_t i = atomicAdd(&s_ne, 1);
        const uint64_t le =
            ((uint64_t)(uint32_t)(v | (u << 16)) << 32) | (uint32_t)e;
        if (i < kLE)
          s_el[i] = le;
        else if (i < t.gcap)
          t.elist[i] = le;
        else
          raise_err(ctl, kErrInternal);
      });
      __syncthreads();
      const int32_t ne = min(s_ne, t.gcap);
      // Steps 1-2, pass 1: each listed edge's gain, and each end's largest
      // candidate gain (two edges per thread in flight)
      for (int32_t i0 = threadIdx.x; i0 < ne; i0 += 2 * kTailNT) {
        uint64_t ev[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int32_t i = min(i0 + j * kTailNT, ne - 1);
          ev[j] = i < kLE ? s_el[i] : t.elist[i];
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int32_t i = i0 + j * kTailNT;
          if (i >= ne) break;
          const uint32_t vu = (uint32_t)(ev[j] >> 32);
          const int32_t v = (int32_t)(vu & 0xffffu), u = (int32_t)(vu >> 16);
          const int32_t w = (int32_t)(uint32_t)ev[j];
          const double g = tail_gain<DT>(t.mu, v, u, d, (double)s_size[v],
                                         (double)s_size[u], w, lambda);
          if (i < kLE)
            s_gn[i] = g;
          else
            t.gain[i] = g;
          const unsigned long long kg = gain_key(g);
          if (g > 0.0 || (long long)s_size[v] < smin) atomicMax(&s_key[v], kg);
          if (g > 0.0 || (long long)s_size[u] < smin) atomicMax(&s_key[u], kg);
        }
      }
      __syncthreads();
      // pass 2: the same edges; at each end whose largest candidate gain
      // this is, the neighbour with the smallest minpt (minpt is unique per
      // node, so the 64-bit minimum of (minpt, neighbour) names it)
      for (int32_t i0 = threadIdx.x; i0 < ne; i0 += kTU * kTailNT) {
        uint64_t ev[kTU];
        double gv[kTU];
#pragma unroll
        for (int j = 0; j < kTU; ++j) {
          const int32_t i = min(i0 + j * kTailNT, ne - 1);  // no branch
          ev[j] = i < kLE ? s_el[i] : t.elist[i];
          gv[j] = i < kLE ? s_gn[i] : t.gain[i];
        }
#pragma unroll
        for (int j = 0; j < kTU; ++j) {
          if (i0 + j * kTailNT >= ne) break;
          const uint32_t vu = (uint32_t)(ev[j] >> 32);
          const int32_t v = (int32_t)(vu & 0xffffu), u = (int32_t)(vu >> 16);
          const unsigned long long kv = s_key[v], ku = s_key[u];
          const unsigned long long kg = gain_key(gv[j]);
          if (kv != 0ull && kg == kv)
            atomicMin(&s_pick[v],
                      ((unsigned long long)(uint32_t)s_minpt[u] << 32) |
                          (uint32_t)u);
          if (ku != 0ull && kg == ku)
            atomicMin(&s_pick[u],
                      ((unsigned long long)(uint32_t)s_minpt[v] << 32) |
                          (uint32_t)v);
        }
      }
      __syncthreads();
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
        const unsigned long long pk = s_pick[v];
        s_L[v] = (s_live[v] && pk != ~0ull) ? (int32_t)(uint32_t)pk : -1;
        if (s_L[v] >= 0) s_any = 1;
      }
      __syncthreads();
      if (!s_any) break;  // Step 1: no candidate merge
      // Step 3: hook (s_sel = parent), pointer jumping
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
        const int32_t tg = s_L[v];
        s_sel[v] = tg < 0 ? v : ((s_L[tg] == v && v < tg) ? v : tg);
      }
      __syncthreads();
      for (int pass = 0;; ++pass) {
        if (threadIdx.x == 0) s_flag = 0;
        __syncthreads();
        for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
          const int32_t p = s_sel[v];
          const int32_t pp = s_sel[p];
          if (pp != p) {
            s_sel[v] = pp;
            s_flag = 1;
          }
        }
        __syncthreads();
        const int more = s_flag;
        __syncthreads();  // all have read the flag before the next reset
        if (!more) break;
        if (pass == kTailJumps) {
          if (threadIdx.x == 0) raise_err(ctl, kErrJump);
          return;
        }
      }
      // Step 4 statistics: members add into their roots (size and smallest
      // point in LDS, the sums in global memory)
      int32_t members = 0;
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
        const int32_t r = s_sel[v];
        if (s_live[v] && r != v) {
          ++members;
          s_new[r] = 1;
          atomicAdd(&s_size[r], s_size[v]);
          atomicMin(&s_minpt[r], s_minpt[v]);
        }
      }
      members = wave_sum(members);
      if (lane == 0 && members) atomicAdd(&s_cnt, members);
      // lists of the members (in s_L, free after the hook) and of the
      // merged roots (in s_pick, free after the choices)
      int32_t *s_ml = s_L;
      int32_t *s_rl = reinterpret_cast<int32_t *>(s_pick);
      const int32_t nm = tail_scan(
          N, [&](int32_t v) { return (s_live[v] && s_sel[v] != v) ? 1 : 0; },
          s_pos, wsum);
      for (int32_t v = threadIdx.x; v < N; v += kTailNT)
        if (s_live[v] && s_sel[v] != v) s_ml[s_pos[v]] = v;
      const int32_t nr =
          tail_scan(N, [&](int32_t v) { return (int32_t)s_new[v]; }, s_nws, wsum);
      for (int32_t v = threadIdx.x; v < N; v += kTailNT)
        if (s_new[v]) s_rl[s_nws[v]] = v;
      __syncthreads();
      // the members' sums, one (member, dimension) pair per thread
      for (int32_t q0 = threadIdx.x; q0 < nm * d; q0 += kTU * kTailNT) {
        int64_t sv[kTU];
        int32_t mv[kTU];
#pragma unroll
        for (int j = 0; j < kTU; ++j) {
          const int32_t q = min(q0 + j * kTailNT, nm * d - 1);  // no branch
          const int32_t m = s_ml[q / d];
          mv[j] = m;
          sv[j] = t.S[(int64_t)m * d + (q - (q / d) * d)];
        }
#pragma unroll
        for (int j = 0; j < kTU; ++j) {
          const int32_t q = q0 + j * kTailNT;
          if (q >= nm * d) break;
          wg_add64(&t.S[(int64_t)s_sel[mv[j]] * d + (q - (q / d) * d)], sv[j]);
        }
      }
      // rows that list a member are rebuilt: by symmetry, they are the
      // rows that a member lists
      const int32_t Pm = tail_scan(
          N,
          [&](int32_t v) {
            return (s_live[v] && s_sel[v] != v) ? s_wl[v] : 0;
          },
          s_pos, wsum);
      tail_entries<8>(s_pos, N, Pm, s_ws, tb,
                      [&](int32_t, int32_t, uint64_t e) {
                        const int32_t u = (int32_t)(e >> 32);
                        if ((uint32_t)u < (uint32_t)N && s_sel[u] == u &&
                            !s_new[u])
                          s_touch[u] = 1;
                      });
      __syncthreads();
      // Step 4 means of the merged roots (their sums are complete)
      for (int32_t q0 = threadIdx.x; q0 < nr * d; q0 += kTU * kTailNT) {
        int64_t sv[kTU];
#pragma unroll
        for (int j = 0; j < kTU; ++j) {
          const int32_t q = min(q0 + j * kTailNT, nr * d - 1);  // no branch
          sv[j] = t.S[(int64_t)s_rl[q / d] * d + (q - (q / d) * d)];
        }
#pragma unroll
        for (int j = 0; j < kTU; ++j) {
          const int32_t q = q0 + j * kTailNT;
          if (q >= nr * d) break;
          const int32_t r = s_rl[q / d];
          const double m = (double)sv[j] / (double)s_size[r];
          t.mu[(int64_t)r * d + (q - (q / d) * d)] = m * sIF;
        }
      }
      // Step 4 contraction.  Windows: every rebuilt row gets its sources'
      // summed entry count, twice when the table has room (open addressing
      // at load factor <= 1/2 keeps the probe chains short).
      auto rebuilt = [&](int32_t A) { return s_new[A] || s_touch[A]; };
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) s_cap[v] = 0;
      __syncthreads();
      for (int32_t v = threadIdx.x; v < N; v += kTailNT)
        if (s_live[v] && rebuilt(s_sel[v])) atomicAdd(&s_cap[s_sel[v]], s_deg[v]);
      __syncthreads();
      int32_t need = tail_scan(
          N, [&](int32_t A) { return rebuilt(A) ? s_cap[A] : 0; }, s_nws, wsum);
      // room for the new windows past the end of the table, else every
      // live row is rebuilt into the other buffer
      int spread = 2;
      bool whole = false;
      if (t.rebuild_all || top + 2 * need > t.tcap) {
        if (!t.rebuild_all && top + need <= t.tcap) {
          spread = 1;
        } else {
          whole = true;
          for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
            s_cap[v] = 0;
            if (s_live[v] && s_sel[v] == v) s_touch[v] = 1;
          }
          __syncthreads();
          for (int32_t v = threadIdx.x; v < N; v += kTailNT)
            if (s_live[v]) atomicAdd(&s_cap[s_sel[v]], s_deg[v]);
          __syncthreads();
          need = tail_scan(
              N, [&](int32_t A) { return rebuilt(A) ? s_cap[A] : 0; }, s_nws,
              wsum);
          spread = 2 * need <= t.tcap ? 2 : 1;
          if (need > t.tcap) {
            if (threadIdx.x == 0) raise_err(ctl, kErrInternal);
            return;
          }
        }
      }
      const int tn = whole ? 1 - tc : tc;
      const int32_t base = whole ? 0 : top;
      uint64_t *tn_tbl = t.tbl[tn];
      // the windows are built in LDS when they fit (their probes are then
      // LDS atomics, not L2 round trips), else in place in the table; LDS
      // at load factor <= 1 beats the table at <= 1/2
      if (spread == 2 && 2 * need > kTailWin && need <= kTailWin) spread = 1;
      const bool in_lds = spread * need <= kTailWin;
      for (int32_t q = threadIdx.x; q < spread * need; q += kTailNT) {
        if (in_lds)
          s_win[q] = kEmpty;
        else
          tn_tbl[base + q] = kEmpty;
      }
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) s_ndeg[v] = 0;
      // sources: the rows of every live node whose root is rebuilt
      const int32_t Ps = tail_scan(
          N,
          [&](int32_t v) {
            return (s_live[v] && rebuilt(s_sel[v])) ? s_wl[v] : 0;
          },
          s_pos, wsum);  // (its barrier also orders the clears above)
      // every source entry (v, u, w) becomes (root of v, root of u, w) in
      // the root's new window.  A thread's kIU entries probe together: each
      // step issues one compare-and-swap per pending entry before waiting.
      constexpr int kIU = 4;
      auto insert_all = [&](auto *win) {
      for (int32_t p0 = threadIdx.x; p0 < Ps; p0 += kIU * kTailNT) {
        int32_t A[kIU], B[kIU], W[kIU], np[kIU], pp[kIU], vv[kIU];
        uint32_t h[kIU];
        bool pend[kIU];
#pragma unroll
        for (int j = 0; j < kIU; ++j) pp[j] = min(p0 + j * kTailNT, Ps - 1);
        tail_rows<kIU>(s_pos, N, pp, vv);
#pragma unroll
        for (int j = 0; j < kIU; ++j) {
          const int32_t v = vv[j];
          const uint64_t e = tb[s_ws[v] + (pp[j] - s_pos[v])];
          const int32_t u = (int32_t)(e >> 32);
          A[j] = s_sel[v];
          B[j] = (e != kEmpty && (uint32_t)u < (uint32_t)N &&
                  p0 + j * kTailNT < Ps)
                     ? s_sel[u]
                     : A[j];  // nothing to add
          W[j] = (int32_t)(uint32_t)e;
          pend[j] = A[j] != B[j];  // not inside a component
          np[j] = 0;
          h[j] = pend[j] ? window_slot(B[j], spread * s_cap[A[j]]) : 0u;
        }
        for (bool any = true; any;) {
          uint64_t cur[kIU];
          bool got[kIU];
#pragma unroll
          for (int j = 0; j < kIU; ++j) {
            cur[j] = kEmpty;
            got[j] = false;
            if (pend[j])
              got[j] = __hip_atomic_compare_exchange_strong(
                  win + spread * s_nws[A[j]] + h[j], &cur[j],
                  ((uint64_t)(uint32_t)B[j] << 32) | (uint32_t)W[j],
                  __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                  __HIP_MEMORY_SCOPE_WORKGROUP);
          }
          any = false;
#pragma unroll
          for (int j = 0; j < kIU; ++j) {
            if (!pend[j]) continue;
            const int32_t cap = spread * s_cap[A[j]];
            if (got[j]) {
              atomicAdd(&s_ndeg[A[j]], 1);
              pend[j] = false;
            } else if ((int32_t)(cur[j] >> 32) == B[j]) {
              __hip_atomic_fetch_add(win + spread * s_nws[A[j]] + h[j],
                                     (uint64_t)(uint32_t)W[j], __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_WORKGROUP);
              pend[j] = false;
            } else if (++np[j] >= cap) {
              raise_err(ctl, kErrInternal);
              pend[j] = false;
            } else {
              h[j] = h[j] + 1 == (uint32_t)cap ? 0u : h[j] + 1;
              any = true;
            }
          }
        }
      }
      };
      if (in_lds) {
        insert_all(s_win);
        __syncthreads();
        for (int32_t q = threadIdx.x; q < spread * need; q += kTailNT)
          tn_tbl[base + q] = s_win[q];
      } else {
        insert_all(tn_tbl + base);
      }
      __syncthreads();
      // the new state: rebuilt windows, members dead, merge flags for the
      // next round's selection, the map of the tail's start nodes
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
        if (s_live[v] && s_sel[v] != v) {
          s_live[v] = 0;
          s_deg[v] = 0;
          s_wl[v] = 0;
        } else if (s_live[v] && rebuilt(v)) {
          s_ws[v] = base + spread * s_nws[v];
          s_wl[v] = spread * s_cap[v];
          s_deg[v] = s_ndeg[v];
        }
        s_mrg[v] = s_new[v];
        s_Mt[v] = s_sel[s_Mt[v]];
      }
      __syncthreads();
      for (int32_t v = threadIdx.x; v < N; v += kTailNT) {
        s_new[v] = 0;
        s_touch[v] = 0;
        s_sel[v] = v;
      }
      nn -= s_cnt;
      top = base + spread * need;
      tc = tn;
      ed = tail_scan(N, [&](int32_t v) { return s_deg[v]; }, s_nws, wsum);
      if (threadIdx.x == 0) s_cnt = 0;
      __syncthreads();
    }
    // level end: live nodes numbered in id order, snapshots for the labels
    // and the energy
    const int32_t C = tail_scan(
        N, [&](int32_t v) { return (int32_t)s_live[v]; }, s_pos, wsum);
    if (threadIdx.x == 0) {
      t.lvl_nc[l] = C;
      s_cut = 0;
    }
    for (int32_t i = threadIdx.x; i < N; i += kTailNT) {
      t.lvl_map[(int64_t)l * N + i] = s_pos[s_Mt[i]];
      if (s_live[i]) t.lvl_minpt[(int64_t)l * N + s_pos[i]] = s_minpt[i];
    }
    // (the canonical numbers, ranks of these smallest points, are counted
    // after the tail by k_tail_rank on many CUs)
    __syncthreads();
    if (t.want_energy) {
      for (int32_t q = threadIdx.x; q < N * d; q += kTailNT) {
        const int32_t v = q / d;
        if (s_live[v])
          t.lvl_mu[((int64_t)l * N + s_pos[v]) * d + (q - v * d)] = t.mu[q];
      }
      const int32_t Pc = tail_scan(
          N, [&](int32_t v) { return s_live[v] ? s_wl[v] : 0; }, s_nws, wsum);
      long long acc = 0;
      tail_entries(s_nws, N, Pc, s_ws, t.tbl[tc],
                   [&](int32_t, int32_t, uint64_t e) {
                     acc += (int32_t)(uint32_t)e;
                   });
      acc = wave_sum(acc);
      if (lane == 0 && acc)
        atomicAdd(reinterpret_cast<unsigned long long *>(&s_cut),
                  (unsigned long long)acc);
      __syncthreads();
      if (threadIdx.x == 0) t.lvl_cut2[l] = s_cut;
    }
    __syncthreads();
  }
}

// Canonical number of every component of every level the tail ended: the
// rank of its smallest point among the level's components.  64 components
// per block, four lanes per component counting a quarter each over the
// level's smallest points staged in LDS.  A level count out of range (only
// after a device error, whose outputs are discarded) is clamped to nt.
__global__ __launch_bounds__(256) void k_tail_rank(
    const int32_t *__restrict__ lvl_minpt, const int32_t *__restrict__ lvl_nc,
    int32_t nt, int32_t level0, int32_t *__restrict__ lvl_rank) {
  __shared__ int32_t sm[kTailNodes];
  const int32_t l = level0 + (int32_t)blockIdx.y;
  const int32_t nc = min(max(lvl_nc[l], 0), min(nt, kTailNodes));
  const int32_t *mp = lvl_minpt + (int64_t)l * nt;
  for (int32_t c = threadIdx.x; c < nc; c += blockDim.x) sm[c] = mp[c];
  __syncthreads();
  const int32_t c = (int32_t)blockIdx.x * 64 + (int32_t)(threadIdx.x >> 2);
  const int q = threadIdx.x & 3;
  int32_t r = 0;
  if (c < nc) {
    const int32_t m = sm[c];
    for (int32_t j = q; j < nc; j += 4) r += sm[j] < m ? 1 : 0;
  }
  r += __shfl_xor(r, 1, kWave);
  r += __shfl_xor(r, 2, kWave);
  if (c < nc && q == 0) lvl_rank[(int64_t)l * nt + c] = r;
}

// Point labels of every level the tail ended: point p -> its node at the
// tail's start -> that level's component -> the component's canonical rank.
__global__ __launch_bounds__(256) void k_tail_labels(
    int32_t n, const int32_t *__restrict__ inv, const int32_t *__restrict__ M,
    const int32_t *__restrict__ lvl_map, const int32_t *__restrict__ lvl_rank,
    const int32_t *__restrict__ lvl_nc, int32_t nt, int32_t level0,
    int32_t n_levels, int32_t *__restrict__ labels, Ctl *ctl) {
  const int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t i = inv ? inv[p] : p;
  const int32_t c0 = ((uint32_t)i < (uint32_t)n) ? M[i] : -1;
  for (int32_t l = level0; l < n_levels; ++l) {
    int32_t out = -1;
    if ((uint32_t)c0 < (uint32_t)nt) {
      const int32_t c = lvl_map[(int64_t)l * nt + c0];
      if ((uint32_t)c < (uint32_t)min(lvl_nc[l], nt))
        out = lvl_rank[(int64_t)l * nt + c];
    }
    if (out < 0) raise_err(ctl, kErrInternal);
    labels[(int64_t)l * n + p] = out;
  }
}

// Rows of the table the tail starts from, copied into windows packed end
// to end, each row's entries moved to the front of its window (wl2 = the
// entry count).  A wave per row, lanes striding over its slots (hub rows
// are long).
__global__ __launch_bounds__(256) void k_repack(
    int32_t nn, const int32_t *__restrict__ ws, const int32_t *__restrict__ wl,
    const uint64_t *__restrict__ tbl, const int32_t *__restrict__ ws2,
    int32_t *__restrict__ wl2, uint64_t *__restrict__ tbl2) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t v = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                              threadIdx.x / kWave);
  if (v >= nn) return;
  const int32_t len = wl[v];
  const uint64_t *src = tbl + ws[v];
  uint64_t *dst = tbl2 + ws2[v];
  int32_t cnt = 0;
  for (int32_t j0 = 0; j0 < len; j0 += kWave) {
    const int32_t j = j0 + lane;
    const uint64_t e = j < len ? src[j] : kEmpty;
    const uint64_t m = __ballot(e != kEmpty);
    if (e != kEmpty)
      dst[cnt + __popcll(m & ((1ull << lane) - 1ull))] = e;
    cnt += __popcll(m);
  }
  if (lane == 0) wl2[v] = cnt;
}

// ---------------------------------------------------------------------------
// host driver
// ---------------------------------------------------------------------------
namespace {

// ---------------------------------------------------------------------------
// prepare_graph's linking of isolated nodes (App. Alg. A-2), optional: at the
// start of a round with more than one node, every node whose row is empty
// gets an edge of weight 1 to each of its min(k, nn - 1) nearest nodes, by
// the squared distance of the centroids and then the smaller minpt (the
// canonical order); a pair linked from both ends is one edge.  Centroids are
// exact: int64 fixed-point position sums, c = (double)Sx / |P|, and the
// squared distance ((dx*dx) + (dy*dy)) + (dz*dz) in fp64 without
// contraction.  The table is then rebuilt, rows compacted, with the links
// appended.
// ---------------------------------------------------------------------------

// max |coordinate| over the points (x, y, z of the internal float4 array)
__global__ __launch_bounds__(256) void k_link_maxabs(const float4 *pts,
                                                     int32_t n, Ctl *ctl) {
  uint32_t m = 0;
  for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += gridDim.x * blockDim.x) {
    const float4 p = pts[i];
    m = max(m, __float_as_uint(fabsf(p.x)));
    m = max(m, __float_as_uint(fabsf(p.y)));
    m = max(m, __float_as_uint(fabsf(p.z)));
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1)
    m = max(m, (uint32_t)__shfl_xor((int)m, off, kWave));
  if ((threadIdx.x & (kWave - 1)) == 0) atomicMax(&ctl->maxabs_x_bits, m);
}

// fixed-point shift of the positions, the same rule as for the embeddings
__global__ void k_link_shift(Ctl *ctl, int32_t n) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  ctl->Fx = fixshift_rule(__uint_as_float(ctl->maxabs_x_bits), n);
  if (ctl->Fx < 16) raise_err(ctl, kErrRange);
}

// After a contraction: the next table's nodes whose row is empty (a scan
// that stops at the first occupied slot), listed for the host.  Live count
// n_next from the control block; nothing to do when the round merged none.
__global__ __launch_bounds__(256) void k_link_detect(const int32_t *ws,
                                                     const int32_t *wl,
                                                     const uint64_t *tbl,
                                                     int32_t *iso,
                                                     int32_t *iso_of,
                                                     Ctl *ctl) {
  if (!round_live(ctl)) return;
  int32_t v;
  if (!xcd_item(ctl->n_next, v)) return;
  const uint64_t *t = tbl + ws[v];
  const int32_t len = wl[v];
  bool empty = true;
  for (int32_t j = 0; j < len && empty; ++j) empty = t[j] == kEmpty;
  int32_t slot = -1;
  if (empty) {
    slot = atomicAdd(&ctl->n_iso, 1);
    iso[slot] = v;
  }
  iso_of[v] = slot;
}

// Position sums of the next round's components from their members: int64
// fixed point, exact in any order.  In the first round the members are
// points, rint(x * 2^Fx) on the fly.  A thread per component with at most
// kBigComp members; the larger ones (listed by the statistics) a block each.
template <bool FIRST>
__device__ __forceinline__ void member_pos(const float4 *pts,
                                           const int64_t *sx_in, int32_t m,
                                           double sF, long long a[3]) {
  if (FIRST) {
    const float4 q = pts[m];
    a[0] += (long long)rint((double)q.x * sF);
    a[1] += (long long)rint((double)q.y * sF);
    a[2] += (long long)rint((double)q.z * sF);
  } else {
    a[0] += sx_in[3 * (int64_t)m + 0];
    a[1] += sx_in[3 * (int64_t)m + 1];
    a[2] += sx_in[3 * (int64_t)m + 2];
  }
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_link_accum(
    const int32_t *mem, const int32_t *moff, const float4 *pts,
    const int64_t *sx_in, int64_t *sx_out, Ctl *ctl) {
  if (!round_live(ctl)) return;
  int32_t c;
  if (!xcd_item(ctl->n_next, c)) return;
  const int32_t m0 = moff[c], m1 = moff[c + 1];
  if (m1 - m0 > kBigComp) return;
  const double sF = ldexp(1.0, ctl->Fx);
  long long a[3] = {0, 0, 0};
  for (int32_t i = m0; i < m1; ++i) member_pos<FIRST>(pts, sx_in, mem[i], sF, a);
#pragma unroll
  for (int q = 0; q < 3; ++q) sx_out[3 * (int64_t)c + q] = a[q];
}

template <bool FIRST>
__global__ __launch_bounds__(256) void k_link_accum_big(
    const int32_t *mem, const int32_t *moff, const float4 *pts,
    const int64_t *sx_in, int64_t *sx_out, const int32_t *big, Ctl *ctl) {
  __shared__ unsigned long long acc[3];
  if (!round_live(ctl)) return;
  const int32_t n_big = ctl->n_big;
  const double sF = ldexp(1.0, ctl->Fx);
  for (int32_t bi = blockIdx.x; bi < n_big; bi += gridDim.x) {
    const int32_t c = big[bi];
    if (threadIdx.x < 3) acc[threadIdx.x] = 0ull;
    __syncthreads();
    long long a[3] = {0, 0, 0};
    for (int32_t i = moff[c] + threadIdx.x; i < moff[c + 1]; i += blockDim.x)
      member_pos<FIRST>(pts, sx_in, mem[i], sF, a);
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const long long r = wave_sum(a[q]);
      if ((threadIdx.x & (kWave - 1)) == 0)
        atomicAdd(&acc[q], (unsigned long long)r);
    }
    __syncthreads();
    if (threadIdx.x < 3) sx_out[3 * (int64_t)c + threadIdx.x] = (int64_t)acc[threadIdx.x];
    __syncthreads();
  }
}

// Occupied slots per row, a wave per row.
__global__ __launch_bounds__(256) void k_link_rowcount(int32_t nn, Adj a,
                                                       int32_t *cntv) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t w0 = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                               threadIdx.x / kWave);
  const int32_t nw = (int32_t)(gridDim.x * (blockDim.x / kWave));
  for (int32_t v = w0; v < nn; v += nw) {
    const uint64_t *t = a.tbl + a.ws[v];
    const int32_t len = a.wl[v];
    int32_t c = 0;
    for (int32_t j = lane; j < len; j += kWave) c += t[j] != kEmpty;
    c = wave_sum(c);
    if (lane == 0) cntv[v] = c;
  }
}

// Centroids of all nodes, (double)Sx / |P| per axis.
__global__ __launch_bounds__(256) void k_link_centroids(int32_t nn,
                                                        const int64_t *Sx,
                                                        const int32_t *size,
                                                        double *cen) {
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t >= 3 * (int64_t)nn) return;
  cen[t] = __ddiv_rn((double)Sx[t], (double)size[t / 3]);
}

struct NearKey {
  double d2;
  int32_t mp, u;
};
__device__ __forceinline__ bool near_before(const NearKey &a,
                                            const NearKey &b) {
  return a.d2 < b.d2 || (a.d2 == b.d2 && a.mp < b.mp);
}

constexpr int kLinkNT = 128;

// One block per isolated node: every thread keeps the best T candidates of
// its share of the nodes, sorted, in LDS; then T block-wide minima.
__global__ __launch_bounds__(kLinkNT) void k_link_near(
    int32_t nn, const int32_t *iso, const Ctl *cn, const double *cen,
    const int32_t *minpt, int32_t T, int32_t kstride, int32_t *near,
    Ctl *ctl) {
  extern __shared__ unsigned char link_lds[];
  NearKey *lst = reinterpret_cast<NearKey *>(link_lds);  // [kLinkNT][T]
  __shared__ NearKey red[kLinkNT];
  __shared__ int32_t red_t[kLinkNT];
  __shared__ int32_t head[kLinkNT];
  const int32_t n_iso = cn->n_iso;
  NearKey *mine = lst + threadIdx.x * T;
  for (int32_t it = blockIdx.x; it < n_iso; it += gridDim.x) {
    const int32_t v = iso[it];
    const double cx = cen[3 * (int64_t)v], cy = cen[3 * (int64_t)v + 1],
                 cz = cen[3 * (int64_t)v + 2];
    int32_t cnt = 0;
    for (int32_t u = threadIdx.x; u < nn; u += kLinkNT) {
      if (u == v) continue;
      const double dx = __dsub_rn(cen[3 * (int64_t)u], cx);
      const double dy = __dsub_rn(cen[3 * (int64_t)u + 1], cy);
      const double dz = __dsub_rn(cen[3 * (int64_t)u + 2], cz);
      const double t = __dadd_rn(__dmul_rn(dx, dx), __dmul_rn(dy, dy));
      const NearKey c{__dadd_rn(t, __dmul_rn(dz, dz)), minpt[u], u};
      if (cnt == T && !near_before(c, mine[T - 1])) continue;
      int32_t pos = cnt < T ? cnt++ : T - 1;
      while (pos > 0 && near_before(c, mine[pos - 1])) {
        mine[pos] = mine[pos - 1];
        --pos;
      }
      mine[pos] = c;
    }
    head[threadIdx.x] = 0;
    __syncthreads();
    for (int32_t r = 0; r < T; ++r) {
      const int32_t h = head[threadIdx.x];
      red[threadIdx.x] = h < cnt ? mine[h] : NearKey{INFINITY, INT32_MAX, -1};
      red_t[threadIdx.x] = threadIdx.x;
      __syncthreads();
      for (int off = kLinkNT / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off &&
            near_before(red[threadIdx.x + off], red[threadIdx.x])) {
          red[threadIdx.x] = red[threadIdx.x + off];
          red_t[threadIdx.x] = red_t[threadIdx.x + off];
        }
        __syncthreads();
      }
      if (threadIdx.x == 0) {
        near[(int64_t)it * kstride + r] = red[0].u;
        if (red[0].u < 0) raise_err(ctl, kErrInternal);
        head[red_t[0]] += 1;
      }
      __syncthreads();
    }
  }
}

// The kept links (a pair listed from both isolated ends counts once, from
// the end with the smaller internal id) and the extra entries per node.
__global__ __launch_bounds__(256) void k_link_count(
    const Ctl *cn, const int32_t *iso, const int32_t *iso_of,
    const int32_t *near, int32_t T, int32_t kstride, int32_t *ext,
    uint8_t *keep, Ctl *ctl) {
  const int64_t total = (int64_t)cn->n_iso * T;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t it = (int32_t)(i / T), r = (int32_t)(i - (int64_t)it * T);
    const int32_t v = iso[it], u = near[(int64_t)it * kstride + r];
    bool k = true;
    const int32_t iu = iso_of[u];
    if (iu >= 0 && u < v)
      for (int32_t t = 0; t < T && k; ++t)
        k = near[(int64_t)iu * kstride + t] != v;
    keep[i] = k ? 1 : 0;
    if (k) {
      atomicAdd(&ext[v], 1);
      atomicAdd(&ext[u], 1);
      atomicAdd(&ctl->n_link, 1);
    }
  }
}

// Rebuilt rows, a wave per row: the occupied slots of the old window,
// compacted in order by ballot, then room for the links (the cursor fill[v]
// starts after the copied entries).
__global__ __launch_bounds__(256) void k_link_copy(int32_t nn, Adj a,
                                                   const int32_t *cntv,
                                                   const int32_t *ext,
                                                   const int32_t *ws2,
                                                   int32_t *wl2,
                                                   uint64_t *tbl2,
                                                   int32_t *fill) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
  const int32_t w0 = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                               threadIdx.x / kWave);
  const int32_t nw = (int32_t)(gridDim.x * (blockDim.x / kWave));
  for (int32_t v = w0; v < nn; v += nw) {
    const int32_t base = ws2[v];
    const uint64_t *t = a.tbl + a.ws[v];
    const int32_t len = a.wl[v];
    int32_t c = 0;
    for (int32_t j0 = 0; j0 < len; j0 += kWave) {
      const int32_t j = j0 + lane;
      const uint64_t e = j < len ? t[j] : kEmpty;
      const uint64_t occ = __ballot(e != kEmpty);
      if (e != kEmpty) tbl2[base + c + __popcll(occ & lt)] = e;
      c += __popcll(occ);
    }
    if (lane == 0) {
      fill[v] = cntv[v];
      wl2[v] = cntv[v] + ext[v];
    }
  }
}

__global__ __launch_bounds__(256) void k_link_append(
    const Ctl *cn, const int32_t *iso, const int32_t *near, int32_t T,
    int32_t kstride, const uint8_t *keep, const int32_t *ws2,
    const int32_t *wl2, uint64_t *tbl2, int32_t *fill, Ctl *ctl) {
  const int64_t total = (int64_t)cn->n_iso * T;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (!keep[i]) continue;
    const int32_t it = (int32_t)(i / T), r = (int32_t)(i - (int64_t)it * T);
    const int32_t v = iso[it], u = near[(int64_t)it * kstride + r];
    const int32_t pv = atomicAdd(&fill[v], 1), pu = atomicAdd(&fill[u], 1);
    if (pv < wl2[v] && pu < wl2[u]) {
      tbl2[ws2[v] + pv] = ((uint64_t)(uint32_t)u << 32) | 1u;
      tbl2[ws2[u] + pu] = ((uint64_t)(uint32_t)v << 32) | 1u;
    } else {
      raise_err(ctl, kErrInternal);
    }
  }
}

// Scan functor for the rebuilt windows: length cntv + ext.
struct ScanLinkWin {
  const int32_t *cntv, *ext;
  int32_t *ws2;
  int32_t n;
  __device__ int32_t value(int32_t i) const {
    return i < n ? cntv[i] + ext[i] : 0;
  }
  __device__ void emit(int32_t i, int32_t excl, int32_t) const {
    if (i <= n) ws2[i] = excl;
  }
};

// Cut weight of the input graph (Eq. gmpp's second term on E0) for the
// point -> node map M: both directions of every first-round edge.
__global__ __launch_bounds__(256) void k_cut_e0(int32_t n, Adj a0,
                                                const int32_t *M, Ctl *ctl) {
  long long acc = 0;
  for (int32_t v = blockIdx.x * blockDim.x + threadIdx.x; v < n;
       v += gridDim.x * blockDim.x) {
    const int32_t mv = M[v];
    for_row<true>(a0, v, 0, 1, [&](int32_t u, int32_t w) {
      if (M[u] != mv) acc += w;
    });
  }
  acc = wave_sum(acc);
  if ((threadIdx.x & (kWave - 1)) == 0 && acc)
    atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->cut_w2),
              (unsigned long long)acc);
}

// ---------------------------------------------------------------------------
// Incremental rounds.  In a level whose rounds merge few nodes (the aerial
// tile merges 2-13 % of its nodes per round over dozens of rounds), node ids
// stay fixed from one round to the next instead of being renumbered: a
// component formed by a merge keeps the id of its root and its other
// members' ids die.  A round then touches only
//   - its worklist: the nodes formed by a merge in the last round and their
//     neighbours, the only nodes whose gains changed (every other node had
//     no candidate in the last round, since a node with one merges, and its
//     gains are the same now);
//   - the merged components: their sums (exact int64, added with atomics,
//     so the order does not matter) and their rows, rebuilt into fresh
//     windows past the end of the table (open addressing at load <= 1/2,
//     then compacted);
//   - the unmerged rows that listed a merged node: relabelled, and their
//     parallel entries summed, in place.
// rep[m] records the root a dead node merged into.  Compaction (at the level
// end, before the tail, or when the table fills) renumbers the live nodes,
// rewrites their rows and composes the point map through rep.  Marks hold
// stamps (a round counter), so nothing is cleared between rounds.  The
// decisions are those of the renumbering rounds: the same sums, means,
// rows and weights, only under other ids (and the tie rule uses minpt).
// ---------------------------------------------------------------------------
// Slot of a list append made by the lanes of a wave with `take` set: one
// atomic on the counter per wave (millions of appends to one counter
// would serialise at the memory side).  Every lane of the wave must call
// it; returns -1 for the lanes that do not append.
__device__ __forceinline__ int32_t wave_slot(bool take, int32_t *counter) {
  const uint64_t m = __ballot(take);
  if (!m) return -1;
  const int lane = threadIdx.x & (kWave - 1);
  const int leader = __builtin_ctzll(m);
  int32_t base = 0;
  if (lane == leader) base = atomicAdd(counter, __popcll(m));
  base = __shfl(base, leader, kWave);
  return take ? base + __popcll(m & ((1ull << lane) - 1)) : -1;
}

__global__ __launch_bounds__(256) void k_incr_init(
    int32_t nn, int32_t *target, int32_t *parent, int32_t *rep, int32_t *rcap,
    int32_t *rmark, int32_t *fixmark, int32_t *wmark, long long span,
    Ctl *ctl) {
  const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v == 0) {
    ctl->n_work = 0;
    ctl->span_live = span;
  }
  if (v >= nn) return;
  target[v] = -1;
  parent[v] = v;
  rep[v] = v;
  rcap[v] = 0;
  rmark[v] = -1;
  fixmark[v] = -1;
  wmark[v] = -1;
}

// First worklist after a renumbering round: the nodes formed by a merge and
// their neighbours (the nodes selection would evaluate).
__global__ __launch_bounds__(256) void k_build_work(
    int32_t nn, Adj a, const uint8_t *__restrict__ merged,
    int32_t *__restrict__ work, int32_t *__restrict__ cnt, Ctl *ctl) {
  const int32_t v = xcd_tid();
  bool take = false;
  if (v < nn) {
    take = merged[v] != 0;
    int32_t k = 0;
    for_row<false>(a, v, 0, 1, [&](int32_t u, int32_t) {
      ++k;
      if ((uint32_t)u < (uint32_t)nn && merged[u]) take = true;
    });
    cnt[v] = k;  // entries of the row (its span may hold empty slots)
  }
  const uint64_t m = __ballot(take);
  if (!m) return;
  const int lane = threadIdx.x & (kWave - 1);
  int32_t base = 0;
  if (lane == __builtin_ctzll(m)) base = atomicAdd(&ctl->n_work, __popcll(m));
  base = __shfl(base, __builtin_ctzll(m), kWave);
  if (take) work[base + __popcll(m & ((1ull << lane) - 1))] = v;
}

__global__ void k_incr_round_init(Ctl *ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctl->n_roots = 0;
    ctl->n_fix = 0;
    ctl->n_work = 0;
    ctl->n_dead = 0;
    ctl->win_total = 0;
    ctl->n_members = 0;
    ctl->n_contrib = 0;
    ctl->n_owners = 0;
    ctl->chunk_total = 0;
    ctl->n_lfill = 0;
  }
}

// Step 3 on the worklist (every other node keeps parent = itself and
// target = -1): hook, then the capped jumping walk of k_jump.
__global__ __launch_bounds__(256) void k_hook_w(int32_t n_work,
                                                const int32_t *work,
                                                const int32_t *target,
                                                int32_t *parent, int32_t nn,
                                                Ctl *ctl) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_work) return;
  const int32_t v = work[i];
  if ((uint32_t)v >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
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

__global__ __launch_bounds__(256) void k_jump_w(int32_t n_work,
                                                const int32_t *work,
                                                int32_t *parent, int32_t nn,
                                                Ctl *ctl) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_work) return;
  const int32_t v = work[i];
  int32_t p = parent[v];
  int it = 0;
  for (; it < kJumpWalk; ++it) {
    if ((uint32_t)p >= (uint32_t)nn) {
      raise_err(ctl, kErrInternal);
      p = v;
      break;
    }
    const int32_t pp = __atomic_load_n(&parent[p], __ATOMIC_RELAXED);
    if (pp == p) break;
    p = pp;
  }
  __atomic_store_n(&parent[v], p, __ATOMIC_RELAXED);
  if (it == kJumpWalk) __atomic_store_n(&ctl->any_choice, -1, __ATOMIC_RELAXED);
}

// Step 4 statistics of the merged components: every member adds its size,
// smallest point, entry count and exact sums into its root and records the
// root in rep; it enters the contributor list (its row goes into its
// root's new row); each root enters the root list once.  A block first
// combines its members' values per root in LDS (a component absorbing
// thousands of nodes in one round would otherwise serialise on its root's
// addresses), then adds each root's share with one atomic per value.
constexpr int kMergeSlots = 256;  // = block size: room for every key
template <int DT>
__global__ __launch_bounds__(256) void k_incr_merge(
    int32_t n_work, const int32_t *__restrict__ work,
    const int32_t *__restrict__ parent, int32_t *size, int64_t *S,
    int32_t *minpt, const int32_t *__restrict__ wl,
    const int32_t *__restrict__ cnt, int32_t *rep, int32_t *rmark,
    int32_t *roots, int32_t *rcap, int32_t *cy, int32_t *cY, int32_t d,
    int32_t stamp, Ctl *ctl) {
  constexpr int SD = DT > 0 ? DT : 1;
  __shared__ int32_t h_key[kMergeSlots], h_size[kMergeSlots],
      h_min[kMergeSlots], h_cnt[kMergeSlots];
  __shared__ unsigned long long h_S[kMergeSlots * SD];
  if (!round_live(ctl)) return;
  const int t = threadIdx.x;
  h_key[t] = -1;
  h_size[t] = 0;
  h_min[t] = INT32_MAX;
  h_cnt[t] = 0;
  if constexpr (DT > 0)
    for (int q = 0; q < DT; ++q) h_S[q * kMergeSlots + t] = 0ull;
  __syncthreads();
  const int32_t i = blockIdx.x * blockDim.x + t;
  int32_t v = -1, r = -1;
  if (i < n_work) {
    v = work[i];
    r = parent[v];
  }
  const bool member = v >= 0 && r != v;
  long long gone = 0;
  if (member) {
    uint32_t h = ((uint32_t)r * 2654435761u) % kMergeSlots;
    for (;;) {  // at most one key per thread: a slot is always found
      const int32_t k = atomicCAS(&h_key[h], -1, r);
      if (k == -1 || k == r) break;
      h = (h + 1) % kMergeSlots;
    }
    atomicAdd(&h_size[h], size[v]);
    atomicMin(&h_min[h], minpt[v]);
    atomicAdd(&h_cnt[h], cnt[v]);
    if constexpr (DT > 0) {
      const longlong2 *p = reinterpret_cast<const longlong2 *>(S + (int64_t)v * DT);
#pragma unroll
      for (int q = 0; q < DT / 2; ++q) {
        const longlong2 x = p[q];
        atomicAdd(&h_S[(2 * q) * kMergeSlots + h], (unsigned long long)x.x);
        atomicAdd(&h_S[(2 * q + 1) * kMergeSlots + h], (unsigned long long)x.y);
      }
    } else {
      for (int32_t q = 0; q < d; ++q)
        atomicAdd(reinterpret_cast<unsigned long long *>(&S[(int64_t)r * d + q]),
                  (unsigned long long)S[(int64_t)v * d + q]);
    }
    rep[v] = r;
    gone = wl[v];
  }
  const int32_t c = wave_slot(member, &ctl->n_contrib);
  if (c >= 0) {
    cy[c] = v;
    cY[c] = r;
  }
  const int32_t dead = wave_sum(member ? 1 : 0);
  gone = wave_sum(gone);
  if ((t & (kWave - 1)) == 0 && dead) {
    atomicAdd(&ctl->n_dead, dead);
    atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->span_live),
              (unsigned long long)(-gone));
  }
  __syncthreads();
  // flush: one thread per slot
  const int32_t R = h_key[t];
  bool fresh = false;
  if (R >= 0) {
    atomicAdd(&size[R], h_size[t]);
    atomicMin(&minpt[R], h_min[t]);
    atomicAdd(&rcap[R], h_cnt[t]);
    if constexpr (DT > 0)
      for (int q = 0; q < DT; ++q)
        atomicAdd(reinterpret_cast<unsigned long long *>(&S[(int64_t)R * DT + q]),
                  h_S[q * kMergeSlots + t]);
    fresh = atomicExch(&rmark[R], stamp) != stamp;
  }
  const int32_t o = wave_slot(fresh, &ctl->n_roots);
  if (o >= 0) roots[o] = R;
}

// Per root: its new means, the capacity of its new window (twice the
// entries of its own row and its members'), its place in the owner list
// (roots first), and itself as a contributor and on the next worklist.
__global__ __launch_bounds__(256) void k_incr_roots(
    const int32_t *__restrict__ roots, const int32_t *__restrict__ size,
    const int64_t *__restrict__ S, double *mu, const int32_t *__restrict__ wl,
    const int32_t *__restrict__ cnt, int32_t *rcap, int32_t *ocap,
    int32_t *rpos, int32_t *cy, int32_t *cY, int32_t *wmark, int32_t d,
    int32_t stamp, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t nr = ctl->n_roots;
  const int32_t nm = ctl->n_members;  // members' contributor entries
  const double sIF = ldexp(1.0, -ctl->F);
  long long gone = 0;
  const int lane = threadIdx.x & (kWave - 1);
  for (int32_t i0 = blockIdx.x * blockDim.x + (threadIdx.x - lane); i0 < nr;
       i0 += gridDim.x * blockDim.x) {  // wave-uniform: wave_slot below
    const int32_t i = i0 + lane;
    if (i >= nr) continue;
    const int32_t r = roots[i];
    wmark[r] = stamp;  // on the next worklist
    const int64_t ent = (int64_t)rcap[r] + cnt[r];
    rcap[r] = 0;
    gone += wl[r];
    // the host keeps top + 2 * (live slots) within the table, so a window
    // fits; the clamp only keeps a corrupt count from wrapping
    ocap[i] = (int32_t)std::min<int64_t>(std::max<int64_t>(2 * ent, 1),
                                         INT32_MAX / 2);
    rpos[r] = i;
    cy[nm + i] = r;
    cY[nm + i] = r;
    const double dsz = (double)size[r];
    for (int32_t q = 0; q < d; ++q) {
      const double qv = (double)S[(int64_t)r * d + q] / dsz;
      mu[(int64_t)r * d + q] = qv * sIF;
    }
  }
  gone = wave_sum(gone);
  if ((threadIdx.x & (kWave - 1)) == 0 && gone)
    atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->span_live),
              (unsigned long long)(-gone));
}

// Counts fixed between the kernels of a round: the members' contributor
// entries, then the owners (roots, then long rebuilt rows) and all
// contributors.
__global__ void k_incr_counts(Ctl *ctl, int stage) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  if (stage == 0) {
    ctl->n_members = ctl->n_contrib;
  } else if (stage == 1) {
    ctl->n_contrib = ctl->n_members + ctl->n_roots;
    ctl->n_owners = ctl->n_roots;
  }
}

// Rows to fix, kIncrLanes lanes per member (from the contributor list):
// every unmerged live node the member lists is flagged (its entry for the
// member now belongs to the member's root).
constexpr int kIncrLanes = 8;
__global__ __launch_bounds__(256) void k_incr_mark(
    const int32_t *__restrict__ cy, const int32_t *__restrict__ parent,
    const int32_t *__restrict__ rmark, Adj a, int32_t *fixmark, int32_t nn,
    int32_t stamp, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t nm = ctl->n_members;
  const int32_t tid = blockIdx.x * blockDim.x + threadIdx.x;
  const int lg = tid & (kIncrLanes - 1);
  for (int32_t i = tid / kIncrLanes; i < nm;
       i += gridDim.x * blockDim.x / kIncrLanes) {
    for_row<false>(a, cy[i], lg, kIncrLanes, [&](int32_t u, int32_t) {
      if ((uint32_t)u >= (uint32_t)nn) {
        raise_err(ctl, kErrInternal);
        return;
      }
      if (parent[u] == u && rmark[u] != stamp) fixmark[u] = stamp;
    });
  }
}

// A pass over all nodes: each flagged row to fix either goes to the owner
// list (rows longer than kFixInPlace slots are rebuilt like a root's, with
// themselves as the one contributor) or is fixed in place: every entry
// whose relabelled neighbour X (its root) was formed this round is, at the
// first entry with that X, replaced by (X, the summed weights of all of
// them), and emptied at the others.  Entries are taken in order, so an
// earlier entry already rewritten still carries its X (a root is its own
// parent).
constexpr int32_t kFixInPlace = 64;
__global__ __launch_bounds__(256) void k_incr_fixpass(
    int32_t nn, const int32_t *__restrict__ fixmark,
    const int32_t *__restrict__ parent, const int32_t *__restrict__ rmark,
    const int32_t *__restrict__ ws, const int32_t *__restrict__ wl,
    uint64_t *tbl, int32_t *cnt, int32_t *owners, int32_t *ocap,
    int32_t *rpos, int32_t *cy, int32_t *cY, int32_t stamp, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t v = xcd_tid();
  const bool fix = v < nn && fixmark[v] == stamp;
  const bool rebuild = fix && wl[v] > kFixInPlace;
  const int32_t o = wave_slot(rebuild, &ctl->n_owners);
  const int32_t c = wave_slot(rebuild, &ctl->n_contrib);
  long long gone = 0;
  if (rebuild) {
    owners[o] = v;
    ocap[o] = (int32_t)std::min<int64_t>(
        std::max<int64_t>(2 * (int64_t)cnt[v], 1), INT32_MAX / 2);
    rpos[v] = o;
    cy[c] = v;
    cY[c] = v;
    gone = wl[v];
  } else if (fix) {
    uint64_t *row = tbl + ws[v];
    const int32_t len = wl[v];
    auto label = [&](uint64_t e) {
      const int32_t y = (int32_t)(e >> 32);
      return (uint32_t)y < (uint32_t)nn ? parent[y] : -1;
    };
    int32_t emptied = 0;
    for (int32_t j = 0; j < len; ++j) {
      const uint64_t e = row[j];
      if (e == kEmpty) continue;
      const int32_t X = label(e);
      if (X < 0) {
        raise_err(ctl, kErrInternal);
        continue;
      }
      if (rmark[X] != stamp) continue;  // not a merged component
      bool first = true;
      for (int32_t i = 0; i < j && first; ++i) {
        const uint64_t q = row[i];
        if (q != kEmpty && label(q) == X) first = false;
      }
      if (!first) {
        row[j] = kEmpty;
        ++emptied;
        continue;
      }
      uint32_t w = (uint32_t)e;
      for (int32_t i = j + 1; i < len; ++i) {
        const uint64_t q = row[i];
        if (q != kEmpty && label(q) == X) w += (uint32_t)q;
      }
      row[j] = ((uint64_t)(uint32_t)X << 32) | w;
    }
    if (emptied) cnt[v] -= emptied;
  }
  gone = wave_sum(gone);
  if ((threadIdx.x & (kWave - 1)) == 0 && gone)
    atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->span_live),
              (unsigned long long)(-gone));
}

// The owners' new windows start at `top`, past every live window; each
// owner's entry count restarts at 0 for the fill to count.
__global__ __launch_bounds__(256) void k_incr_clear(
    const int32_t *__restrict__ owners, const int32_t *__restrict__ obase,
    const int32_t *__restrict__ ocap, uint64_t *tbl, int32_t *cnt,
    int64_t top, int64_t tcap, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t no = ctl->n_owners;
  for (int32_t o = blockIdx.x; o < no; o += gridDim.x) {
    const int64_t base = top + obase[o];
    const int32_t cp = ocap[o];
    if (base + cp > tcap) {
      raise_err(ctl, kErrInternal);
      continue;
    }
    if (threadIdx.x == 0) cnt[owners[o]] = 0;
    for (int32_t t = threadIdx.x; t < cp; t += blockDim.x)
      tbl[base + t] = kEmpty;
  }
}

// Contraction into the owners' new windows: every entry of a contributor's
// row, relabelled to its root, is added to its owner's window (edges inside
// the owner's component are dropped, parallel edges add their weights);
// new slots are counted, and a root's neighbours are flagged for the next
// worklist.  kIncrLanes lanes per contributor; rows longer than kLongFill
// slots are listed in chunks of kLongFill for k_incr_fill_long.
constexpr int32_t kLongFill = 1024;
__device__ __forceinline__ int32_t incr_add(
    uint64_t e, int32_t Y, bool root, const int32_t *__restrict__ parent,
    uint64_t *tbl, int64_t base, int32_t cp, int32_t *wmark, int32_t nn,
    int32_t stamp, Ctl *ctl) {
  if (e == kEmpty) return 0;
  const int32_t u = (int32_t)(e >> 32);
  if ((uint32_t)u >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return 0;
  }
  const int32_t U = parent[u];
  if (U == Y) return 0;
  if (!table_add(tbl, 0, cp, U, (int32_t)(uint32_t)e, ctl, base)) return 0;
  if (root) wmark[U] = stamp;
  return 1;
}

__global__ __launch_bounds__(256) void k_incr_fill(
    const int32_t *__restrict__ cy, const int32_t *__restrict__ cY,
    const int32_t *__restrict__ parent, const int32_t *__restrict__ rmark,
    const int32_t *__restrict__ rpos, const int32_t *__restrict__ obase,
    const int32_t *__restrict__ ocap, Adj a, uint64_t *tbl, int32_t *cnt,
    int32_t *wmark, int32_t *lch_i, int32_t *lch_j, int32_t lch_cap,
    int64_t top, int64_t tcap, int32_t nn, int32_t stamp, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t nc = ctl->n_contrib;
  const int32_t tid = blockIdx.x * blockDim.x + threadIdx.x;
  const int lg = tid & (kIncrLanes - 1);
  for (int32_t i = tid / kIncrLanes; i < nc;
       i += gridDim.x * blockDim.x / kIncrLanes) {
    const int32_t y = cy[i], Y = cY[i];
    const int32_t o = rpos[Y];
    const int64_t base = top + obase[o];
    const int32_t cp = ocap[o];
    if (base + cp > tcap) continue;  // k_incr_clear raised the error
    const int32_t span = a.wl[y];
    if (span > kLongFill) {
      if (lg == 0) {
        const int32_t nch = (span + kLongFill - 1) / kLongFill;
        const int32_t c0 = atomicAdd(&ctl->n_lfill, nch);
        if (c0 + nch > lch_cap) {
          raise_err(ctl, kErrInternal);
        } else {
          for (int32_t q = 0; q < nch; ++q) {
            lch_i[c0 + q] = i;
            lch_j[c0 + q] = q * kLongFill;
          }
        }
      }
      continue;
    }
    const bool root = rmark[Y] == stamp;
    const uint64_t *row = a.tbl + a.ws[y];
    int32_t added = 0;
    for (int32_t j = lg; j < span; j += kIncrLanes)
      added += incr_add(row[j], Y, root, parent, tbl, base, cp, wmark, nn,
                        stamp, ctl);
    if (added) atomicAdd(&cnt[Y], added);
  }
}

// The chunks of the long contributor rows, a wave each.
__global__ __launch_bounds__(256) void k_incr_fill_long(
    const int32_t *__restrict__ cy, const int32_t *__restrict__ cY,
    const int32_t *__restrict__ parent, const int32_t *__restrict__ rmark,
    const int32_t *__restrict__ rpos, const int32_t *__restrict__ obase,
    const int32_t *__restrict__ ocap, Adj a, uint64_t *tbl, int32_t *cnt,
    int32_t *wmark, const int32_t *__restrict__ lch_i,
    const int32_t *__restrict__ lch_j, int64_t top, int32_t nn,
    int32_t stamp, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t nch = ctl->n_lfill;
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t wave0 = (int32_t)(blockIdx.x * (blockDim.x / kWave) +
                                  threadIdx.x / kWave);
  const int32_t nwaves = (int32_t)(gridDim.x * (blockDim.x / kWave));
  for (int32_t c = wave0; c < nch; c += nwaves) {
    const int32_t i = lch_i[c];
    const int32_t y = cy[i], Y = cY[i];
    const int32_t o = rpos[Y];
    const int64_t base = top + obase[o];
    const int32_t cp = ocap[o];
    const bool root = rmark[Y] == stamp;
    const uint64_t *row = a.tbl + a.ws[y];
    const int32_t j1 = min(a.wl[y], lch_j[c] + kLongFill);
    int32_t added = 0;
    for (int32_t j = lch_j[c] + lane; j < j1; j += kWave)
      added += incr_add(row[j], Y, root, parent, tbl, base, cp, wmark, nn,
                        stamp, ctl);
    added = wave_sum(added);
    if (lane == 0 && added) atomicAdd(&cnt[Y], added);
  }
}

// The owners' rows are their new windows (empty slots included).
__global__ __launch_bounds__(256) void k_incr_owners(
    const int32_t *__restrict__ owners, const int32_t *__restrict__ obase,
    const int32_t *__restrict__ ocap, int32_t *ws, int32_t *wl, int64_t top,
    Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t no = ctl->n_owners;
  long long added = 0;
  for (int32_t o = blockIdx.x * blockDim.x + threadIdx.x; o < no;
       o += gridDim.x * blockDim.x) {
    const int32_t Y = owners[o];
    ws[Y] = (int32_t)(top + obase[o]);
    wl[Y] = ocap[o];
    added += ocap[o];
  }
  added = wave_sum(added);
  if ((threadIdx.x & (kWave - 1)) == 0 && added)
    atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->span_live),
              (unsigned long long)added);
}

// The next worklist: every node flagged with this round's stamp (the roots
// and their neighbours), in id order within each wave.
__global__ __launch_bounds__(256) void k_incr_nextwork(
    int32_t nn, const int32_t *__restrict__ wmark, int32_t *work_next,
    int32_t stamp, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t v = xcd_tid();
  const int32_t slot = wave_slot(v < nn && wmark[v] == stamp, &ctl->n_work);
  if (slot >= 0) work_next[slot] = v;
}

// The worklist's nodes back to target = -1 and parent = themselves.
__global__ __launch_bounds__(256) void k_incr_cleanup(
    int32_t n_work, const int32_t *__restrict__ work, int32_t *target,
    int32_t *parent, Ctl *ctl) {
  if (!round_live(ctl)) return;
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_work) return;
  const int32_t v = work[i];
  target[v] = -1;
  parent[v] = v;
}

// Compaction: live nodes (rep[v] == v once rep is resolved to roots)
// numbered in id order.
struct ScanLive {
  const int32_t *rep;
  int32_t *newid;
  int32_t nn;
  __device__ int32_t value(int32_t v) const {
    return (v < nn && rep[v] == v) ? 1 : 0;
  }
  __device__ void emit(int32_t v, int32_t excl, int32_t val) const {
    if (val) newid[v] = excl;
  }
};

// One pointer-doubling pass over rep (dead nodes' chains to their roots).
__global__ __launch_bounds__(256) void k_rep_double(int32_t nn, int32_t *rep,
                                                    Ctl *ctl) {
  const int32_t v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= nn) return;
  const int32_t p = rep[v];
  if ((uint32_t)p >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
  const int32_t pp = rep[p];
  if (pp != p) {
    rep[v] = pp;
    ctl->jump_changed = 1;
  }
}

// Node state of the live nodes under their new ids (means recomputed from
// the sums, bit for bit as the statistics compute them), the entry count
// of their rows, and the merged flag of the last round's roots.
__global__ __launch_bounds__(256) void k_compact_nodes(
    int32_t nn, const int32_t *__restrict__ rep,
    const int32_t *__restrict__ newid, NodeIn s, int32_t *size_o,
    int32_t *minpt_o, int64_t *S_o, double *mu, Adj a, int32_t *cnt,
    const int32_t *__restrict__ rmark, int32_t last_stamp, uint8_t *merged,
    int32_t d, Ctl *ctl) {
  const int32_t v = xcd_tid();
  if (v >= nn || rep[v] != v) return;
  const int32_t c = newid[v];
  size_o[c] = s.size[v];
  minpt_o[c] = s.minpt[v];
  for (int32_t q = 0; q < d; ++q)
    S_o[(int64_t)c * d + q] = s.S[(int64_t)v * d + q];
  int32_t k = 0;
  for_row<false>(a, v, 0, 1, [&](int32_t, int32_t) { ++k; });
  cnt[c] = k;
  merged[c] = rmark[v] == last_stamp ? 1 : 0;
}

// Means of the compacted nodes (a second pass: the old means of other
// nodes may sit where a new one goes).
__global__ __launch_bounds__(256) void k_compact_mu(int32_t nl,
                                                    const int32_t *size,
                                                    const int64_t *S,
                                                    double *mu, int32_t d,
                                                    Ctl *ctl) {
  const int32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= nl * d) return;
  const double sIF = ldexp(1.0, -ctl->F);
  const double qv = (double)S[t] / (double)size[t / d];
  mu[t] = qv * sIF;
}

// Rows of the live nodes, their entries relabelled, packed into the other
// table buffer from the offsets of the scan.
__global__ __launch_bounds__(256) void k_compact_rows(
    int32_t nn, const int32_t *__restrict__ rep,
    const int32_t *__restrict__ newid, Adj a, const int32_t *__restrict__ ws_o,
    int32_t *wl_o, uint64_t *tbl_o, Ctl *ctl) {
  const int32_t v = xcd_tid();
  if (v >= nn || rep[v] != v) return;
  const int32_t c = newid[v];
  uint64_t *out = tbl_o + ws_o[c];
  int32_t k = 0;
  for_row<false>(a, v, 0, 1, [&](int32_t u, int32_t w) {
    if ((uint32_t)u >= (uint32_t)nn || rep[u] != u) {
      raise_err(ctl, kErrInternal);
      return;
    }
    out[k++] = ((uint64_t)(uint32_t)newid[u] << 32) | (uint32_t)w;
  });
  wl_o[c] = k;
}

// The point map through the dead nodes' roots and the new ids.
__global__ __launch_bounds__(256) void k_compose_rep(
    int32_t n, int32_t nn, int32_t *M, const int32_t *__restrict__ rep,
    const int32_t *__restrict__ newid, Ctl *ctl) {
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const int32_t c = M[i];
  if ((uint32_t)c >= (uint32_t)nn) {
    raise_err(ctl, kErrInternal);
    return;
  }
  M[i] = newid[rep[c]];
}

struct Bufs {
  float *emb_int;
  int32_t *nbr_clean;                   // sanitised caller table
  int32_t *rrp, *rcol, *rev, *cursor;  // first-round reverse lists
  uint64_t *nmask;                      // non-mutual entries of each row
  int32_t *ws[2], *wl[2];               // row windows (= toff, cap)
  uint64_t *tbl[2];
  int32_t *size[2], *minpt[2];
  int64_t *S[2];
  double *mu;
  int32_t *target, *deg, *parent, *newid, *L, *cnt, *rank, *moff, *mem;
  int32_t *long_rows, *big, *cbig, *capn, *tile_c, *tile_i;
  int32_t *lbase, *lnch, *litem, *lmp, *lu, *lcnt;  // long-row chunks
  double *lg;
  int32_t lcap;
  int32_t *cstart;  // first component of every contraction chunk
  int32_t qcap;     // entries of cstart
  int32_t *M, *mark, *lrank;
  int32_t *Mn;  // node map of the rounds since M was last brought up to date
  uint8_t *merged;  // per node: formed by a merge in the last round
  // incremental rounds
  int32_t *work[2];  // this round's worklist, the next one
  int32_t *rep, *rcap, *rmark, *fixmark, *wmark, *roots, *rcapl, *rbase,
      *rpos, *fixl;
  int32_t *ecnt;      // entries of every row
  int32_t *cy, *cY;   // contributor rows and their owners
  int32_t *lch_i, *lch_j;  // chunks of long contributor rows
  int32_t lch_cap;
  int32_t nt;  // nodes the tail can start from
  double *tgain;    // per-edge gains in the tail
  uint64_t *telist; // the tail's edges to evaluate
  int32_t tslots;   // entries of tgain and telist
  int32_t *lvl_map, *lvl_minpt, *lvl_rank;
  double *lvl_mu;
  int32_t *bsum, *tmp;
  double *partial;
  // linking of isolated nodes (only with the flag)
  bool link;
  const float4 *pts;  // points in internal order (linking only)
  int64_t *lk_sx[2];  // position sums of the nodes, double-buffered
  double *lk_cen;
  int32_t *lk_cnt, *lk_iso, *lk_iso_of, *lk_ext, *lk_fill, *lk_near;
  uint8_t *lk_keep;
};

int64_t edge_bound(int32_t n, int32_t k) { return 2 * (int64_t)n * k; }

void carve(Arena &a, int32_t n, int32_t d, int32_t k, bool link, Bufs *b) {
  const int64_t ed = edge_bound(n, k);
  const size_t n1 = (size_t)n + 1;
  b->emb_int = a.take<float>((size_t)n * d);
  b->nbr_clean = a.take<int32_t>((size_t)n * pad4(k));
  b->rrp = a.take<int32_t>(n1);
  b->rcol = a.take<int32_t>((size_t)n * k);
  b->rev = a.take<int32_t>(n1);
  b->cursor = a.take<int32_t>(n1);
  b->nmask = a.take<uint64_t>(n1);
  for (int j = 0; j < 2; ++j) {
    b->ws[j] = a.take<int32_t>(n1);
    b->wl[j] = a.take<int32_t>(n1);
    b->tbl[j] = a.take<uint64_t>(2 * ed);  // big windows take twice
    b->size[j] = a.take<int32_t>(n1);
    b->minpt[j] = a.take<int32_t>(n1);
    b->S[j] = a.take<int64_t>((size_t)n * d);
  }
  b->mu = a.take<double>((size_t)n * d);
  b->target = a.take<int32_t>(n1);
  b->deg = a.take<int32_t>(n1);
  b->parent = a.take<int32_t>(n1);
  b->newid = a.take<int32_t>(n1);
  b->L = a.take<int32_t>(n1);
  b->cnt = a.take<int32_t>(n1);
  b->rank = a.take<int32_t>(n1);
  b->moff = a.take<int32_t>(n1);
  b->mem = a.take<int32_t>(n1);
  b->long_rows = a.take<int32_t>(n1);
  b->lbase = a.take<int32_t>(n1);
  b->lnch = a.take<int32_t>(n1);
  b->lcap = (int32_t)(n1 + ed / kLongChunk + 64);
  b->litem = a.take<int32_t>(b->lcap);
  b->lmp = a.take<int32_t>(b->lcap);
  b->lu = a.take<int32_t>(b->lcap);
  b->lcnt = a.take<int32_t>(b->lcap);
  b->lg = a.take<double>(b->lcap);
  b->big = a.take<int32_t>(n1);
  b->cbig = a.take<int32_t>(n1);
  b->capn = a.take<int32_t>(n1);
  b->tile_c = a.take<int32_t>(2 * n1);
  b->tile_i = a.take<int32_t>(2 * n1);
  b->qcap = (int32_t)(2 * ed / 64 + 16);  // chunks are >= 64 slots
  b->cstart = a.take<int32_t>(b->qcap);
  b->M = a.take<int32_t>(n1);
  b->Mn = a.take<int32_t>(n1);
  b->merged = a.take<uint8_t>(n1);
  b->work[0] = a.take<int32_t>(n1);
  b->work[1] = a.take<int32_t>(n1);
  b->rep = a.take<int32_t>(n1);
  b->rcap = a.take<int32_t>(n1);
  b->rmark = a.take<int32_t>(n1);
  b->fixmark = a.take<int32_t>(n1);
  b->wmark = a.take<int32_t>(n1);
  b->roots = a.take<int32_t>(n1);
  b->rcapl = a.take<int32_t>(n1 + 1);
  b->rbase = a.take<int32_t>(n1 + 1);
  b->rpos = a.take<int32_t>(n1);
  b->fixl = a.take<int32_t>(n1);
  b->ecnt = a.take<int32_t>(n1);
  b->cy = a.take<int32_t>(n1);
  b->cY = a.take<int32_t>(n1);
  b->lch_cap = (int32_t)(n1 + 2 * ed / kLongFill + 64);
  b->lch_i = a.take<int32_t>(b->lch_cap);
  b->lch_j = a.take<int32_t>(b->lch_cap);
  b->mark = a.take<int32_t>(n1);
  b->lrank = a.take<int32_t>(n1);
  b->nt = std::min<int32_t>(n, kTailNodes);
  b->tslots = (int32_t)std::min<int64_t>(2 * ed, kTailSlots);
  b->tgain = a.take<double>(b->tslots);
  b->telist = a.take<uint64_t>(b->tslots);
  b->lvl_map = a.take<int32_t>((size_t)kTailLevels * b->nt);
  b->lvl_minpt = a.take<int32_t>((size_t)kTailLevels * b->nt);
  b->lvl_rank = a.take<int32_t>((size_t)kTailLevels * b->nt);
  b->lvl_mu = a.take<double>((size_t)kTailLevels * b->nt * d);
  b->bsum = a.take<int32_t>(scan_blocks(ed + n1) + 2);
  b->tmp = a.take<int32_t>(8);
  b->partial = a.take<double>(kEnergyBlocks);
  b->link = link;
  b->pts = nullptr;
  b->lk_sx[0] = b->lk_sx[1] = nullptr;
  b->lk_cen = nullptr;
  b->lk_cnt = b->lk_iso = b->lk_iso_of = b->lk_ext = b->lk_fill = nullptr;
  b->lk_near = nullptr;
  b->lk_keep = nullptr;
  if (link) {
    b->lk_sx[0] = a.take<int64_t>(3 * n1);
    b->lk_sx[1] = a.take<int64_t>(3 * n1);
    b->lk_cen = a.take<double>(3 * n1);
    b->lk_cnt = a.take<int32_t>(n1);
    b->lk_iso = a.take<int32_t>(n1);
    b->lk_iso_of = a.take<int32_t>(n1);
    b->lk_ext = a.take<int32_t>(n1);
    b->lk_fill = a.take<int32_t>(n1);
    b->lk_near = a.take<int32_t>(n1 * (size_t)k);
    b->lk_keep = a.take<uint8_t>(n1 * (size_t)k);
  }
}


inline dim3 blocks_for(int64_t n, int nt = 256) {
  int64_t b = (n + nt - 1) / nt;
  if (b < 1) b = 1;
  return dim3((unsigned)b);
}
inline dim3 xblocks_for(int64_t n) { return dim3(xcd_grid(blocks_for(n).x)); }


// Brings the point map up to date through the node map of the rounds since
// (mn nodes; nothing to do when mn is 0), and resets mn.
void sync_map(const Bufs &b, int32_t n, int32_t &mn, Ctl *ctl,
              hipStream_t st) {
  if (mn == 0) return;
  hipLaunchKernelGGL(k_sync_map, xblocks_for(n), dim3(256), 0, st, n, mn, b.M,
                     b.Mn, ctl);
  mn = 0;
}

// One merge round on nn nodes whose rows hold ed directed entries.
// With rest_only, only the kernels after pointer jumping are launched: the
// second half of a round whose jumping the host completed (finish_jump).
// mn: nodes of the node map Mn (0: the point map M is up to date).
template <bool FIRST, int DT>
void launch_round(const Bufs &b, const Adj &adj, int cur, int32_t n,
                  int32_t k, int32_t nn, int32_t ed, int32_t d,
                  const NodeIn &s, double lambda, int64_t smin, Ctl *ctl,
                  hipStream_t st, bool rest_only, int32_t mn) {
  const int nxt = 1 - cur;
  const int32_t tcap = (int32_t)(2 * edge_bound(n, k));
  // G lanes per short row; long rows in chunks of entries, a wave each
  const LongWork lw{b.long_rows, b.lbase, b.lnch, b.litem, b.lg,
                    b.lmp,       b.lu,    b.lcnt, b.lcap};
  const dim3 long_grid((unsigned)std::max<int64_t>(
      1, std::min<int64_t>(kLongGrid, ((int64_t)ed / kLongChunk + nn) / 4 + 1)));
  const dim3 big_grid(
      (unsigned)std::max<int64_t>(1, std::min<int64_t>(kBigGrid, nn / 16)));
  if (!rest_only) {
    hipLaunchKernelGGL(k_round_init, dim3(1), dim3(64), 0, st, ctl);
    prof_begin("select", st);
    constexpr int G = FIRST ? kSelLanesFirst : kSelLanes;
    if constexpr (FIRST && DT > 0) {
      constexpr int32_t R = kSelFirstBytes / (4 * DT);
      hipLaunchKernelGGL((k_select_first<DT, G>),
                         dim3(xcd_grid(((int64_t)nn + R - 1) / R)),
                         dim3(kSelFirstNT),
                         0, st, nn, adj, s, lambda, smin, b.target, b.deg, lw,
                         ctl);
    } else {
      hipLaunchKernelGGL((k_select<FIRST, DT, G>),
                         xblocks_for((int64_t)nn * G), dim3(256), 0, st, nn,
                         adj, s, d, lambda, smin, b.target, b.deg, lw,
                         (const int32_t *)nullptr, 0, ctl);
    }
    hipLaunchKernelGGL((k_select_long<FIRST, DT>), long_grid, dim3(256), 0,
                       st, nn, adj, s, d, lambda, smin, lw, ctl);
    hipLaunchKernelGGL(k_select_combine, dim3(64), dim3(256), 0, st, lw,
                       b.target, b.deg, ctl);
    prof_end(st);
  }
  prof_begin("union", st);
  if (!rest_only) {
    hipLaunchKernelGGL(k_hook, blocks_for(nn), dim3(256), 0, st, nn,
                       b.target, b.parent, ctl);
    hipLaunchKernelGGL(k_jump,
                       dim3(xcd_grid(((int64_t)nn + kJumpR - 1) / kJumpR)),
                       dim3(256), 0, st, nn,
                       b.parent, ctl);
  }
  device_scan(ScanRoots{b.parent, b.newid, b.cnt, nn}, nn, b.bsum,
              &ctl->n_next, st);
  hipLaunchKernelGGL(k_assign, xblocks_for(nn), dim3(256), 0, st, nn,
                     b.parent, b.newid, b.L, b.cnt, b.rank, ctl);
  prof_end(st);
  prof_begin("stats", st);
  device_scan(ScanArray{b.cnt, b.moff, nn, &ctl->n_next}, nn + 1, b.bsum,
              b.tmp, st);
  hipLaunchKernelGGL(k_place, xblocks_for(nn), dim3(256), 0, st, nn, b.L,
                     b.moff, b.rank, b.mem, b.merged, ctl);

  // contraction chunks: enough blocks to fill the chip, at most kChunk
  // (halved while fewer than 1024: measured faster than 2048 or 4096, and
  // than chunks of 512 slots throughout)
  int32_t chunk = kChunk;
  while (chunk > 64 && (int64_t)ed / chunk < 1024) chunk >>= 1;
  const NodeOut o{b.size[nxt], b.S[nxt],  b.mu,
                  b.minpt[nxt], b.capn,    b.wl[nxt],
                  b.cbig,      chunk,     kBigComp,
                  b.tile_c,    b.tile_i};
  if constexpr (DT > 0) {
    constexpr int G = kStatsLanes;
    hipLaunchKernelGGL((k_stats_s<FIRST, DT, G>),
                       xblocks_for((int64_t)nn * G + kXcd * G), dim3(256), 0,
                       st, nn, b.mem, b.moff, s, b.deg, o, b.big, ctl);
  } else {
    hipLaunchKernelGGL((k_stats<FIRST, DT>), xblocks_for(nn), dim3(256), 0,
                       st, nn, b.mem, b.moff, s, b.deg, d, o, b.big, ctl);
  }
  if constexpr (DT > 0)
    hipLaunchKernelGGL((k_stats_big_t<FIRST, DT>), big_grid, dim3(256), 0, st,
                       b.mem, b.moff, s, b.deg, o, b.big, ctl);
  else
    hipLaunchKernelGGL(k_stats_big<FIRST>, big_grid, dim3(256), 0, st,
                     b.mem, b.moff, s, b.deg, d, o, b.big, ctl);
  if (b.link) {  // position sums of the next round's nodes
    hipLaunchKernelGGL(k_link_accum<FIRST>, xblocks_for(nn), dim3(256), 0, st,
                       b.mem, b.moff, b.pts, b.lk_sx[cur], b.lk_sx[nxt], ctl);
    hipLaunchKernelGGL(k_link_accum_big<FIRST>, big_grid, dim3(256), 0, st,
                       b.mem, b.moff, b.pts, b.lk_sx[cur], b.lk_sx[nxt], b.big,
                       ctl);
  }
  prof_end(st);
  prof_begin("contract", st);
  device_scan(ScanWindows{b.capn, b.ws[nxt], &ctl->n_next, b.cstart, chunk,
                          b.qcap, ctl},
              nn + 1, b.bsum, &ctl->slots, st);
  hipLaunchKernelGGL(k_contract_chunk<FIRST>,
                     dim3(xcd_grid((ed + chunk - 1) / chunk)), dim3(256), 0,
                     st, nn, adj, b.L, b.mem, b.moff, b.ws[nxt], b.capn,
                     b.cstart, b.tbl[nxt], b.wl[nxt], chunk, ctl);
  hipLaunchKernelGGL(k_clear_big, big_grid, dim3(256), 0, st, b.cbig,
                     b.ws[nxt], b.capn, b.tbl[nxt], tcap, ctl);
  hipLaunchKernelGGL(k_contract_big<FIRST>, big_grid, dim3(256), 0, st, nn,
                     adj, b.L, b.mem, b.moff, b.ws[nxt], b.capn, b.tile_c,
                     b.tile_i, b.tbl[nxt], tcap, ctl);
  hipLaunchKernelGGL(k_contract_long<FIRST>, long_grid, dim3(256), 0, st, nn,
                     adj, b.L, b.ws[nxt], b.capn, chunk, lw, b.tbl[nxt], tcap,
                     ctl);
  prof_end(st);
  if (b.link) {  // the next round's empty rows, read back with the round
    prof_begin("link", st);
    hipLaunchKernelGGL(k_link_detect, xblocks_for(nn), dim3(256), 0, st,
                       b.ws[nxt], b.wl[nxt], b.tbl[nxt], b.lk_iso,
                       b.lk_iso_of, ctl);
    prof_end(st);
  }
  prof_begin("compose", st);
  if (FIRST)
    hipLaunchKernelGGL(k_compose_first, xblocks_for(n), dim3(256), 0, st, n,
                       b.M, b.L, ctl);
  else if (mn == 0)
    hipLaunchKernelGGL(k_compose_nodes<true>, xblocks_for(nn), dim3(256), 0,
                       st, nn, nn, b.Mn, b.L, ctl);
  else
    hipLaunchKernelGGL(k_compose_nodes<false>, xblocks_for(mn), dim3(256), 0,
                       st, mn, nn, b.Mn, b.L, ctl);
  prof_end(st);
}

// Dispatch on the embedding width: 8, 16 and 32 get unrolled kernels.
template <bool FIRST>
void round_d(const Bufs &b, const Adj &adj, int cur, int32_t n, int32_t k,
             int32_t nn, int32_t ed, int32_t d, const NodeIn &s,
             double lambda, int64_t smin, Ctl *ctl, hipStream_t st,
             int32_t mn, bool rest_only = false) {
  switch (d) {
    case 8:
      launch_round<FIRST, 8>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin,
                             ctl, st, rest_only, mn);
      break;
    case 16:
      launch_round<FIRST, 16>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin,
                              ctl, st, rest_only, mn);
      break;
    case 32:
      launch_round<FIRST, 32>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin,
                              ctl, st, rest_only, mn);
      break;
    default:
      launch_round<FIRST, 0>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin,
                             ctl, st, rest_only, mn);
  }
}

// Completes the merge forest of a round whose jumping walks stopped at
// their cap: doubling passes, four per readback, until a batch moves no
// parent.  Each pass at least halves the depth, which is below nn, so
// ceil(log2 nn) passes reach every root and one batch more sees no change;
// needing more is an internal error.
int finish_jump(const Bufs &b, int32_t nn, Ctl *ctl, Ctl *h, hipStream_t st) {
  int lg = 0;
  while (((int64_t)1 << lg) < (int64_t)nn) ++lg;
  const int batches = (lg + 3) / 4 + 1;
  for (int bt = 0; bt < batches; ++bt) {
    hipLaunchKernelGGL(k_jump_state, dim3(1), dim3(64), 0, st, ctl, 0);
    for (int j = 0; j < 4; ++j)
      hipLaunchKernelGGL(k_double, blocks_for(nn), dim3(256), 0, st, nn,
                         b.parent, ctl);
    int rc = read_ctl(ctl, h, st);
    if (rc) return rc;
    if (h->err) return status_from_err(h->err);
    if (!h->jump_changed) {
      hipLaunchKernelGGL(k_jump_state, dim3(1), dim3(64), 0, st, ctl, 1);
      return 0;
    }
  }
  set_error("pointer jumping did not reach the roots in %d passes",
            4 * batches);
  return -5;
}

// ---- incremental rounds: host side --------------------------------------
struct IncrState {
  bool on = false;
  int32_t n_work = 0;     // nodes of the current worklist
  int wc = 0;             // buffer of the current worklist
  int32_t stamp = 0;      // this round's mark value
  int64_t top = 0;        // table slots in use (windows lie below)
  int64_t span_live = 0;  // slots of the live rows (an upper bound)
  int32_t n_live = 0;     // live nodes
};

// A level switches to incremental rounds when a round kept more than this
// share of its nodes, on graphs of at least kIncrMinNodes nodes.
constexpr double kIncrKeep = 0.8;
constexpr int32_t kIncrMinNodes = 1 << 15;
constexpr int kIncrFlatBlocks = 4096;  // grid of the chunk-flattened kernels

// Starts incremental rounds on the nn nodes of the current table (its
// windows end at slot `slots`): identity forest, no marks, and the first
// worklist from the merged flags of the renumbering round just done.
int incr_enter(const Bufs &b, const Adj &adj, int32_t nn, int64_t slots,
               IncrState &is, Ctl *ctl, Ctl *h, hipStream_t st) {
  hipLaunchKernelGGL(k_incr_init, blocks_for(nn), dim3(256), 0, st, nn,
                     b.target, b.parent, b.rep, b.rcap, b.rmark, b.fixmark,
                     b.wmark, (long long)slots, ctl);
  hipLaunchKernelGGL(k_build_work, xblocks_for(nn), dim3(256), 0, st, nn, adj,
                     (const uint8_t *)b.merged, b.work[0], b.ecnt, ctl);
  int rc = read_ctl(ctl, h, st);
  if (rc) return rc;
  if (h->err) return status_from_err(h->err);
  is.on = true;
  is.n_work = h->n_work;
  is.wc = 0;
  is.stamp = 0;
  is.top = slots;
  is.span_live = slots;
  is.n_live = nn;
  return 0;
}

// One incremental round on the worklist (rest_only: the kernels after
// pointer jumping, as in launch_round).
template <int DT>
void incr_round(const Bufs &b, const Adj &adj, int cur, int32_t n, int32_t k,
                int32_t nn, int32_t d, double lambda, int64_t smin,
                const IncrState &is, Ctl *ctl, hipStream_t st,
                bool rest_only) {
  const int32_t nw = is.n_work;
  const int32_t *work = b.work[is.wc];
  int32_t *work_next = b.work[1 - is.wc];
  const int64_t tcap = 2 * edge_bound(n, k);
  const int32_t stamp = is.stamp;
  const int nblk = (int)std::max<int64_t>(1, std::min<int64_t>(4096, (nw + 255) / 256));
  if (!rest_only) {
    hipLaunchKernelGGL(k_round_init, dim3(1), dim3(64), 0, st, ctl);
    hipLaunchKernelGGL(k_incr_round_init, dim3(1), dim3(64), 0, st, ctl);
    prof_begin("select", st);
    const LongWork lw{b.long_rows, b.lbase, b.lnch, b.litem, b.lg,
                      b.lmp,       b.lu,    b.lcnt, b.lcap};
    const dim3 long_grid((unsigned)std::max<int64_t>(
        1, std::min<int64_t>(kLongGrid,
                             (is.span_live / kLongChunk + nw) / 4 + 1)));
    NodeIn s;
    s.size = b.size[cur];
    s.S = b.S[cur];
    s.mu = b.mu;
    s.minpt = b.minpt[cur];
    s.emb = nullptr;
    s.perm = nullptr;
    s.merged = nullptr;  // every worklist node is evaluated
    constexpr int G = kSelLanes;
    hipLaunchKernelGGL((k_select<false, DT, G, true>),
                       xblocks_for((int64_t)nw * G), dim3(256), 0, st, nn,
                       adj, s, d, lambda, smin, b.target, b.deg, lw, work, nw,
                       ctl);
    hipLaunchKernelGGL((k_select_long<false, DT>), long_grid, dim3(256), 0,
                       st, nn, adj, s, d, lambda, smin, lw, ctl);
    hipLaunchKernelGGL(k_select_combine, dim3(64), dim3(256), 0, st, lw,
                       b.target, b.deg, ctl);
    prof_end(st);
    prof_begin("union", st);
    hipLaunchKernelGGL(k_hook_w, blocks_for(nw), dim3(256), 0, st, nw, work,
                       (const int32_t *)b.target, b.parent, nn, ctl);
    hipLaunchKernelGGL(k_jump_w, blocks_for(nw), dim3(256), 0, st, nw, work,
                       b.parent, nn, ctl);
    prof_end(st);
  }
  prof_begin("stats", st);
  hipLaunchKernelGGL(k_incr_merge<DT>, blocks_for(nw), dim3(256), 0, st, nw,
                     work,
                     (const int32_t *)b.parent, b.size[cur], b.S[cur],
                     b.minpt[cur], (const int32_t *)b.wl[cur],
                     (const int32_t *)b.ecnt, b.rep, b.rmark, b.roots, b.rcap,
                     b.cy, b.cY, d, stamp, ctl);
  hipLaunchKernelGGL(k_incr_counts, dim3(1), dim3(64), 0, st, ctl, 0);
  hipLaunchKernelGGL(k_incr_roots, dim3(nblk), dim3(256), 0, st,
                     (const int32_t *)b.roots, (const int32_t *)b.size[cur],
                     (const int64_t *)b.S[cur], b.mu,
                     (const int32_t *)b.wl[cur], (const int32_t *)b.ecnt, b.rcap,
                     b.rcapl, b.rpos, b.cy, b.cY, b.wmark, d, stamp, ctl);
  hipLaunchKernelGGL(k_incr_counts, dim3(1), dim3(64), 0, st, ctl, 1);
  prof_end(st);
  prof_begin("contract", st);
  const dim3 flat(kIncrFlatBlocks);
  // rows to fix: flagged from the members' rows, then fixed in place or
  // listed as owners by a pass over all nodes
  hipLaunchKernelGGL(k_incr_mark, flat, dim3(256), 0, st,
                     (const int32_t *)b.cy, (const int32_t *)b.parent,
                     (const int32_t *)b.rmark, adj, b.fixmark, nn, stamp, ctl);
  hipLaunchKernelGGL(k_incr_fixpass, xblocks_for(nn), dim3(256), 0, st, nn,
                     (const int32_t *)b.fixmark, (const int32_t *)b.parent,
                     (const int32_t *)b.rmark, (const int32_t *)b.ws[cur],
                     (const int32_t *)b.wl[cur], b.tbl[cur], b.ecnt, b.roots,
                     b.rcapl, b.rpos, b.cy, b.cY, stamp, ctl);
  // windows of the owners (roots, long rows to fix), then every
  // contributor's row into its owner's window
  device_scan(ScanArray{b.rcapl, b.rbase, nn, &ctl->n_owners}, nn + 1, b.bsum,
              &ctl->win_total, st);
  hipLaunchKernelGGL(k_incr_clear, flat, dim3(256), 0, st,
                     (const int32_t *)b.roots, (const int32_t *)b.rbase,
                     (const int32_t *)b.rcapl, b.tbl[cur], b.ecnt,
                     (int64_t)is.top, tcap, ctl);
  hipLaunchKernelGGL(k_incr_fill, flat, dim3(256), 0, st,
                     (const int32_t *)b.cy, (const int32_t *)b.cY,
                     (const int32_t *)b.parent, (const int32_t *)b.rmark,
                     (const int32_t *)b.rpos, (const int32_t *)b.rbase,
                     (const int32_t *)b.rcapl, adj, b.tbl[cur], b.ecnt,
                     b.wmark, b.lch_i, b.lch_j, b.lch_cap, (int64_t)is.top,
                     tcap, nn, stamp, ctl);
  hipLaunchKernelGGL(k_incr_fill_long, flat, dim3(256), 0, st,
                     (const int32_t *)b.cy, (const int32_t *)b.cY,
                     (const int32_t *)b.parent, (const int32_t *)b.rmark,
                     (const int32_t *)b.rpos, (const int32_t *)b.rbase,
                     (const int32_t *)b.rcapl, adj, b.tbl[cur], b.ecnt,
                     b.wmark, (const int32_t *)b.lch_i,
                     (const int32_t *)b.lch_j, (int64_t)is.top, nn, stamp,
                     ctl);
  hipLaunchKernelGGL(k_incr_owners, dim3(nblk), dim3(256), 0, st,
                     (const int32_t *)b.roots, (const int32_t *)b.rbase,
                     (const int32_t *)b.rcapl, b.ws[cur], b.wl[cur],
                     (int64_t)is.top, ctl);
  hipLaunchKernelGGL(k_incr_nextwork, xblocks_for(nn), dim3(256), 0, st, nn,
                     (const int32_t *)b.wmark, work_next, stamp, ctl);
  hipLaunchKernelGGL(k_incr_cleanup, blocks_for(nw), dim3(256), 0, st, nw,
                     work, b.target, b.parent, ctl);
  prof_end(st);
}

void incr_round_any(const Bufs &b, const Adj &adj, int cur, int32_t n,
                    int32_t k, int32_t nn, int32_t d, double lambda,
                    int64_t smin, const IncrState &is, Ctl *ctl,
                    hipStream_t st, bool rest_only) {
  switch (d) {
    case 8:
      incr_round<8>(b, adj, cur, n, k, nn, d, lambda, smin, is, ctl, st,
                    rest_only);
      break;
    case 16:
      incr_round<16>(b, adj, cur, n, k, nn, d, lambda, smin, is, ctl, st,
                     rest_only);
      break;
    case 32:
      incr_round<32>(b, adj, cur, n, k, nn, d, lambda, smin, is, ctl, st,
                     rest_only);
      break;
    default:
      incr_round<0>(b, adj, cur, n, k, nn, d, lambda, smin, is, ctl, st,
                    rest_only);
  }
}

// Leaves incremental rounds: the dead nodes' rep chains resolved to their
// roots (doubling passes until one moves nothing), the live nodes numbered
// in id order, their state and rows copied into the other buffers under the
// new ids, and the point map composed.  Updates nn, ed (= the slots of the
// packed table) and cur.
int incr_compact(const Bufs &b, Adj &adj, int &cur, int32_t n, int32_t &nn,
                 int32_t &ed, int32_t d, IncrState &is, Ctl *ctl, Ctl *h,
                 hipStream_t st) {
  int rc;
  int lg = 0;
  while (((int64_t)1 << lg) < (int64_t)nn) ++lg;
  bool done = false;
  for (int bt = 0; bt < (lg + 3) / 4 + 1 && !done; ++bt) {
    hipLaunchKernelGGL(k_jump_state, dim3(1), dim3(64), 0, st, ctl, 0);
    for (int j = 0; j < 4; ++j)
      hipLaunchKernelGGL(k_rep_double, blocks_for(nn), dim3(256), 0, st, nn,
                         b.rep, ctl);
    if ((rc = read_ctl(ctl, h, st))) return rc;
    if (h->err) return status_from_err(h->err);
    done = !h->jump_changed;
  }
  if (!done) {
    set_error("merge aliases did not reach their roots");
    return -5;
  }
  const int nxt = 1 - cur;
  device_scan(ScanLive{b.rep, b.newid, nn}, nn, b.bsum, &ctl->n_live, st);
  NodeIn s;
  s.size = b.size[cur];
  s.S = b.S[cur];
  s.mu = b.mu;
  s.minpt = b.minpt[cur];
  s.emb = nullptr;
  s.perm = nullptr;
  s.merged = nullptr;
  hipLaunchKernelGGL(k_compact_nodes, xblocks_for(nn), dim3(256), 0, st, nn,
                     (const int32_t *)b.rep, (const int32_t *)b.newid, s,
                     b.size[nxt], b.minpt[nxt], b.S[nxt], b.mu, adj, b.capn,
                     (const int32_t *)b.rmark, is.stamp - 1, b.merged, d, ctl);
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  const int32_t nl = h->n_live;
  if (nl < 1 || nl > nn) {
    set_error("live node count out of range (%d of %d)", nl, nn);
    return -5;
  }
  hipLaunchKernelGGL(k_compact_mu, blocks_for((int64_t)nl * d), dim3(256), 0,
                     st, nl, (const int32_t *)b.size[nxt],
                     (const int64_t *)b.S[nxt], b.mu, d, ctl);
  device_scan(ScanArray{b.capn, b.ws[nxt], nl, nullptr}, nl + 1, b.bsum,
              &ctl->slots, st);
  hipLaunchKernelGGL(k_compact_rows, xblocks_for(nn), dim3(256), 0, st, nn,
                     (const int32_t *)b.rep, (const int32_t *)b.newid, adj,
                     (const int32_t *)b.ws[nxt], b.wl[nxt], b.tbl[nxt], ctl);
  hipLaunchKernelGGL(k_compose_rep, xblocks_for(n), dim3(256), 0, st, n, nn,
                     b.M, (const int32_t *)b.rep, (const int32_t *)b.newid,
                     ctl);
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  if (h->slots < 0 || h->slots > is.span_live) {
    set_error("packed table out of range (%d slots)", h->slots);
    return -5;
  }
  nn = nl;
  ed = h->slots;
  cur = nxt;
  adj.ws = b.ws[cur];
  adj.wl = b.wl[cur];
  adj.tbl = b.tbl[cur];
  is.on = false;
  return 0;
}

// The rest of the ladder in the tail kernel, then the labels (and energy)
// of every level it ended.
int run_tail(const LadderArgs &g, const Bufs &b, const float *emb,
             const Adj &adj, int cur, int32_t nn, int32_t ed, int32_t level0,
             int32_t round0, int32_t max_rounds, Ctl *ctl, Ctl *h,
             hipStream_t st) {
  const int32_t n = g.n, d = g.d;
  TailState t;
  for (int j = 0; j < 2; ++j) {
    t.ws[j] = b.ws[j];
    t.wl[j] = b.wl[j];
    t.tbl[j] = b.tbl[j];
  }
  t.size = b.size[cur];
  t.minpt = b.minpt[cur];
  t.S = b.S[cur];
  t.mu = b.mu;
  t.gain = b.tgain;
  t.elist = b.telist;
  t.lvl_map = b.lvl_map;
  t.lvl_minpt = b.lvl_minpt;
  t.lvl_nc = ctl->tail_nc;  // read back with the control block
  t.lvl_rank = b.lvl_rank;
  t.lvl_mu = b.lvl_mu;
  t.lvl_cut2 = reinterpret_cast<long long *>(ctl->tail_cut2);
  t.nn0 = nn;
  // the table goes to the other buffer, its rows packed: the tail's passes
  // run over the entries only
  const int nxt = 1 - cur;
  device_scan(ScanArray{b.wl[cur], b.ws[nxt], nn, nullptr}, nn + 1, b.bsum,
              b.tmp, st);
  hipLaunchKernelGGL(k_repack, blocks_for((int64_t)nn * kWave), dim3(256), 0, st, nn, b.ws[cur],
                     b.wl[cur], b.tbl[cur], b.ws[nxt], b.wl[nxt], b.tbl[nxt]);
  t.tcur0 = nxt;
  t.d = d;
  t.tcap = (int32_t)(2 * edge_bound(n, g.k));
  t.gcap = b.tslots;
  t.n_levels = g.n_levels;
  t.level0 = level0;
  t.round0 = round0;
  t.max_rounds = max_rounds;
  t.want_energy = (g.want_energy && g.energy) ? 1 : 0;
  // EZSP_TAIL_REBUILD=1: the path a full table takes (every live row
  // rebuilt into the other buffer) in every round, for tests
  const char *rb = getenv("EZSP_TAIL_REBUILD");
  t.rebuild_all = (rb && strtol(rb, nullptr, 10) > 0) ? 1 : 0;
  for (int l = 0; l < kTailLevels; ++l) {
    t.lambda[l] = l < g.n_levels ? g.lambdas[l] : 0.0;
    t.smin[l] = (l < g.n_levels && g.min_size) ? g.min_size[l] : 0;
  }
  (void)adj;
  prof_begin("tail", st);
  switch (d) {
    case 8:
      hipLaunchKernelGGL(k_tail<8>, dim3(1), dim3(kTailNT), 0, st, t, ctl);
      break;
    case 16:
      hipLaunchKernelGGL(k_tail<16>, dim3(1), dim3(kTailNT), 0, st, t, ctl);
      break;
    case 32:
      hipLaunchKernelGGL(k_tail<32>, dim3(1), dim3(kTailNT), 0, st, t, ctl);
      break;
    default:
      hipLaunchKernelGGL(k_tail<0>, dim3(1), dim3(kTailNT), 0, st, t, ctl);
  }
  prof_end(st);
  // ranks and labels straight from the snapshots (no host round trip in
  // between); on a device error they are discarded
  hipLaunchKernelGGL(k_tail_rank, dim3((nn + 63) / 64, g.n_levels - level0),
                     dim3(256), 0, st, b.lvl_minpt, t.lvl_nc, nn, level0,
                     b.lvl_rank);
  hipLaunchKernelGGL(k_tail_labels, blocks_for(n), dim3(256), 0, st, n, g.inv,
                     b.M, b.lvl_map, b.lvl_rank, t.lvl_nc, nn, level0,
                     g.n_levels, g.labels, ctl);
  int rc = read_ctl(ctl, h, st);
  if (rc) return rc;
  const int32_t *nc = h->tail_nc;
  const int64_t *cut2 = h->tail_cut2;
  if (h->err & kErrNotConv) {
    set_error("level %d reached max_rounds = %d", h->tail_level, max_rounds);
    return -6;
  }
  if (h->err) return status_from_err(h->err);
  for (int32_t l = level0; l < g.n_levels; ++l) {
    if (nc[l] < 1 || nc[l] > nn) {
      set_error("tail level %d: %d superpoints", l, nc[l]);
      return -5;
    }
    g.n_comp[l] = nc[l];
  }
  if (t.want_energy) {
    for (int32_t l = level0; l < g.n_levels; ++l) {
      // level snapshots have a stride of the tail's start size nn
      const int32_t *map = b.lvl_map + (int64_t)l * nn;
      hipLaunchKernelGGL(k_energy_reset, dim3(1), dim3(64), 0, st, ctl);
      hipLaunchKernelGGL(k_energy_fid<false>, dim3(kEnergyBlocks), dim3(256),
                         0, st, n, d, nc[l], emb, b.M, map, nn,
                         b.lvl_mu + (int64_t)l * nn * d, ctl, b.partial);
      hipLaunchKernelGGL(k_energy_sum, dim3(1), dim3(64), 0, st, b.partial,
                         kEnergyBlocks, ctl);
      if ((rc = read_ctl(ctl, h, st))) return rc;
      if (h->err) return status_from_err(h->err);
      const double cut = (double)(cut2[l] / 2);
      const double reg = g.lambdas[l] * cut;
      g.energy[l] = h->fid_total + reg;
    }
  }
  return 0;
}

}  // namespace

// prepare_graph's linking before the next round, when the last round left
// n_iso nodes with an empty row (listed by k_link_detect): their links, then
// the table rebuilt (compacted, links appended) in the idle buffers and
// copied back.  Updates ed.
int link_round(const LadderArgs &g, const Bufs &b, const Adj &adj, int cur,
               int32_t nn, int32_t n_iso, int32_t &ed, Ctl *ctl, Ctl *h,
               hipStream_t st) {
  int rc;
  if (n_iso > nn) {
    set_error("isolated-node count out of range");
    return -5;
  }
  const int32_t n = g.n, k = g.k;
  const int32_t T = std::min<int32_t>(k, nn - 1);
  const int nxt = 1 - cur;
  const unsigned wave_grid = (unsigned)std::min<int64_t>(16384, nn / 4 + 1);
  prof_begin("link", st);
  hipLaunchKernelGGL(k_link_centroids, blocks_for(3 * (int64_t)nn), dim3(256),
                     0, st, nn, b.lk_sx[cur], b.size[cur], b.lk_cen);
  const size_t lds = (size_t)kLinkNT * T * sizeof(NearKey);
  hipLaunchKernelGGL(k_link_near, dim3((unsigned)std::min<int32_t>(n_iso, 2048)),
                     dim3(kLinkNT), lds, st, nn, b.lk_iso, ctl, b.lk_cen,
                     b.minpt[cur], T, k, b.lk_near, ctl);
  hipLaunchKernelGGL(k_fill_i32, blocks_for(nn + 1), dim3(256), 0, st,
                     b.lk_ext, (int64_t)nn + 1, 0);
  hipLaunchKernelGGL(k_link_count, blocks_for((int64_t)n_iso * T), dim3(256),
                     0, st, ctl, b.lk_iso, b.lk_iso_of, b.lk_near, T, k,
                     b.lk_ext, b.lk_keep, ctl);
  hipLaunchKernelGGL(k_link_rowcount, dim3(wave_grid), dim3(256), 0, st, nn,
                     adj, b.lk_cnt);
  device_scan(ScanLinkWin{b.lk_cnt, b.lk_ext, b.ws[nxt], nn}, nn + 1, b.bsum,
              &ctl->slots, st);
  hipLaunchKernelGGL(k_link_copy, dim3(wave_grid), dim3(256), 0, st, nn, adj,
                     b.lk_cnt, b.lk_ext, b.ws[nxt], b.wl[nxt], b.tbl[nxt],
                     b.lk_fill);
  hipLaunchKernelGGL(k_link_append, blocks_for((int64_t)n_iso * T), dim3(256),
                     0, st, ctl, b.lk_iso, b.lk_near, T, k, b.lk_keep,
                     b.ws[nxt], b.wl[nxt], b.tbl[nxt], b.lk_fill, ctl);
  prof_end(st);
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  const int64_t total = h->slots;
  if (total < 0 || total > (int64_t)ed + 2 * (int64_t)n_iso * T ||
      total > 2 * edge_bound(n, k)) {
    set_error("linked table size out of range (%lld)", (long long)total);
    return -5;
  }
  // back into the current buffers (the idle ones take the next contraction)
  rc = check_hip(hipMemcpyAsync(b.tbl[cur], b.tbl[nxt], sizeof(uint64_t) * total,
                                hipMemcpyDeviceToDevice, st), "link copy");
  if (!rc)
    rc = check_hip(hipMemcpyAsync(b.ws[cur], b.ws[nxt], sizeof(int32_t) * (nn + 1),
                                  hipMemcpyDeviceToDevice, st), "link copy");
  if (!rc)
    rc = check_hip(hipMemcpyAsync(b.wl[cur], b.wl[nxt], sizeof(int32_t) * (nn + 1),
                                  hipMemcpyDeviceToDevice, st), "link copy");
  if (rc) return rc;
  ed = (int32_t)total;
  prof_bytes("link", 48.0 * nn + 16.0 * total);
  return 0;
}

void ladder_reserve(Arena &a, int32_t n, int32_t d, int32_t k, bool link) {
  Bufs b;
  carve(a, n, d, k, link, &b);
}

float *ladder_emb_slot(Arena a, int32_t n, int32_t d, int32_t k, bool link) {
  Bufs b;
  carve(a, n, d, k, link, &b);  // on a copy of the arena
  return b.emb_int;
}

int ladder_run(const LadderArgs &g, Ctl *ctl, Arena &a, hipStream_t st) {
  Bufs b;
  carve(a, g.n, g.d, g.k, g.link, &b);
  b.pts = g.pts;
  if (g.link && !g.pts) {
    set_error("linking isolated nodes needs the positions");
    return -1;
  }
  Ctl *h = pinned_ctl();
  if (!h) {
    set_error("hipHostMalloc of the control block failed");
    return -5;
  }
  const int32_t n = g.n, d = g.d, k = g.k;
  int rc;

  // embeddings in internal order, fixed-point shift (Step 0)
  // (always a copy in the workspace: aligned rows for vector loads)
  const float *emb = b.emb_int;
  // rows of 4k floats at a 16-byte aligned base: vector gather with the
  // max |e| reduction fused in
  const bool fused = g.perm && d % 4 == 0 &&
                     (reinterpret_cast<uintptr_t>(g.emb) & 15) == 0;
  if (g.emb_ready) {
    // copied by the kNN kernel, max |e| included
  } else if (g.perm) {
    if (fused) {
      const int64_t t4 = (int64_t)n * (d / 4);
      const unsigned grid =
          (unsigned)std::min<int64_t>((t4 + 255) / 256, 8192);
      hipLaunchKernelGGL(k_gather_rows4, dim3(grid), dim3(256), 0, st,
                         reinterpret_cast<const float4 *>(g.emb), g.perm, n,
                         d / 4, reinterpret_cast<float4 *>(b.emb_int), ctl);
    } else {
      hipLaunchKernelGGL(k_gather_rows, blocks_for((int64_t)n * d), dim3(256),
                         0, st, g.emb, g.perm, n, d, b.emb_int);
    }
  } else {
    rc = check_hip(hipMemcpyAsync(b.emb_int, g.emb, sizeof(float) * n * d,
                                  hipMemcpyDeviceToDevice, st),
                   "hipMemcpyAsync(emb)");
    if (rc) return rc;
  }
  if (!fused && !g.emb_ready)
    hipLaunchKernelGGL(k_maxabs, dim3(2048), dim3(256), 0, st, emb,
                       (int64_t)n * d, ctl);
  hipLaunchKernelGGL(k_fixshift, dim3(1), dim3(64), 0, st, ctl, n);
  if (g.link) {
    hipLaunchKernelGGL(k_link_maxabs, dim3(1024), dim3(256), 0, st, g.pts, n,
                       ctl);
    hipLaunchKernelGGL(k_link_shift, dim3(1), dim3(64), 0, st, ctl, n);
  }

  // first-round graph (Step 0: the superpoint adjacency is the kNN graph)
  prof_begin("graph_build", st);
  const int32_t *nbr = g.nbr;
  if (g.check_nbr) {
    hipLaunchKernelGGL(k_sanitize, blocks_for(n), dim3(256), 0, st, g.nbr, n,
                       k, b.nbr_clean, ctl);
    nbr = b.nbr_clean;
  }
  hipLaunchKernelGGL(k_fill_i32, blocks_for(n), dim3(256), 0, st, b.rev,
                     (int64_t)n, 0);
  hipLaunchKernelGGL(k_fill_i32, blocks_for(n), dim3(256), 0, st, b.cursor,
                     (int64_t)n, 0);
  const bool blk = g.kth && g.pts;  // block-local count and fill
  const dim3 rev_grid(xcd_grid(((int64_t)n + kRevR - 1) / kRevR));
  if (blk)
    hipLaunchKernelGGL(k_rev_count_blk, rev_grid, dim3(kRevNT), 0, st, nbr, n, k,
                       g.pts, g.kth, b.rev, b.nmask, ctl);
  else
    hipLaunchKernelGGL(k_rev_count, xblocks_for(n), dim3(256), 0, st, nbr, n,
                       k, b.rev, b.nmask, ctl);
  device_scan(ScanArray{b.rev, b.rrp, n, nullptr}, n + 1, b.bsum, &ctl->e_rev,
              st);
  if (blk)
    hipLaunchKernelGGL(k_rev_fill_blk, rev_grid, dim3(kRevNT), 0, st, nbr, n, k,
                       b.nmask, b.rrp, b.cursor, b.rcol, ctl);
  else
    hipLaunchKernelGGL(k_rev_fill, xblocks_for(n), dim3(256), 0, st, nbr, n, k,
                       b.nmask, b.rrp, b.cursor, b.rcol, ctl);
  prof_end(st);
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  int64_t ed64 = (int64_t)h->e_fwd + h->e_rev;
  if (ed64 > edge_bound(n, k) || h->e_rev < 0 || h->e_fwd < 0) {
    set_error("graph larger than its bound");
    return -5;
  }
  int32_t ed = (int32_t)ed64;  // directed entries of the current graph
  const int32_t ed0 = ed;
  prof_bytes("graph_build", 4.0 * n * k + 12.0 * (ed / 2));

  Adj adj;
  adj.nbr = nbr;
  adj.k = k;
  adj.kp = pad4(k);
  adj.rrp = b.rrp;
  adj.rcol = b.rcol;
  adj.n_rev = h->e_rev;
  adj.ws = nullptr;
  adj.wl = nullptr;
  adj.tbl = nullptr;

  const Adj adj0 = adj;  // the input graph, for the cut term with links
  int cur = 0;
  bool first = true;
  int32_t nn = n;
  const int32_t max_rounds = g.max_rounds > 0 ? g.max_rounds : 256;
  int32_t tail_level = -1, tail_round = 0;
  int64_t slots = 0;  // slots of the current table (its windows' total)
  // EZSP_TAIL_NODES (at most kTailNodes; 0 = never) moves the switch to the
  // tail kernel, so that both paths can be exercised on small inputs
  int32_t tail_nodes = kTailStart;
  if (const char *e = getenv("EZSP_TAIL_NODES")) {
    const long v = strtol(e, nullptr, 10);
    tail_nodes = (int32_t)std::max<long>(0, std::min<long>(v, kTailNodes));
  }
  if (g.link) tail_nodes = 0;  // the tail kernel does not link
  bool relinked = false;
  int32_t mn = 0;  // nodes of the node map b.Mn (0: b.M is up to date)
  // incremental rounds (stable ids within a level) are opt-in:
  // EZSP_INCREMENTAL=1 switches graphs of kIncrMinNodes nodes and more,
  // larger values set the smallest graph that switches (so that tests reach
  // these rounds on small inputs); unset or 0 keeps every round on the
  // renumbering path, which measured faster on the aerial tile
  IncrState is;
  bool incr_allowed = false;
  int32_t incr_min = kIncrMinNodes;
  if (const char *e = getenv("EZSP_INCREMENTAL")) {
    const long v = strtol(e, nullptr, 10);
    incr_allowed = v > 0 && !g.link;
    if (v > 1) incr_min = (int32_t)std::min<long>(v, INT32_MAX);
  }
  // EZSP_INCR_COMPACT_EVERY=r renumbers after every r incremental rounds
  // (the path a filling table takes), for tests
  int32_t compact_every = 0;
  if (const char *e = getenv("EZSP_INCR_COMPACT_EVERY"))
    compact_every = (int32_t)std::max<long>(0, strtol(e, nullptr, 10));
  const int64_t tcap = 2 * edge_bound(n, k);
  for (int32_t l = 0; l < g.n_levels; ++l) {
    const double lambda = g.lambdas[l];
    const int64_t smin = g.min_size ? g.min_size[l] : 0;
    for (int32_t round = 0;; ++round) {
      if (is.on && (is.n_live <= tail_nodes ||
                    is.top + 2 * is.span_live > tcap ||
                    (compact_every > 0 && is.stamp >= compact_every))) {
        // back to renumbered ids: for the tail, or for table room
        if ((rc = incr_compact(b, adj, cur, n, nn, ed, d, is, ctl, h, st)))
          return rc;
        slots = ed;
      }
      if (!is.on) {
        if (ed == 0) break;  // no edge left: nothing can merge
        if (!first && nn <= tail_nodes && ed <= kTailEdges &&
            slots <= b.tslots) {
          tail_level = l;  // the rest runs in the tail kernel
          tail_round = round;
          break;
        }
      }
      if (round >= max_rounds) {
        set_error("level %d reached max_rounds = %d", l, max_rounds);
        return -6;
      }
      if (is.on) {
        incr_round_any(b, adj, cur, n, k, nn, d, lambda, smin, is, ctl, st,
                       false);
        if ((rc = read_ctl(ctl, h, st))) return rc;
        if (h->err) return status_from_err(h->err);
        if (h->any_choice < 0) {
          if ((rc = finish_jump(b, nn, ctl, h, st))) return rc;
          incr_round_any(b, adj, cur, n, k, nn, d, lambda, smin, is, ctl, st,
                         true);
          if ((rc = read_ctl(ctl, h, st))) return rc;
          if (h->err) return status_from_err(h->err);
        }
        if (prof_on()) {
          // algorithmic bytes, from the round's counts: the worklist's rows
          // (at the mean row span) and node statistics, the members' sums,
          // the rebuilt windows written and read back
          const double S1 = 8.0 * d + 8.0;
          const double span = is.n_live ? (double)is.span_live / is.n_live : 0;
          prof_bytes("select", is.n_work * (8.0 * span + S1 + 4.0));
          if (h->any_choice) {
            prof_bytes("union", 8.0 * is.n_work);
            prof_bytes("stats", 2.0 * S1 * h->n_dead + S1 * h->n_roots);
            prof_bytes("contract", 8.0 * span * (h->n_dead + h->n_roots) +
                                       16.0 * h->win_total);
          }
        }
        if (!h->any_choice) break;  // Step 1: no candidate merge
        if (h->n_dead < 1 || h->n_dead >= is.n_live || h->n_work < 0 ||
            h->n_work > nn || h->win_total < 0 || h->span_live < 0) {
          set_error("incremental round sizes out of range (%d merged, %d "
                    "listed)", h->n_dead, h->n_work);
          return -5;
        }
        is.n_live -= h->n_dead;
        is.top += h->win_total;
        is.span_live = h->span_live;
        is.n_work = h->n_work;
        is.wc = 1 - is.wc;
        ++is.stamp;
        if (is.n_live == 1) break;  // a single component is left
        continue;
      }
      NodeIn s;
      s.emb = emb;
      s.perm = g.perm;
      // merged flags hold from the second round of a level on, when no
      // link has changed the graph since
      s.merged = (first || round == 0 || relinked) ? nullptr : b.merged;
      relinked = false;
      if (first) {
        s.size = nullptr;
        s.S = nullptr;
        s.mu = nullptr;
        s.minpt = nullptr;
        round_d<true>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin, ctl, st,
                      mn);
      } else {
        s.size = b.size[cur];
        s.S = b.S[cur];
        s.mu = b.mu;
        s.minpt = b.minpt[cur];
        round_d<false>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin, ctl,
                       st, mn);
      }
      if ((rc = read_ctl(ctl, h, st))) return rc;
      if (h->err) return status_from_err(h->err);
      if (h->any_choice < 0) {
        // a merge chain deeper than a jumping walk: complete the forest,
        // then the rest of the round
        if ((rc = finish_jump(b, nn, ctl, h, st))) return rc;
        if (first)
          round_d<true>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin, ctl,
                        st, mn, true);
        else
          round_d<false>(b, adj, cur, n, k, nn, ed, d, s, lambda, smin, ctl,
                         st, mn, true);
        if ((rc = read_ctl(ctl, h, st))) return rc;
        if (h->err) return status_from_err(h->err);
      }
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
          prof_bytes("compose", 8.0 * (first ? n : (mn ? mn : nn)));
        }
      }
      if (!h->any_choice) break;  // Step 1: no candidate merge
      if (h->n_next < 1 || h->n_next >= nn || h->e_next < 0 ||
          h->e_next > ed || h->slots < ed || h->slots > 2 * (int64_t)ed) {
        set_error("round sizes out of range (%d nodes, %d edges, %d slots)",
                  h->n_next, h->e_next, h->slots);
        return -5;
      }
      const int32_t nn_before = nn;
      if (!first && mn == 0) mn = nn;  // the node map now spans this graph
      cur = 1 - cur;
      first = false;
      slots = h->slots;
      nn = h->n_next;
      ed = h->e_next;
      adj.ws = b.ws[cur];
      adj.wl = b.wl[cur];
      adj.tbl = b.tbl[cur];
      if (nn == 1) break;  // a single component is left
      if (incr_allowed && nn >= incr_min &&
          (double)nn > kIncrKeep * (double)nn_before) {
        // few nodes merged: the next rounds keep their ids
        sync_map(b, n, mn, ctl, st);
        if ((rc = incr_enter(b, adj, nn, slots, is, ctl, h, st))) return rc;
      }
      if (g.link && h->n_iso > 0) {  // prepare_graph of the next round
        if ((rc = link_round(g, b, adj, cur, nn, h->n_iso, ed, ctl, h, st)))
          return rc;
        slots = ed;
        relinked = true;
      }
    }

    if (is.on) {  // the level's nodes under consecutive ids again
      if ((rc = incr_compact(b, adj, cur, n, nn, ed, d, is, ctl, h, st)))
        return rc;
      slots = ed;
    }
    sync_map(b, n, mn, ctl, st);  // the point map, for the outputs and tail
    if (tail_level >= 0) break;
    // level output
    int32_t *out = g.labels + (int64_t)l * n;
    if (first) {
      hipLaunchKernelGGL(k_iota, blocks_for(n), dim3(256), 0, st, n, out);
    } else {
      hipLaunchKernelGGL(k_fill_i32, blocks_for(n), dim3(256), 0, st, b.mark,
                         (int64_t)n, 0);
      hipLaunchKernelGGL(k_mark, blocks_for(nn), dim3(256), 0, st, nn,
                         b.minpt[cur], b.mark, n, ctl);
      device_scan(ScanArray{b.mark, b.lrank, n, nullptr}, n, b.bsum, b.tmp,
                  st);
      hipLaunchKernelGGL(k_labels, blocks_for(n), dim3(256), 0, st, n, nn,
                         g.inv, b.M, (const int32_t *)nullptr, 0,
                         b.minpt[cur], b.lrank, out, ctl);
    }
    g.n_comp[l] = nn;
    if (g.want_energy && g.energy) {
      hipLaunchKernelGGL(k_energy_reset, dim3(1), dim3(64), 0, st, ctl);
      if (first)
        hipLaunchKernelGGL(k_energy_fid<true>, dim3(kEnergyBlocks), dim3(256),
                           0, st, n, d, nn, emb, b.M, (const int32_t *)nullptr,
                           0, b.mu, ctl, b.partial);
      else
        hipLaunchKernelGGL(k_energy_fid<false>, dim3(kEnergyBlocks),
                           dim3(256), 0, st, n, d, nn, emb, b.M,
                           (const int32_t *)nullptr, 0, b.mu, ctl, b.partial);
      hipLaunchKernelGGL(k_energy_sum, dim3(1), dim3(64), 0, st, b.partial,
                         kEnergyBlocks, ctl);
      if (!first && g.link)  // the cut of the input graph, links aside
        hipLaunchKernelGGL(k_cut_e0, dim3(1024), dim3(256), 0, st, n, adj0,
                           b.M, ctl);
      else if (!first)
        hipLaunchKernelGGL(k_weight_sum, dim3(256), dim3(256), 0, st, nn, adj,
                           ctl);
      if ((rc = read_ctl(ctl, h, st))) return rc;
      if (h->err) return status_from_err(h->err);
      const int64_t cut2 = first ? (int64_t)ed0 : h->cut_w2;
      const double cut = (double)(cut2 / 2);
      const double reg = lambda * cut;
      g.energy[l] = h->fid_total + reg;
    }
  }
  if (tail_level >= 0) {
    // the tail's own readback comes after its last kernel
    return run_tail(g, b, emb, adj, cur, nn, ed, tail_level, tail_round,
                    max_rounds, ctl, h, st);
  }
  if ((rc = read_ctl(ctl, h, st))) return rc;
  if (h->err) return status_from_err(h->err);
  return 0;
}

}  // namespace ezsp
