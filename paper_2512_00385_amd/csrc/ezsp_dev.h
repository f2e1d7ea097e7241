// ezsp_dev.h -- device-side building blocks shared by the HIP kernels of the
// EZ-SP partition library (gfx950, wave64): the device control block, wave
// and block scans, a device-wide scan driven by functors, and an LSD radix
// sort of 64-bit keys with 32-bit payloads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ezsp {

constexpr int kWave = 64;

// Error bits raised on the device and read back by the host.
enum : uint32_t {
  kErrNonFinite = 1u,  // NaN / Inf in xyz or emb
  kErrRange = 2u,      // fixed-point shift below 16
  kErrInternal = 4u,   // an index or capacity check failed
  kErrBadIndex = 8u,   // caller data out of range (neighbour id, label)
  kErrJump = 16u,      // pointer jumping hit its iteration cap
  kErrNotConv = 32u,   // a level reached max_rounds inside the tail kernel
};

// Small block of device scalars, one per call, at the start of the
// workspace.  The host reads it back once per merge round.
// Counters that many blocks add to at once are spread over kStripes cache
// lines: device-scope atomics on one address are serialised at the memory
// side.  Only the host reads them (read_ctl folds the stripes).
constexpr int kStripes = 32;
struct alignas(128) Stripe {
  int32_t v;
  int32_t pad[31];
};

struct Ctl {
  uint32_t err;
  int32_t F;            // fixed-point shift of the embeddings
  int32_t any_choice;   // some node kept a merge edge this round; -1 when
                        // one did but pointer jumping stopped at its walk
                        // cap (the round's later kernels then wait)
  int32_t jump_changed; // a pointer-doubling pass moved some parent
  // incremental rounds (stable node ids within a level)
  int32_t n_roots;      // components formed by a merge this round
  int32_t n_fix;        // unmerged rows that listed a merged node
  int32_t n_work;       // nodes of the next round's worklist
  int32_t n_dead;       // nodes merged into another this round
  int32_t n_live;       // live nodes after compaction
  int32_t win_total;    // slots of this round's rebuilt windows
  int32_t n_members;    // contributors that are members of a root
  int32_t n_contrib;    // rows that go into rebuilt windows
  int32_t n_owners;     // rows rebuilt into new windows
  int32_t chunk_total;  // wavefront chunks of the contributors' rows
  int32_t n_lfill;      // chunks of the long contributor rows
  long long span_live;  // slots of the live rows (their windows' lengths)
  long long work_slots; // slots of the worklist rows selection scanned
  int32_t n_next;       // components after this round
  int32_t e_next;       // directed edges after this round (host: folded)
  int32_t slots;        // adjacency-table slots of the next round
  uint32_t maxabs_bits; // max |e| as fp32 bits (monotone for >= 0)
  int32_t n_long;       // rows longer than a short-row group takes
  int32_t n_lchunk;     // entry chunks of those rows
  int32_t bbox_enc[6];  // min xyz, max xyz in order-preserving int form
  int32_t n_big;        // components that go to the block-per-component path
  int32_t e_rev;        // reverse-only entries of the first-round graph
  int32_t e_fwd;        // valid forward entries of the first-round graph
                        // (host: folded)
  int32_t n_cbig;       // components whose table window exceeds one chunk
  int32_t n_tiles;      // member tiles of those components
  int32_t tail_level;   // level that reached max_rounds in the tail kernel
  int64_t cut_w2;       // 2 * cut weight (directed sum) of the current graph
  double fid_total;     // fidelity term of the energy
  Stripe e_next_s[kStripes];  // device side of e_next
  Stripe e_fwd_s[kStripes];   // device side of e_fwd
  Stripe maxabs_s[kStripes];  // max |e| bits from the fused gather
  Stripe bbox_s[6][kStripes]; // bbox_enc's min xyz, max xyz per stripe
                              // (folded into bbox_enc by k_bbox_fold)
  int32_t tail_nc[16];        // superpoints of every level the tail ended
  int64_t tail_cut2[16];      // ... and 2 x their cut weight
  // linking of isolated nodes
  uint32_t maxabs_x_bits;     // max |coordinate| as fp32 bits
  int32_t Fx;                 // fixed-point shift of the positions
  int32_t n_iso;              // nodes with an empty row this round
  int32_t n_link;             // links kept this round
  // results of the grid-subsampling, edge-loss and purity entry points
  int32_t n_out;              // points kept by the grid subsampling
  int32_t sel_mode;           // intra sample: 0 none, 1 all, 2 by threshold
  uint64_t sel_prefix;        // radix select: key bits fixed so far
  uint64_t sel_mask;          // ... and which bits those are
  int64_t sel_rank;           // rank still wanted below the prefix
  unsigned long long le_edges, le_intra, le_keep;
  double le_loss;             // Eq. loss over the sample
  double pu_miou, pu_purity;
  int64_t pu_present;
  uint32_t seq;               // host copy only: export number, written last
};

__device__ __forceinline__ void stripe_add(Stripe *s, int32_t v) {
  atomicAdd(&s[blockIdx.x % kStripes].v, v);
}
__device__ __forceinline__ void stripe_max(Stripe *s, int32_t v) {
  atomicMax(&s[blockIdx.x % kStripes].v, v);
}
__device__ __forceinline__ void stripe_zero(Stripe *s) {
  for (int i = threadIdx.x; i < kStripes; i += blockDim.x) s[i].v = 0;
}

// --- order-preserving float <-> int (for atomic min/max on floats) --------
__device__ __forceinline__ int32_t f2ord(float f) {
  int32_t i = __float_as_int(f);
  return i >= 0 ? i : (i ^ 0x7fffffff);
}
__host__ __device__ __forceinline__ float ord2f(int32_t i) {
  int32_t b = i >= 0 ? i : (i ^ 0x7fffffff);
  union { int32_t i; float f; } u;
  u.i = b;
  return u.f;
}

// F = min(40, 61 - ceil(log2 n) - max(0, ceil(log2 A))), A = max |value|.
__device__ __forceinline__ int fixshift_rule(float A, int32_t n) {
  int cn = 0;
  while (((int64_t)1 << cn) < (int64_t)n) ++cn;
  int ca = 0;
  if (A > 0.0f) {
    int e;
    const float m = frexpf(A, &e);  // A = m * 2^e, m in [0.5, 1)
    ca = (m == 0.5f) ? e - 1 : e;
    if (ca < 0) ca = 0;
  }
  const int F = 61 - cn - ca;
  return F > 40 ? 40 : F;
}

// The kernels after Step 3 run only when some node chose and every parent
// reached its root.
__device__ __forceinline__ bool round_live(const Ctl *ctl) {
  return ctl->any_choice > 0;
}

__device__ __forceinline__ void raise_err(Ctl *ctl, uint32_t bits) {
  atomicOr(&ctl->err, bits);
}

// --- wave / block scans (wave64) ------------------------------------------
template <class T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T t = __shfl_up(v, off, kWave);
    if (lane >= off) v += t;
  }
  return v;
}

template <class T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Exclusive scan over a block of NT threads; *total gets the block sum.
// `wsum` is LDS scratch of NT/64 elements.  Contains barriers.
template <int NT, class T>
__device__ __forceinline__ T block_excl_scan(T v, T *wsum, T *total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  T inc = wave_incl_scan(v);
  if (lane == kWave - 1) wsum[wid] = inc;
  __syncthreads();
  T off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / kWave; ++w) {
    T s = wsum[w];
    off += (w < wid) ? s : T(0);
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return off + inc - v;
}

// --- device-wide exclusive scan of int32 values produced by a functor -----
// Op provides:  __device__ int32_t value(int32_t i) const;
//               __device__ void emit(int32_t i, int32_t excl, int32_t v) const;
// The scan runs over [0, n_bound); op.value must return 0 past the real end.
// Four items a thread: more tiles, each with a shorter chain, measured
// about 70 us faster per driving-tile step than eight or sixteen (a step
// runs some forty scans).
constexpr int kScanNT = 256;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanNT * kScanItems;

template <class Op>
__global__ __launch_bounds__(kScanNT) void k_scan_reduce(Op op, int32_t n,
                                                         int32_t *bsum) {
  __shared__ int32_t wsum[kScanNT / kWave];
  const int32_t base = blockIdx.x * kScanTile + threadIdx.x * kScanItems;
  int32_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    int32_t i = base + j;
    if (i < n) s += op.value(i);
  }
  int32_t tot;
  block_excl_scan<kScanNT>(s, wsum, &tot);
  if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

// One block: exclusive scan of bsum[0, nb) in place, total to *total.
__global__ __launch_bounds__(1024) void k_scan_bsums(int32_t *bsum, int32_t nb,
                                                     int32_t *total);

template <class Op>
__global__ __launch_bounds__(kScanNT) void k_scan_apply(Op op, int32_t n,
                                                        const int32_t *bsum) {
  __shared__ int32_t wsum[kScanNT / kWave];
  const int32_t base = blockIdx.x * kScanTile + threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    int32_t i = base + j;
    v[j] = (i < n) ? op.value(i) : 0;
    s += v[j];
  }
  int32_t tot;
  int32_t run = block_excl_scan<kScanNT>(s, wsum, &tot) + bsum[blockIdx.x];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    int32_t i = base + j;
    if (i < n) op.emit(i, run, v[j]);
    run += v[j];
  }
}

// Apply pass that finds its own tile offset: the sum of the raw tile sums
// before it (a few thousand at most, read from L2), so no separate pass
// scans the tile sums.  Tile 0 also writes the total.
template <class Op>
__global__ __launch_bounds__(kScanNT) void k_scan_apply_sum(
    Op op, int32_t n, const int32_t *bsum, int32_t nb, int32_t *total) {
  __shared__ int32_t wsum[kScanNT / kWave];
  const int32_t b = blockIdx.x;
  const int32_t upto = b == 0 ? nb : b;
  int32_t pre = 0, all = 0;
  for (int32_t t = threadIdx.x; t < upto; t += kScanNT) {
    const int32_t x = bsum[t];
    all += x;
    pre += t < b ? x : 0;
  }
  int32_t pre_tot, all_tot;
  block_excl_scan<kScanNT>(pre, wsum, &pre_tot);
  block_excl_scan<kScanNT>(all, wsum, &all_tot);
  if (b == 0 && threadIdx.x == 0) *total = all_tot;
  const int32_t base = b * kScanTile + threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    int32_t i = base + j;
    v[j] = (i < n) ? op.value(i) : 0;
    s += v[j];
  }
  int32_t tot;
  int32_t run = block_excl_scan<kScanNT>(s, wsum, &tot) + pre_tot;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    int32_t i = base + j;
    if (i < n) op.emit(i, run, v[j]);
    run += v[j];
  }
}

inline int32_t scan_blocks(int64_t n) {
  return (int32_t)((n + kScanTile - 1) / kScanTile);
}

// Small scans in one launch: one block of 1024 threads, 4 items each (a
// single block is a long chain: larger scans are faster in two launches).
constexpr int kOneNT = 1024;
constexpr int kOneItems = 4;
constexpr int kOneMax = kOneNT * kOneItems;

template <class Op>
__global__ __launch_bounds__(kOneNT) void k_scan_one(Op op, int32_t n,
                                                     int32_t *total) {
  __shared__ int32_t wsum[kOneNT / kWave];
  const int32_t base = threadIdx.x * kOneItems;
  int32_t v[kOneItems];
  int32_t s = 0;
#pragma unroll
  for (int j = 0; j < kOneItems; ++j) {
    const int32_t i = base + j;
    v[j] = (i < n) ? op.value(i) : 0;
    s += v[j];
  }
  int32_t tot;
  int32_t run = block_excl_scan<kOneNT>(s, wsum, &tot);
#pragma unroll
  for (int j = 0; j < kOneItems; ++j) {
    const int32_t i = base + j;
    if (i < n) op.emit(i, run, v[j]);
    run += v[j];
  }
  if (threadIdx.x == 0) *total = tot;
}

// Exclusive scan; `bsum` needs scan_blocks(n) ints; `total` (device) gets the
// sum.  n may be 0.
template <class Op>
inline void device_scan(const Op &op, int32_t n, int32_t *bsum, int32_t *total,
                        hipStream_t st) {
  if (n <= kOneMax) {
    hipLaunchKernelGGL(k_scan_one<Op>, dim3(1), dim3(kOneNT), 0, st, op, n,
                       total);
    return;
  }
  int32_t nb = scan_blocks(n);
  if (nb == 0) {
    hipLaunchKernelGGL(k_scan_bsums, dim3(1), dim3(1024), 0, st, bsum, 0,
                       total);
    return;
  }
  hipLaunchKernelGGL(k_scan_reduce<Op>, dim3(nb), dim3(kScanNT), 0, st, op, n,
                     bsum);
  hipLaunchKernelGGL(k_scan_apply_sum<Op>, dim3(nb), dim3(kScanNT), 0, st, op,
                     n, bsum, nb, total);
}

// Common functor: exclusive scan of an int32 array into another.  The real
// length is `n` or, when `n_dev` is set, the device value *n_dev; items past
// it count as 0, and out[len] receives the total, so a scan over len+1
// items produces a CSR offset array.
struct ScanArray {
  const int32_t *in;
  int32_t *out;
  int32_t n;
  const int32_t *n_dev;
  __device__ int32_t len() const { return n_dev ? *n_dev : n; }
  __device__ int32_t value(int32_t i) const {
    return (i < len()) ? in[i] : 0;
  }
  __device__ void emit(int32_t i, int32_t excl, int32_t) const {
    if (i <= len()) out[i] = excl;
  }
};

// --- LSD radix sort of (uint64 key, uint32 value) -------------------------
constexpr int kSortNT = 256;
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortNT * kSortItems;
constexpr int kSortBins = 256;

inline int32_t sort_blocks(int64_t n) {
  return (int32_t)((n + kSortTile - 1) / kSortTile);
}

}  // namespace ezsp
