// ezsp_internal.h -- host-side internal interface between the C ABI layer
// and the kernel launchers of the EZ-SP partition library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ezsp_dev.h"

namespace ezsp {

// XCD-aware block order.  Workgroups are dispatched round-robin over the 8
// XCDs (each with its own L2), so physical block b runs on XCD b % 8.  The
// grid is rounded up to a multiple of 8 and block b takes logical block
// (b % 8) * (grid / 8) + b / 8: each XCD works on one contiguous range of
// logical blocks, and neighbouring data stays in one L2.
constexpr int kXcd = 8;
inline unsigned xcd_grid(int64_t logical_blocks) {
  int64_t g = (logical_blocks + kXcd - 1) / kXcd * kXcd;
  return (unsigned)(g < kXcd ? kXcd : g);
}
__device__ __forceinline__ int32_t xcd_block() {
  const int32_t per = (int32_t)(gridDim.x / kXcd);
  return (int32_t)(blockIdx.x % kXcd) * per + (int32_t)(blockIdx.x / kXcd);
}
// Global thread index under the XCD-aware block order.
__device__ __forceinline__ int32_t xcd_tid() {
  return xcd_block() * (int32_t)blockDim.x + (int32_t)threadIdx.x;
}
// Item of this thread when only m <= gridDim.x * blockDim.x items are live
// (m known on the device only, grid sized by an upper bound): XCD x takes
// the x-th contiguous eighth of [0, m), so every XCD gets work however small
// m is.  Needs gridDim.x % kXcd == 0 (xcd_grid); then each XCD has
// (gridDim.x / kXcd) * blockDim.x >= ceil(m / kXcd) threads.  Returns false
// for threads without an item.
__device__ __forceinline__ bool xcd_item(int32_t m, int32_t &c) {
  const int32_t per = (m + kXcd - 1) / kXcd;
  const int32_t j =
      (int32_t)(blockIdx.x / kXcd) * (int32_t)blockDim.x + (int32_t)threadIdx.x;
  c = (int32_t)(blockIdx.x % kXcd) * per + j;
  return j < per && c < m;
}

// Row stride of the internal neighbour tables: k rounded up to a multiple
// of 4 (16-byte rows for vector loads), padded with -1.
__host__ __device__ __forceinline__ int32_t pad4(int32_t k) {
  return (k + 3) & ~3;
}

// Bump allocator over the caller's workspace.  With base == nullptr it only
// measures: every take() returns nullptr and `off` ends at the bytes needed.
struct Arena {
  char *base = nullptr;
  size_t cap = 0;
  size_t off = 0;
  template <class T>
  T *take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// Implicit 8-ary tree of boxes over the Morton-ordered points: level 0 holds
// one box per bucket of kBucket consecutive points, level l+1 one box per 8
// boxes of level l, up to a single root at level `top`.  A bucket is also
// the query group of the kNN kernel: 16 lanes, one DPP row.
constexpr int kBucket = 16;
// n rounded up to whole buckets, and the index carried by padding points.
__host__ __device__ __forceinline__ int32_t pad_bucket(int32_t n) {
  return (n + kBucket - 1) / kBucket * kBucket;
}
constexpr int32_t kPadIndex = 0x7fffffff;
constexpr int kFan = 8;
constexpr int kMaxTreeLevels = 16;
struct Tree {
  int32_t off[kMaxTreeLevels];
  int32_t cnt[kMaxTreeLevels];
  int32_t top;
  int32_t total;
};
Tree make_tree(int32_t n);

// Radix sort of (key, value) pairs on bits [0, nbits).  Returns true when
// the sorted result ended in the *_alt buffers.
bool radix_sort_pairs(uint64_t *keys, uint32_t *vals, uint64_t *keys_alt,
                      uint32_t *vals_alt, int32_t n, int nbits,
                      int32_t *hist, int32_t *bsum, int32_t *total, Ctl *ctl,
                      hipStream_t st);
size_t radix_hist_ints(int32_t n);
// Radix sort of 64-bit keys alone on bits [shift0, shift0 + nbits) (stable,
// so bits below shift0 keep their input order within equal digits).
// Returns true when the sorted result ended in keys_alt.
bool radix_sort_keys(uint64_t *keys, uint64_t *keys_alt, int32_t n,
                     int shift0, int nbits, int32_t *hist, int32_t *bsum,
                     int32_t *total, Ctl *ctl, hipStream_t st);

// kNN: Morton sort, box tree, exact query.  Produces the internal
// (Morton-order) neighbour table nbr_int (n rows of pad4(k), -1 padded) and
// the maps
// perm (internal -> original) and inv (original -> internal); optionally the
// caller-facing tables in original order.
struct KnnWork {
  int32_t *perm = nullptr;     // n
  int32_t *inv = nullptr;      // n
  int32_t *nbr_int = nullptr;  // n*k
  uint64_t *keys = nullptr, *keys2 = nullptr;
  uint32_t *vals = nullptr, *vals2 = nullptr;
  float4 *pts = nullptr, *blo = nullptr, *bhi = nullptr;
  uint64_t *kth = nullptr;     // n: every point's k-th key (d2 bits, index)
  int32_t *hist = nullptr, *bsum = nullptr, *total = nullptr;
};
void knn_reserve(Arena &a, int32_t n, int32_t k, KnnWork *w);
hipError_t knn_launch(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                      const KnnWork &w, int32_t *nbr_out, float *d2_out,
                      hipStream_t st);
// The same, also copying the embedding rows (n x d floats, d a multiple of
// 4 up to 16, 16-byte aligned) into internal order in emb_out and taking
// Step 0's max |e| into the control block, as the ladder's first gather does.
hipError_t knn_launch_emb(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                          const KnnWork &w, const float *emb, int32_t d,
                          float *emb_out, hipStream_t st);
// knn_launch with the walk statistics: per 16-point query group, the
// buckets scanned (st_scan) and the inner tree nodes entered (st_node).
hipError_t knn_launch_stats(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                            const KnnWork &w, int32_t *nbr_out,
                            int32_t *st_scan, int32_t *st_node,
                            hipStream_t st);

// Merge ladder on a neighbour table (internal ids; perm/inv may be null
// when internal == original order).
struct LadderArgs {
  const int32_t *nbr;   // n rows: stride pad4(k), or k when check_nbr
  const float4 *pts;    // nullable: points in internal order (x, y, z, index)
  const uint64_t *kth;  // nullable: each point's k-th key from the kNN
  const int32_t *perm;  // nullable
  const int32_t *inv;   // nullable
  const float *emb;     // n*d, caller order
  int32_t n, d, k;
  int32_t n_levels;
  const double *lambdas;
  const int64_t *min_size;
  int32_t max_rounds;
  bool want_energy;
  bool link;            // prepare_graph's linking of isolated nodes (needs pts)
  bool check_nbr;       // validate caller-supplied neighbour ids
  bool emb_ready;       // the ladder's embedding buffer already holds the
                        // rows in internal order, max |e| taken (kNN copy)
  int32_t *labels;      // L*n, caller order
  int64_t *n_comp;      // host
  double *energy;       // host, nullable
};
void ladder_reserve(Arena &a, int32_t n, int32_t d, int32_t k, bool link);
// Where ladder_run, given the arena as it is now, keeps the embeddings in
// internal order (n x d floats).
float *ladder_emb_slot(Arena a, int32_t n, int32_t d, int32_t k, bool link);
// Returns an ezsp_status code; detail text goes through set_error().
int ladder_run(const LadderArgs &args, Ctl *ctl, Arena &a, hipStream_t st);

// Component statistics of a labelling.
void stats_reserve(Arena &a, int32_t n, int64_t n_comp, int32_t d);
int stats_run(const int32_t *labels, int32_t n, int32_t n_comp,
              const float *emb, int32_t d, const float *xyz, int64_t *size,
              float *emb_mean, float *centroid, Ctl *ctl, Arena &a,
              hipStream_t st);

// Grid subsampling: kept point indices in increasing order.
void grid_reserve(Arena &a, int32_t n);
int grid_run(const float *xyz, int32_t n, float h, int32_t *keep,
             int64_t *n_keep, Ctl *ctl, Arena &a, hipStream_t st);

// Affinity and contrastive edge loss over a neighbour table.
struct LossArgs {
  const float *emb;
  int32_t n, d;
  const int32_t *nbr;
  int32_t k;
  const int32_t *cls;
  const uint32_t *word;
  double tau, rho;
  float *affinity;   // n*k, nullable
  float *grad;       // n*d, nullable
  uint8_t *sampled;  // n*k, nullable
};
struct LossResult {
  double loss;
  int64_t n_edges, n_intra, n_inter, n_intra_kept;
};
void loss_reserve(Arena &a, int32_t n, int32_t k);
int loss_run(const LossArgs &g, LossResult *res, Ctl *ctl, Arena &a,
             hipStream_t st);

// Purity and oracle mIoU of a labelling against class ids.
struct PurityResult {
  double miou, purity;
  int64_t n_present;
};
void purity_reserve(Arena &a, int32_t n, int32_t n_comp, int32_t n_cls);
int purity_run(const int32_t *labels, int32_t n, int32_t n_comp,
               const int32_t *cls, int32_t n_cls, int32_t *majority,
               double *iou, PurityResult *res, Ctl *ctl, Arena &a,
               hipStream_t st);

// Point-embedding MLP d_in -> 32 -> 32 -> d_out on the matrix cores.
int mlp_run(const uint16_t *x, int32_t n, int32_t d_in, int32_t d_out,
            const uint16_t *w1, const float *b1, const uint16_t *w2,
            const float *b2, const uint16_t *w3, const float *b3, float *out,
            hipStream_t st);

// Shared host helpers.
void set_error(const char *fmt, ...);
int read_ctl(Ctl *ctl, Ctl *host, hipStream_t st);  // sync + copy back
// ezsp_status of a set of device error bits (detail through set_error).
int status_from_err(uint32_t err);
// Synchronises st and returns the status of the error bits in ctl.
int device_status(const Ctl *ctl, hipStream_t st);
// The static scratch of ezsp_knn_noalloc: its size, and its address on the
// current device (looked up once per device); returns an ezsp_status.
constexpr size_t kNoallocScratchBytes = (size_t)160 << 20;
int noalloc_scratch(void **ptr);
int check_hip(hipError_t e, const char *what);
Ctl *pinned_ctl();
__global__ void k_ctl_init(Ctl *ctl);
__global__ void k_bbox(const float *xyz, int32_t n, Ctl *ctl);
__global__ void k_bbox_fold(Ctl *ctl);
__global__ void k_maxabs(const float *v, int64_t count, Ctl *ctl);
__global__ void k_fixshift(Ctl *ctl, int32_t n);

}  // namespace ezsp

namespace ezsp {
// Optional per-kernel timing with HIP events on the launch stream (off by
// default; a diagnostic for the benchmark).  prof_begin/prof_end bracket one
// launch; prof_flush, called after the stream has synchronised, adds the
// elapsed times to per-name totals.
bool prof_on();
void prof_begin(const char *name, hipStream_t st);
void prof_end(hipStream_t st);
void prof_flush();
// Adds the algorithmic bytes of one launch of a stage to its total.
void prof_bytes(const char *name, double bytes);
}  // namespace ezsp
