// ezsp_grid.hip -- regular-grid subsampling of a point cloud (Sec. 4.1: every
// cloud is subsampled on a regular grid before it is partitioned).
//
// A point's cell is floor((x_i - o_i) / h) per axis in IEEE fp32 (one
// subtraction, one correctly rounded division, floor), o the coordinate-wise
// minimum of the cloud; the cell keeps its smallest point index, and the kept
// indices come out in increasing order.
//
// Cells go into an open-addressing hash table of 16-byte entries (64-bit
// cell key, first index) at load <= 1/2: one pass claims each cell's entry
// with a 64-bit CAS and lowers its first index with atomicMin, recording the
// entry of every point; a device scan over "point p is its entry's first
// index" then writes the kept indices in point order.  The result does not
// depend on the order of the atomics.
#include "ezsp_internal.h"

namespace ezsp {

namespace {

constexpr uint64_t kCellEmpty = ~0ull;
constexpr float kCellLimit = 2097152.0f;  // 2^21 cells per axis

struct alignas(16) CellEntry {
  unsigned long long key;
  uint32_t first;
  uint32_t pad;
};

// splitmix64 finaliser (Steele, Lea and Flood, 2014)
__device__ __forceinline__ uint64_t cell_hash(uint64_t x) {
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

__global__ __launch_bounds__(256) void k_grid_clear(CellEntry *t,
                                                    int64_t cap) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < cap;
       i += (int64_t)gridDim.x * blockDim.x) {
    t[i].key = kCellEmpty;
    t[i].first = 0xffffffffu;
    t[i].pad = 0;
  }
}

__global__ __launch_bounds__(256) void k_grid_insert(
    const float *__restrict__ xyz, int32_t n, float h, const Ctl *box,
    CellEntry *t, uint64_t mask, int32_t *__restrict__ slot, Ctl *ctl) {
  const int32_t p = xcd_tid();
  if (p >= n) return;
  uint64_t c[3];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    const float o = ord2f(box->bbox_enc[a]);
    const float off = __fsub_rn(xyz[3 * (int64_t)p + a], o);
    const float f = floorf(__fdiv_rn(off, h));
    if (!(f >= 0.0f && f < kCellLimit)) {  // also NaN from a bad coordinate
      raise_err(ctl, kErrRange);
      slot[p] = -1;
      return;
    }
    c[a] = (uint64_t)f;
  }
  const uint64_t key = (c[0] << 42) | (c[1] << 21) | c[2];
  uint64_t e = cell_hash(key) & mask;
  for (uint64_t probe = 0; probe <= mask; ++probe) {
    const unsigned long long prev =
        atomicCAS(&t[e].key, (unsigned long long)kCellEmpty,
                  (unsigned long long)key);
    if (prev == kCellEmpty || prev == key) {
      atomicMin(&t[e].first, (uint32_t)p);
      slot[p] = (int32_t)e;
      return;
    }
    e = (e + 1) & mask;
  }
  raise_err(ctl, kErrInternal);  // unreachable at load <= 1/2
  slot[p] = -1;
}

// Scan functor: point i is kept when it is its cell's first index.
struct ScanKeep {
  const int32_t *slot;
  const CellEntry *t;
  int32_t *keep;
  __device__ int32_t value(int32_t i) const {
    const int32_t e = slot[i];
    return (e >= 0 && t[e].first == (uint32_t)i) ? 1 : 0;
  }
  __device__ void emit(int32_t i, int32_t excl, int32_t v) const {
    if (v) keep[excl] = i;
  }
};

uint64_t table_cap(int64_t n) {
  uint64_t cap = 64;
  while (cap < 2 * (uint64_t)n) cap <<= 1;
  return cap;
}

}  // namespace

void grid_reserve(Arena &a, int32_t n) {
  a.take<CellEntry>(table_cap(n));
  a.take<int32_t>(n);
  a.take<int32_t>(scan_blocks(n) + 1);
}

int grid_run(const float *xyz, int32_t n, float h, int32_t *keep,
             int64_t *n_keep, Ctl *ctl, Arena &a, hipStream_t st) {
  const uint64_t cap = table_cap(n);
  CellEntry *t = a.take<CellEntry>(cap);
  int32_t *slot = a.take<int32_t>(n);
  int32_t *bsum = a.take<int32_t>(scan_blocks(n) + 1);
  Ctl *hc = pinned_ctl();
  if (!hc) {
    set_error("hipHostMalloc of the control block failed");
    return -5;
  }
  const int nt = 256;
  const int64_t gb = (n + nt - 1) / nt;
  prof_begin("grid_subsample", st);
  hipLaunchKernelGGL(k_bbox, dim3((unsigned)(gb < 256 ? gb : 256)), dim3(nt),
                     0, st, xyz, n, ctl);
  hipLaunchKernelGGL(k_bbox_fold, dim3(1), dim3(64), 0, st, ctl);
  const int64_t cb = (int64_t)((cap + nt - 1) / nt);
  hipLaunchKernelGGL(k_grid_clear, dim3((unsigned)(cb < 4096 ? cb : 4096)),
                     dim3(nt), 0, st, t, (int64_t)cap);
  hipLaunchKernelGGL(k_grid_insert, dim3(xcd_grid(gb)), dim3(nt), 0, st, xyz,
                     n, h, ctl, t, cap - 1, slot, ctl);
  device_scan(ScanKeep{slot, t, keep}, n, bsum, &ctl->n_out, st);
  prof_end(st);
  int rc = read_ctl(ctl, hc, st);
  if (rc) return rc;
  // algorithmic bytes: read xyz, write the kept indices
  prof_bytes("grid_subsample", 12.0 * n + 4.0 * hc->n_out);
  if (hc->err & kErrNonFinite) {
    set_error("non-finite coordinate in xyz");
    return -2;
  }
  if (hc->err & kErrRange) {
    set_error("the cloud spans 2^21 or more cells of size h on some axis");
    return -3;
  }
  if (hc->err) {
    set_error("internal check failed in the grid subsampling (0x%x)",
              hc->err);
    return -5;
  }
  *n_keep = hc->n_out;
  return 0;
}

}  // namespace ezsp
