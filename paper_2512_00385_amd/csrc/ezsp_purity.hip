// ezsp_purity.hip -- partition purity and oracle mIoU (Sec. 4.2 "Metrics":
// every superpoint takes the majority ground-truth class of its points; the
// mIoU of that labelling bounds what a classifier on the superpoints can
// reach).
//
// Points are sorted by the key component * n_cls + class; each run of equal
// keys is one (component, class) count, found by a binary search from the
// run head, and a 64-bit atomicMax of (count, ~class) per component picks the
// majority with ties to the smallest class.  Per-class TP, ground-truth and
// predicted counts are then exact integer histograms, and one thread forms
// IoU_c = TP / (gt + pred - TP) and their mean in class order, so the result
// is independent of scheduling.
#include "ezsp_internal.h"

namespace ezsp {

namespace {

constexpr int kPuNT = 256;
constexpr int kPuLdsCls = 2048;  // class histograms held in LDS up to here

__global__ __launch_bounds__(kPuNT) void k_pu_keys(
    const int32_t *__restrict__ label, const int32_t *__restrict__ cls,
    int32_t n, int32_t nc, int32_t n_cls, uint64_t *keys, uint32_t *vals,
    Ctl *ctl) {
  const int32_t p = xcd_tid();
  if (p >= n) return;
  const int32_t c = label[p], y = cls[p];
  if ((uint32_t)c >= (uint32_t)nc || (uint32_t)y >= (uint32_t)n_cls) {
    raise_err(ctl, kErrBadIndex);
    keys[p] = 0;
  } else {
    keys[p] = (uint64_t)c * (uint64_t)n_cls + (uint64_t)y;
  }
  vals[p] = (uint32_t)p;
}

__global__ __launch_bounds__(kPuNT) void k_pu_clear(unsigned long long *best,
                                                    int32_t nc,
                                                    unsigned long long *cnt,
                                                    int64_t ncnt) {
  const int64_t i = blockIdx.x * (int64_t)kPuNT + threadIdx.x;
  if (i < nc) best[i] = 0;
  if (i < ncnt) cnt[i] = 0;
}

// One thread per run head: the run's length by binary search, then the
// component's (count, ~class) maximum.
__global__ __launch_bounds__(kPuNT) void k_pu_runs(const uint64_t *__restrict__ key,
                                                   int32_t n, int32_t n_cls,
                                                   unsigned long long *best) {
  const int32_t i = xcd_tid();
  if (i >= n) return;
  const uint64_t x = key[i];
  if (i > 0 && key[i - 1] == x) return;
  int32_t lo = i + 1, hi = n;  // first index past the run
  while (lo < hi) {
    const int32_t mid = lo + (hi - lo) / 2;
    if (key[mid] == x) lo = mid + 1;
    else hi = mid;
  }
  const uint64_t count = (uint64_t)(lo - i);
  const uint32_t comp = (uint32_t)(x / (uint64_t)n_cls);
  const uint32_t c = (uint32_t)(x % (uint64_t)n_cls);
  atomicMax(&best[comp], (unsigned long long)((count << 32) | (0xffffffffu - c)));
}

__global__ __launch_bounds__(kPuNT) void k_pu_major(
    const unsigned long long *best, int32_t nc, int32_t *maj) {
  const int32_t c = xcd_tid();
  if (c >= nc) return;
  const unsigned long long b = best[c];
  maj[c] = b ? (int32_t)(0xffffffffu - (uint32_t)(b & 0xffffffffu)) : -1;
}

// Per-class counts: cnt[0..n_cls) TP, [n_cls..2n_cls) ground truth,
// [2n_cls..3n_cls) predicted.
template <bool LDS>
__global__ __launch_bounds__(kPuNT) void k_pu_count(
    const int32_t *__restrict__ label, const int32_t *__restrict__ cls,
    int32_t n, int32_t nc, const int32_t *__restrict__ maj, int32_t n_cls,
    unsigned long long *cnt) {
  __shared__ uint32_t h[LDS ? 3 * kPuLdsCls : 1];
  if (LDS) {
    for (int32_t i = threadIdx.x; i < 3 * n_cls; i += kPuNT) h[i] = 0;
    __syncthreads();
  }
  for (int64_t p = blockIdx.x * (int64_t)kPuNT + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * kPuNT) {
    const int32_t c = label[p], g = cls[p];
    // out-of-range ids were reported by k_pu_keys; skip them here
    if ((uint32_t)c >= (uint32_t)nc || (uint32_t)g >= (uint32_t)n_cls) continue;
    const int32_t y = maj[c];
    if (y < 0) continue;
    if (LDS) {
      atomicAdd(&h[n_cls + g], 1u);
      atomicAdd(&h[2 * n_cls + y], 1u);
      if (g == y) atomicAdd(&h[g], 1u);
    } else {
      atomicAdd(&cnt[n_cls + g], 1ull);
      atomicAdd(&cnt[2 * n_cls + y], 1ull);
      if (g == y) atomicAdd(&cnt[g], 1ull);
    }
  }
  if (LDS) {
    __syncthreads();
    for (int32_t i = threadIdx.x; i < 3 * n_cls; i += kPuNT)
      if (h[i]) atomicAdd(&cnt[i], (unsigned long long)h[i]);
  }
}

// IoU per class in parallel, staged in LDS a chunk of classes at a time,
// then the mean in class order by one thread.
constexpr int kPuChunk = 4096;

__global__ __launch_bounds__(kPuNT) void k_pu_final(
    const unsigned long long *cnt, int32_t n_cls, int32_t n, double *iou,
    Ctl *ctl) {
  __shared__ double v[kPuChunk];
  __shared__ unsigned long long tps[kPuNT];
  double sum = 0.0;
  int64_t present = 0;
  unsigned long long tp_mine = 0;
  for (int32_t base = 0; base < n_cls; base += kPuChunk) {
    const int32_t len = min(kPuChunk, n_cls - base);
    for (int32_t i = threadIdx.x; i < len; i += kPuNT) {
      const int32_t c = base + i;
      const unsigned long long tp = cnt[c], gt = cnt[n_cls + c],
                               pr = cnt[2 * n_cls + c];
      tp_mine += tp;
      const double x = gt ? __ddiv_rn((double)tp, (double)(gt + pr - tp))
                          : __builtin_nan("");
      iou[c] = x;
      v[i] = x;
    }
    __syncthreads();
    if (threadIdx.x == 0)
      for (int32_t i = 0; i < len; ++i)
        if (v[i] == v[i]) {  // present classes (absent ones are NaN)
          sum = __dadd_rn(sum, v[i]);
          ++present;
        }
    __syncthreads();
  }
  tps[threadIdx.x] = tp_mine;
  __syncthreads();
  if (threadIdx.x != 0) return;
  unsigned long long tp_all = 0;
  for (int t = 0; t < kPuNT; ++t) tp_all += tps[t];
  ctl->pu_miou = __ddiv_rn(sum, (double)present);
  ctl->pu_purity = __ddiv_rn((double)tp_all, (double)n);
  ctl->pu_present = present;
}

int key_bits(int64_t nkeys) {  // bits of nkeys - 1, at least 1
  int b = 1;
  while (b < 64 && ((uint64_t)1 << b) < (uint64_t)nkeys) ++b;
  return b;
}

}  // namespace

void purity_reserve(Arena &a, int32_t n, int32_t n_comp, int32_t n_cls) {
  a.take<uint64_t>(n);
  a.take<uint64_t>(n);
  a.take<uint32_t>(n);
  a.take<uint32_t>(n);
  a.take<int32_t>(radix_hist_ints(n));
  a.take<int32_t>(scan_blocks(radix_hist_ints(n)) + 1);
  a.take<int32_t>(4);
  a.take<unsigned long long>(n_comp);
  a.take<int32_t>(n_comp);
  a.take<unsigned long long>(3 * (size_t)n_cls);
  a.take<double>(n_cls);
}

int purity_run(const int32_t *labels, int32_t n, int32_t nc,
               const int32_t *cls, int32_t n_cls, int32_t *majority,
               double *iou, PurityResult *res, Ctl *ctl, Arena &a,
               hipStream_t st) {
  uint64_t *keys = a.take<uint64_t>(n);
  uint64_t *keys2 = a.take<uint64_t>(n);
  uint32_t *vals = a.take<uint32_t>(n);
  uint32_t *vals2 = a.take<uint32_t>(n);
  int32_t *hist = a.take<int32_t>(radix_hist_ints(n));
  int32_t *bsum = a.take<int32_t>(scan_blocks(radix_hist_ints(n)) + 1);
  int32_t *total = a.take<int32_t>(4);
  unsigned long long *best = a.take<unsigned long long>(nc);
  int32_t *maj_ws = a.take<int32_t>(nc);
  unsigned long long *cnt = a.take<unsigned long long>(3 * (size_t)n_cls);
  double *iou_ws = a.take<double>(n_cls);
  int32_t *maj = majority ? majority : maj_ws;
  double *iou_out = iou ? iou : iou_ws;
  Ctl *hc = pinned_ctl();
  if (!hc) {
    set_error("hipHostMalloc of the control block failed");
    return -5;
  }
  const int nt = kPuNT;
  const int64_t gb = (n + nt - 1) / nt;
  prof_begin("purity", st);
  hipLaunchKernelGGL(k_pu_keys, dim3(xcd_grid(gb)), dim3(nt), 0, st, labels,
                     cls, n, nc, n_cls, keys, vals, ctl);
  const bool alt =
      radix_sort_pairs(keys, vals, keys2, vals2, n,
                       key_bits((int64_t)nc * n_cls), hist, bsum, total, ctl,
                       st);
  const uint64_t *sorted = alt ? keys2 : keys;
  const int64_t ncnt = 3 * (int64_t)n_cls;
  const int64_t cl = (nc > ncnt ? nc : ncnt);
  hipLaunchKernelGGL(k_pu_clear, dim3((unsigned)((cl + nt - 1) / nt)),
                     dim3(nt), 0, st, best, nc, cnt, ncnt);
  hipLaunchKernelGGL(k_pu_runs, dim3(xcd_grid(gb)), dim3(nt), 0, st, sorted,
                     n, n_cls, best);
  hipLaunchKernelGGL(k_pu_major, dim3(xcd_grid((nc + nt - 1) / nt)), dim3(nt),
                     0, st, best, nc, maj);
  const unsigned cg = (unsigned)(gb < 1024 ? gb : 1024);
  if (n_cls <= kPuLdsCls)
    hipLaunchKernelGGL(k_pu_count<true>, dim3(cg), dim3(nt), 0, st, labels,
                       cls, n, nc, maj, n_cls, cnt);
  else
    hipLaunchKernelGGL(k_pu_count<false>, dim3(cg), dim3(nt), 0, st, labels,
                       cls, n, nc, maj, n_cls, cnt);
  hipLaunchKernelGGL(k_pu_final, dim3(1), dim3(nt), 0, st, cnt, n_cls, n,
                     iou_out, ctl);
  prof_end(st);
  prof_bytes("purity", 8.0 * n + 4.0 * nc + 8.0 * n_cls);
  int rc = read_ctl(ctl, hc, st);
  if (rc) return rc;
  if (hc->err & kErrBadIndex) {
    set_error("label outside [0, n_comp) or class outside [0, n_cls)");
    return -1;
  }
  if (hc->err) {
    set_error("internal check failed in the purity (0x%x)", hc->err);
    return -5;
  }
  res->miou = hc->pu_miou;
  res->purity = hc->pu_purity;
  res->n_present = hc->pu_present;
  return 0;
}

}  // namespace ezsp
