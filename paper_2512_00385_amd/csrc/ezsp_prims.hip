// ezsp_prims.hip -- device-wide scan tail, LSD radix sort, control block and
// fixed-point shift kernels, and the host helpers shared by the launchers.
#include <stdarg.h>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>
#include <stdio.h>
#include <stddef.h>
#include <string.h>

#include "ezsp_internal.h"

namespace ezsp {

// ---------------------------------------------------------------------------
// scan of the per-block sums: one block of 1024 threads walks the array in
// chunks of 4096 with a running carry.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_scan_bsums(int32_t *bsum, int32_t nb,
                                                     int32_t *total) {
  __shared__ int32_t wsum[1024 / kWave];
  constexpr int kPer = 4;
  int32_t carry = 0;
  for (int32_t c0 = 0; c0 < nb; c0 += 1024 * kPer) {
    int32_t v[kPer];
    int32_t s = 0;
    const int32_t base = c0 + threadIdx.x * kPer;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      int32_t i = base + j;
      v[j] = (i < nb) ? bsum[i] : 0;
      s += v[j];
    }
    int32_t tot;
    int32_t run = carry + block_excl_scan<1024>(s, wsum, &tot);
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      int32_t i = base + j;
      if (i < nb) bsum[i] = run;
      run += v[j];
    }
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

// ---------------------------------------------------------------------------
// LSD radix sort, 8-bit digits.  Tile of kSortTile keys per block; inside a
// tile, key j*256 + t is handled by thread t at step j, so (step, thread)
// order is the input order and the per-step ranking keeps the sort stable.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSortNT) void k_rs_hist(const uint64_t *keys,
                                                     int32_t n, int shift,
                                                     int32_t *hist, int32_t nb) {
  __shared__ int32_t h[kSortBins];
  for (int d = threadIdx.x; d < kSortBins; d += kSortNT) h[d] = 0;
  __syncthreads();
  const int32_t base = blockIdx.x * kSortTile;
#pragma unroll 4
  for (int j = 0; j < kSortItems; ++j) {
    int32_t i = base + j * kSortNT + threadIdx.x;
    if (i < n) atomicAdd(&h[(keys[i] >> shift) & (kSortBins - 1)], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < kSortBins; d += kSortNT)
    hist[d * nb + blockIdx.x] = h[d];
}

// The scatter takes a tile with twice the histogram's threads, half the
// steps: fewer barriers for the same tile.
constexpr int kScatNT = 2 * kSortNT;
constexpr int kScatItems = kSortTile / kScatNT;

// VALS: keys carry 32-bit values; otherwise the keys alone (a value packed
// into bits the sort does not look at).
template <bool VALS>
__global__ __launch_bounds__(kScatNT) void k_rs_scatter(
    const uint64_t *__restrict__ kin, const uint32_t *__restrict__ vin,
    uint64_t *__restrict__ kout, uint32_t *__restrict__ vout, int32_t n,
    int shift, const int32_t *__restrict__ offs, int32_t nb, Ctl *ctl) {
  constexpr int kW = kScatNT / kWave;
  static_assert(kSortBins <= kScatNT, "one digit per thread in the prefix");
  __shared__ int32_t run[kSortBins];
  // per step: the waves' counts per digit, and the positions they turn
  // into (kept apart so that the counts can be reset while the positions
  // are read: two barriers a step)
  __shared__ int32_t cnt[kW][kSortBins];
  __shared__ int32_t pos0[kW][kSortBins];
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  if (threadIdx.x < kSortBins) {
    run[threadIdx.x] = offs[threadIdx.x * nb + blockIdx.x];
#pragma unroll
    for (int w = 0; w < kW; ++w) cnt[w][threadIdx.x] = 0;
  }
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
  const int32_t base = blockIdx.x * kSortTile;
  // the thread's keys and values of the whole tile, loaded before the first
  // step (clamped indices, no branch): the steps then wait on LDS only
  uint64_t kt[kScatItems];
  uint32_t vt[kScatItems];
#pragma unroll
  for (int j = 0; j < kScatItems; ++j) {
    const int32_t i = min(base + j * kScatNT + (int32_t)threadIdx.x, n - 1);
    kt[j] = kin[i];
    vt[j] = VALS ? vin[i] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kScatItems; ++j) {
    const int32_t i = base + j * kScatNT + threadIdx.x;
    const bool valid = i < n;
    const uint64_t key = valid ? kt[j] : 0ull;
    const uint32_t val = valid ? vt[j] : 0u;
    const int dig = (int)((key >> shift) & (kSortBins - 1));
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const int bit = (dig >> b) & 1;
      const uint64_t bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    const int rank = __popcll(peers & lt_mask);
    if (valid && rank == 0) cnt[wid][dig] = __popcll(peers);
    __syncthreads();
    if (threadIdx.x < kSortBins) {
      const int d = threadIdx.x;
      int32_t p = run[d];
#pragma unroll
      for (int w = 0; w < kW; ++w) {
        const int32_t c = cnt[w][d];
        cnt[w][d] = 0;
        pos0[w][d] = p;
        p += c;
      }
      run[d] = p;
    }
    __syncthreads();
    if (valid) {
      const int32_t pos = pos0[wid][dig] + rank;
      if ((uint32_t)pos < (uint32_t)n) {
        kout[pos] = key;
        if (VALS) vout[pos] = val;
      } else {
        raise_err(ctl, kErrInternal);
      }
    }
  }
}

size_t radix_hist_ints(int32_t n) {
  return (size_t)kSortBins * (size_t)sort_blocks(n);
}

bool radix_sort_pairs(uint64_t *keys, uint32_t *vals, uint64_t *keys_alt,
                      uint32_t *vals_alt, int32_t n, int nbits,
                      int32_t *hist, int32_t *bsum, int32_t *total, Ctl *ctl,
                      hipStream_t st) {
  if (n <= 1) return false;
  const int32_t nb = sort_blocks(n);
  uint64_t *kin = keys, *kout = keys_alt;
  uint32_t *vin = vals, *vout = vals_alt;
  bool flip = false;
  for (int shift = 0; shift < nbits; shift += 8) {
    hipLaunchKernelGGL(k_rs_hist, dim3(nb), dim3(kSortNT), 0, st, kin, n,
                       shift, hist, nb);
    const int32_t nh = kSortBins * nb;
    device_scan(ScanArray{hist, hist, nh, nullptr}, nh, bsum, total, st);
    hipLaunchKernelGGL(k_rs_scatter<true>, dim3(nb), dim3(kScatNT), 0, st,
                       kin, vin, kout, vout, n, shift, hist, nb, ctl);
    uint64_t *tk = kin;
    kin = kout;
    kout = tk;
    uint32_t *tv = vin;
    vin = vout;
    vout = tv;
    flip = !flip;
  }
  return flip;
}

// ---------------------------------------------------------------------------
// control block, max |v| and the fixed-point shift
// ---------------------------------------------------------------------------
__global__ void k_ctl_init(Ctl *ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctl->err = 0;
    ctl->F = 0;
    ctl->any_choice = 0;
    ctl->n_next = 0;
    ctl->e_next = 0;
    ctl->slots = 0;
    ctl->maxabs_bits = 0;
    ctl->n_long = 0;
    ctl->n_lchunk = 0;
    for (int a = 0; a < 3; ++a) {
      ctl->bbox_enc[a] = f2ord(INFINITY);
      ctl->bbox_enc[3 + a] = f2ord(-INFINITY);
    }
    ctl->n_big = 0;
    ctl->e_rev = 0;
    ctl->e_fwd = 0;
    ctl->n_cbig = 0;
    ctl->n_tiles = 0;
    ctl->tail_level = -1;
    ctl->cut_w2 = 0;
    ctl->fid_total = 0.0;
    ctl->maxabs_x_bits = 0;
    ctl->Fx = 0;
    ctl->n_iso = 0;
    ctl->n_link = 0;
    ctl->n_out = 0;
    ctl->sel_mode = 0;
    ctl->sel_prefix = 0;
    ctl->sel_mask = 0;
    ctl->sel_rank = 0;
    ctl->le_edges = 0;
    ctl->le_intra = 0;
    ctl->le_keep = 0;
    ctl->le_loss = 0.0;
    ctl->pu_miou = 0.0;
    ctl->pu_purity = 0.0;
    ctl->pu_present = 0;
  }
  if (blockIdx.x == 0) {
    stripe_zero(ctl->e_next_s);
    stripe_zero(ctl->e_fwd_s);
    stripe_zero(ctl->maxabs_s);
    for (int i = threadIdx.x; i < 6 * kStripes; i += blockDim.x)
      ctl->bbox_s[i / kStripes][i % kStripes].v =
          f2ord(i < 3 * kStripes ? INFINITY : -INFINITY);
  }
}

__global__ __launch_bounds__(256) void k_maxabs(const float *v, int64_t count,
                                                Ctl *ctl) {
  uint32_t m = 0;
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x) {
    float x = v[i];
    if (!isfinite(x)) bad = true;
    else m = max(m, __float_as_uint(fabsf(x)));
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
    atomicMax(&ctl->maxabs_bits, r);
    if (sbad) raise_err(ctl, kErrNonFinite);
  }
}

// F = min(40, 61 - ceil(log2 n) - max(0, ceil(log2 A))), A = max |e|.
__global__ void k_fixshift(Ctl *ctl, int32_t n) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  uint32_t bits = ctl->maxabs_bits;
  for (int i = 0; i < kStripes; ++i)
    bits = max(bits, (uint32_t)ctl->maxabs_s[i].v);
  const int F = fixshift_rule(__uint_as_float(bits), n);
  ctl->F = F;
  if (F < 16) raise_err(ctl, kErrRange);
}

bool radix_sort_keys(uint64_t *keys, uint64_t *keys_alt, int32_t n,
                     int shift0, int nbits, int32_t *hist, int32_t *bsum,
                     int32_t *total, Ctl *ctl, hipStream_t st) {
  if (n <= 1) return false;
  const int32_t nb = sort_blocks(n);
  uint64_t *kin = keys, *kout = keys_alt;
  bool flip = false;
  for (int shift = shift0; shift < shift0 + nbits; shift += 8) {
    hipLaunchKernelGGL(k_rs_hist, dim3(nb), dim3(kSortNT), 0, st, kin, n,
                       shift, hist, nb);
    const int32_t nh = kSortBins * nb;
    device_scan(ScanArray{hist, hist, nh, nullptr}, nh, bsum, total, st);
    hipLaunchKernelGGL(k_rs_scatter<false>, dim3(nb), dim3(kScatNT), 0, st,
                       kin, (const uint32_t *)nullptr, kout, (uint32_t *)nullptr,
                       n, shift, hist, nb, ctl);
    uint64_t *tk = kin;
    kin = kout;
    kout = tk;
    flip = !flip;
  }
  return flip;
}

// ---------------------------------------------------------------------------
// host helpers
// ---------------------------------------------------------------------------
static thread_local char g_msg[512];

void set_error(const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
}

const char *last_error_text() { return g_msg; }

int check_hip(hipError_t e, const char *what) {
  if (e == hipSuccess) return 0;
  set_error("%s: %s", what, hipGetErrorString(e));
  return -5;  // EZSP_ERR_DEVICE
}

// The host copy of the control block: fine-grained (coherent) pinned
// memory, mapped into the device's address space, so that a kernel can
// write it directly (k_ctl_export) instead of a DMA copy.
namespace {
thread_local Ctl *t_host_ctl = nullptr;
thread_local Ctl *t_host_ctl_dev = nullptr;
}  // namespace

Ctl *pinned_ctl() {
  if (!t_host_ctl) {
    void *q = nullptr;
    if (hipHostMalloc(&q, sizeof(Ctl),
                      hipHostMallocMapped | hipHostMallocCoherent) !=
        hipSuccess)
      return nullptr;
    void *d = nullptr;
    if (hipHostGetDevicePointer(&d, q, 0) != hipSuccess || !d) {
      hipHostFree(q);
      return nullptr;
    }
    t_host_ctl = static_cast<Ctl *>(q);
    t_host_ctl_dev = static_cast<Ctl *>(d);
  }
  return t_host_ctl;
}

// Copies the control block to its host copy: every field but the striped
// counters word by word, then e_next and e_fwd as the sums of their
// stripes (-1 beyond int32).
__global__ __launch_bounds__(256) void k_ctl_export(const Ctl *ctl,
                                                    Ctl *host, uint32_t seq) {
  const uint32_t *src = reinterpret_cast<const uint32_t *>(ctl);
  uint32_t *dst = reinterpret_cast<uint32_t *>(host);
  constexpr uint32_t s0 = offsetof(Ctl, e_next_s) / 4;
  constexpr uint32_t s1 = offsetof(Ctl, tail_nc) / 4;
  constexpr uint32_t nw = sizeof(Ctl) / 4;
  constexpr uint32_t en = offsetof(Ctl, e_next) / 4;
  constexpr uint32_t ef = offsetof(Ctl, e_fwd) / 4;
  constexpr uint32_t sq = offsetof(Ctl, seq) / 4;
  static_assert(offsetof(Ctl, e_fwd_s) > offsetof(Ctl, e_next_s) &&
                    offsetof(Ctl, maxabs_s) < offsetof(Ctl, tail_nc),
                "the striped counters lie between e_next_s and tail_nc");
  for (uint32_t i = threadIdx.x; i < nw; i += blockDim.x)
    if ((i < s0 || i >= s1) && i != en && i != ef && i != sq) dst[i] = src[i];
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    long long a = lane < kStripes ? ctl->e_next_s[lane].v : 0;
    long long b = lane < kStripes ? ctl->e_fwd_s[lane].v : 0;
    a = wave_sum(a);
    b = wave_sum(b);
    if (lane == 0) {
      host->e_next = a > INT32_MAX ? -1 : (int32_t)a;
      host->e_fwd = b > INT32_MAX ? -1 : (int32_t)b;
    }
  }
  // every field above is in host memory before the export number
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence_system();
    __hip_atomic_store(&host->seq, seq, __ATOMIC_RELEASE,
                       __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// ---------------------------------------------------------------------------
// per-kernel event timing (diagnostic)
// ---------------------------------------------------------------------------
namespace {
struct ProfRec {
  const char *name;
  hipEvent_t a, b;
};
struct ProfTotal {
  int64_t launches = 0;
  double ms = 0.0;
  double bytes = 0.0;
};
std::mutex g_prof_mu;
bool g_prof = false;
std::vector<hipEvent_t> g_pool;
std::vector<ProfRec> g_pending;
std::unordered_map<std::string, ProfTotal> g_totals;
std::string g_only;  // record events for this stage only ("" = all)

hipEvent_t pool_get() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

bool prof_on() { return g_prof; }

void prof_begin(const char *name, hipStream_t st) {
  if (!g_prof) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_only.empty() && g_only != name) {
    g_pending.push_back(ProfRec{name, nullptr, nullptr});  // not timed
    return;
  }
  ProfRec r{name, pool_get(), pool_get()};
  if (!r.a || !r.b) return;
  hipEventRecord(r.a, st);
  g_pending.push_back(r);
}

void prof_end(hipStream_t st) {
  if (!g_prof) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_pending.empty() && g_pending.back().b)
    hipEventRecord(g_pending.back().b, st);
}

void prof_flush() {
  if (!g_prof) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (const ProfRec &r : g_pending) {
    if (!r.a) continue;
    float ms = 0.0f;
    if (hipEventSynchronize(r.b) == hipSuccess &&
        hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      ProfTotal &t = g_totals[r.name];
      t.launches += 1;
      t.ms += ms;
    }
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_pending.clear();
}

void prof_bytes(const char *name, double bytes) {
  if (!g_prof) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_totals[name].bytes += bytes;
}

int prof_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof = on != 0;
  g_totals.clear();
  g_pending.clear();
  return 0;
}

int prof_only(const char *name) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_only = name ? name : "";
  return 0;
}

int prof_read(const char *name, int64_t *launches, double *ms,
              double *bytes) {
  prof_flush();  // launches of asynchronous entry points still pending
  std::lock_guard<std::mutex> lk(g_prof_mu);
  auto it = g_totals.find(name ? name : "");
  if (it == g_totals.end()) {
    if (launches) *launches = 0;
    if (ms) *ms = 0.0;
    if (bytes) *bytes = 0.0;
    return -1;
  }
  if (launches) *launches = it->second.launches;
  if (ms) *ms = it->second.ms;
  if (bytes) *bytes = it->second.bytes;
  return 0;
}

int read_ctl(Ctl *ctl, Ctl *host, hipStream_t st) {
  int rc = check_hip(hipGetLastError(), "kernel launch");
  if (rc) return rc;
  if (host != t_host_ctl || !t_host_ctl_dev) {
    set_error("read_ctl needs the thread's pinned control block");
    return -5;
  }
  // the host waits for the export number instead of a stream
  // synchronisation (whose wake-up takes tens of microseconds); the stream
  // is polled now and then so that a failed kernel ends the wait
  static thread_local uint32_t t_seq = 0;
  const uint32_t want = ++t_seq;
  hipLaunchKernelGGL(k_ctl_export, dim3(1), dim3(256), 0, st,
                     (const Ctl *)ctl, t_host_ctl_dev, want);
  rc = check_hip(hipGetLastError(), "k_ctl_export launch");
  if (rc) return rc;
  for (uint32_t spin = 1;; ++spin) {
    if (__atomic_load_n(&host->seq, __ATOMIC_ACQUIRE) == want) break;
    if ((spin & 1023) == 0) {
      const hipError_t e = hipStreamQuery(st);
      if (e == hipSuccess) {  // the stream drained: the number is there
        if (__atomic_load_n(&host->seq, __ATOMIC_ACQUIRE) == want) break;
        set_error("control block export did not arrive");
        return -5;
      }
      if (e != hipErrorNotReady) return check_hip(e, "stream");
    }
  }
  prof_flush();
  return 0;
}

int status_from_err(uint32_t err) {
  if (err & kErrNonFinite) {
    set_error("non-finite value in the input");
    return -2;
  }
  if (err & kErrRange) {
    set_error("values too large for exact fixed-point sums (F < 16)");
    return -3;
  }
  if (err & kErrBadIndex) {
    set_error("an index of the input is out of range");
    return -1;
  }
  if (err & kErrJump) {
    set_error("pointer jumping did not reach the roots");
    return -5;
  }
  set_error("internal consistency check failed on the device (0x%x)", err);
  return -5;
}

int device_status(const Ctl *ctl, hipStream_t st) {
  int rc = check_hip(hipGetLastError(), "kernel launch");
  if (rc) return rc;
  rc = check_hip(hipStreamSynchronize(st), "hipStreamSynchronize");
  if (rc) return rc;
  // the stream's work is done: a plain copy of the error word into host
  // memory (no pinned buffer, so the query allocates nothing)
  uint32_t err = 0;
  rc = check_hip(hipMemcpy(&err, &ctl->err, sizeof(err),
                           hipMemcpyDeviceToHost),
                 "hipMemcpy(error word)");
  if (rc) return rc;
  return err ? status_from_err(err) : 0;
}

Tree make_tree(int32_t n) {
  Tree t;
  memset(&t, 0, sizeof(t));
  int32_t cnt = (n + kBucket - 1) / kBucket;
  int32_t off = 0;
  int l = 0;
  for (;;) {
    t.off[l] = off;
    t.cnt[l] = cnt;
    off += cnt;
    if (cnt <= 1 || l + 1 >= kMaxTreeLevels) break;
    cnt = (cnt + kFan - 1) / kFan;
    ++l;
  }
  t.top = l;
  t.total = off;
  return t;
}

}  // namespace ezsp
