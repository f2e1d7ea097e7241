// ezsp_loss.hip -- pairwise affinity and the contrastive edge loss over the
// k-nearest-neighbour graph (Sec. 3.1: Eq. softmax, a = exp(-|e_p - e_q| /
// tau); Eq. loss, -log a over intra-class edges and -log(1 - a) over
// inter-class edges, with intra edges dropped at random until they are at
// most a fraction rho of the sample).
//
// Edges are the unordered pairs of the kNN relation.  The slot p*k + j that
// owns a pair is the smallest slot listing it: slot (p, j) owns its pair
// when q = nbr[p*k+j] does not appear earlier in row p and either p < q or
// row q does not list p.  That slot's caller-supplied random word draws the
// pair.  With rho < 1 the sample keeps m = min(n_intra,
// floor(rho * n_inter / (1 - rho))) intra pairs: those whose 64-bit key
// (word, slot) is among the m smallest, found exactly by an 8-pass MSB radix
// select over the keys (keys are distinct, so the m-th smallest is a sharp
// threshold).  Every inter pair is kept.
//
// Distances, affinities, loss terms and gradient contributions are fp32; the
// loss is summed in fp64.  -log a is d / tau and -log(1 - a) is
// -log(-expm1(-d / tau)); the gradient of |e_p - e_q| at e_p = e_q is 0.
#include "ezsp_internal.h"

namespace ezsp {

namespace {

enum : uint8_t { kSlotNone = 0, kSlotInter = 1, kSlotIntra = 2 };

constexpr int kLeNT = 256;
constexpr int kLeGrid = 2048;  // grid-stride kernels: one atomic per block

template <class T>
__device__ __forceinline__ T block_sum(T v, T *sh) {
  v = wave_sum(v);
  const int wid = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sh[wid] = v;
  __syncthreads();
  T s = 0;
  if (threadIdx.x == 0)
    for (int w = 0; w < kLeNT / kWave; ++w) s += sh[w];
  return s;  // valid in thread 0
}

// Slot status and the pair counts.
__global__ __launch_bounds__(kLeNT) void k_le_classify(
    const int32_t *__restrict__ nbr, int32_t n, int32_t k,
    const int32_t *__restrict__ cls, uint8_t *__restrict__ status, Ctl *ctl) {
  __shared__ unsigned long long sh[kLeNT / kWave];
  const int64_t ns = (int64_t)n * k;
  unsigned long long edges = 0, intra = 0;
  for (int64_t s = blockIdx.x * (int64_t)kLeNT + threadIdx.x; s < ns;
       s += (int64_t)gridDim.x * kLeNT) {
    const int32_t p = (int32_t)(s / k);
    const int32_t j = (int32_t)(s - (int64_t)p * k);
    const int32_t q = nbr[s];
    uint8_t v = kSlotNone;
    if (q < -1 || q >= n) {
      raise_err(ctl, kErrBadIndex);
    } else if (q >= 0 && q != p) {
      bool own = true;
      const int32_t *row = nbr + (int64_t)p * k;
      for (int32_t t = 0; t < j && own; ++t) own = row[t] != q;
      if (own && q < p) {
        const int32_t *rq = nbr + (int64_t)q * k;
        for (int32_t t = 0; t < k && own; ++t) own = rq[t] != p;
      }
      if (own) {
        v = (cls[p] == cls[q]) ? kSlotIntra : kSlotInter;
        edges += 1;
        intra += (v == kSlotIntra);
      }
    }
    status[s] = v;
  }
  const unsigned long long e = block_sum(edges, sh);
  __syncthreads();
  const unsigned long long i = block_sum(intra, sh);
  if (threadIdx.x == 0) {
    if (e) atomicAdd(&ctl->le_edges, e);
    if (i) atomicAdd(&ctl->le_intra, i);
  }
}

// The size of the intra sample and the selection mode.
__global__ void k_le_quota(Ctl *ctl, double rho) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int64_t n_intra = (int64_t)ctl->le_intra;
  const int64_t n_inter = (int64_t)ctl->le_edges - n_intra;
  int64_t m = n_intra;
  if (rho < 1.0) {
    const double cap =
        floor(__ddiv_rn(__dmul_rn(rho, (double)n_inter), __dsub_rn(1.0, rho)));
    if (cap < (double)m) m = (int64_t)cap;
  }
  ctl->le_keep = (unsigned long long)m;
  ctl->sel_mode = (m == 0) ? 0 : (m == n_intra ? 1 : 2);
  ctl->sel_prefix = 0;
  ctl->sel_mask = 0;
  ctl->sel_rank = m - 1;  // 0-based rank of the largest kept key
}

__device__ __forceinline__ uint64_t draw_key(const uint32_t *word, int64_t s) {
  return ((uint64_t)word[s] << 32) | (uint64_t)s;
}

// One radix-select pass: histogram of the 8-bit digit at `shift` over the
// intra keys that match the prefix fixed so far.
__global__ __launch_bounds__(kLeNT) void k_le_hist(
    const uint8_t *__restrict__ status, const uint32_t *__restrict__ word,
    int64_t ns, int shift, const Ctl *ctl, uint32_t *hist) {
  if (ctl->sel_mode != 2) return;
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t prefix = ctl->sel_prefix, mask = ctl->sel_mask;
  for (int64_t s = blockIdx.x * (int64_t)kLeNT + threadIdx.x; s < ns;
       s += (int64_t)gridDim.x * kLeNT) {
    if (status[s] != kSlotIntra) continue;
    const uint64_t key = draw_key(word, s);
    if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & 255], 1u);
  }
  __syncthreads();
  const uint32_t c = h[threadIdx.x];
  if (c) atomicAdd(&hist[threadIdx.x], c);
}

// Fixes the digit at `shift` (256 threads, one per digit) and clears the
// histogram for the next pass.
__global__ __launch_bounds__(256) void k_le_pick(Ctl *ctl, uint32_t *hist,
                                                 int shift) {
  __shared__ int64_t wsum[256 / kWave];
  __shared__ int64_t tot;
  const bool live = ctl->sel_mode == 2;
  const int64_t c = live ? (int64_t)hist[threadIdx.x] : 0;
  hist[threadIdx.x] = 0;
  const int64_t excl = block_excl_scan<256>(c, wsum, &tot);
  if (!live) return;
  const int64_t r = ctl->sel_rank;
  __syncthreads();
  if (c > 0 && excl <= r && r < excl + c) {
    ctl->sel_rank = r - excl;
    ctl->sel_prefix |= (uint64_t)threadIdx.x << shift;
    ctl->sel_mask |= (uint64_t)0xff << shift;
  }
}

// Affinity of every slot; loss and gradient of every sampled pair.
template <bool VEC4>
__global__ __launch_bounds__(kLeNT) void k_le_edges(
    const float *__restrict__ emb, int32_t n, int32_t d,
    const int32_t *__restrict__ nbr, int32_t k,
    const uint8_t *__restrict__ status, const uint32_t *__restrict__ word,
    float tau, const Ctl *sel, float *__restrict__ affinity,
    float *__restrict__ grad, uint8_t *__restrict__ sampled, Ctl *ctl) {
  __shared__ double sh[kLeNT / kWave];
  const int64_t ns = (int64_t)n * k;
  const int mode = sel->sel_mode;
  const uint64_t thr = sel->sel_prefix;
  const float inv_tau = 1.0f / tau;
  double lsum = 0.0;
  for (int64_t s = blockIdx.x * (int64_t)kLeNT + threadIdx.x; s < ns;
       s += (int64_t)gridDim.x * kLeNT) {
    const int32_t q = nbr[s];
    const uint8_t v = status[s];
    const bool take =
        v == kSlotInter ||
        (v == kSlotIntra && (mode == 1 || (mode == 2 && draw_key(word, s) <= thr)));
    if (sampled) sampled[s] = take ? 1 : 0;
    // ids outside [-1, n) were reported by k_le_classify; no read for them
    if (!take && !(affinity && q >= 0 && q < n)) {
      if (affinity) affinity[s] = 0.0f;
      continue;
    }
    const int32_t p = (int32_t)(s / k);
    const float *ep = emb + (int64_t)p * d;
    const float *eq = emb + (int64_t)q * d;
    float acc = 0.0f;
    if (VEC4) {
      for (int32_t i = 0; i < d; i += 4) {
        const float4 a = *reinterpret_cast<const float4 *>(ep + i);
        const float4 b = *reinterpret_cast<const float4 *>(eq + i);
        const float x = a.x - b.x, y = a.y - b.y, z = a.z - b.z, w = a.w - b.w;
        acc += x * x + y * y + z * z + w * w;
      }
    } else {
      for (int32_t i = 0; i < d; ++i) {
        const float x = ep[i] - eq[i];
        acc += x * x;
      }
    }
    const float dist = sqrtf(acc);
    const float x = dist * inv_tau;
    if (affinity) affinity[s] = expf(-x);
    if (!take) continue;
    float term, coef;
    if (v == kSlotIntra) {
      term = x;
      coef = dist > 0.0f ? inv_tau / dist : 0.0f;
    } else {
      term = -logf(-expm1f(-x));
      coef = dist > 0.0f ? -inv_tau / (expm1f(x) * dist) : 0.0f;
    }
    lsum += (double)term;
    if (grad && coef != 0.0f) {
      float *gp = grad + (int64_t)p * d;
      float *gq = grad + (int64_t)q * d;
      for (int32_t i = 0; i < d; ++i) {
        const float g = coef * (ep[i] - eq[i]);
        unsafeAtomicAdd(gp + i, g);
        unsafeAtomicAdd(gq + i, -g);
      }
    }
  }
  const double t = block_sum(lsum, sh);
  if (threadIdx.x == 0 && t != 0.0) atomicAdd(&ctl->le_loss, t);
}

__global__ __launch_bounds__(256) void k_fill0(float *x, int64_t count) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    x[i] = 0.0f;
}

unsigned grid_for(int64_t items) {
  const int64_t b = (items + kLeNT - 1) / kLeNT;
  return (unsigned)(b < kLeGrid ? (b < 1 ? 1 : b) : kLeGrid);
}

}  // namespace

void loss_reserve(Arena &a, int32_t n, int32_t k) {
  a.take<uint8_t>((size_t)n * k);
  a.take<uint32_t>(256);
}

int loss_run(const LossArgs &g, LossResult *res, Ctl *ctl, Arena &a,
             hipStream_t st) {
  const int64_t ns = (int64_t)g.n * g.k;
  uint8_t *status = a.take<uint8_t>((size_t)ns);
  uint32_t *hist = a.take<uint32_t>(256);
  Ctl *hc = pinned_ctl();
  if (!hc) {
    set_error("hipHostMalloc of the control block failed");
    return -5;
  }
  prof_begin("edge_loss", st);
  hipLaunchKernelGGL(k_fill0, dim3(1), dim3(256), 0, st,
                     reinterpret_cast<float *>(hist), (int64_t)256);
  if (g.grad)
    hipLaunchKernelGGL(k_fill0, dim3(grid_for((int64_t)g.n * g.d)), dim3(256),
                       0, st, g.grad, (int64_t)g.n * g.d);
  hipLaunchKernelGGL(k_maxabs, dim3(256), dim3(256), 0, st, g.emb,
                     (int64_t)g.n * g.d, ctl);
  hipLaunchKernelGGL(k_le_classify, dim3(grid_for(ns)), dim3(kLeNT), 0, st,
                     g.nbr, g.n, g.k, g.cls, status, ctl);
  hipLaunchKernelGGL(k_le_quota, dim3(1), dim3(64), 0, st, ctl, g.rho);
  for (int shift = 56; shift >= 0; shift -= 8) {
    hipLaunchKernelGGL(k_le_hist, dim3(grid_for(ns)), dim3(kLeNT), 0, st,
                       status, g.word, ns, shift, ctl, hist);
    hipLaunchKernelGGL(k_le_pick, dim3(1), dim3(256), 0, st, ctl, hist, shift);
  }
  const bool vec4 = (g.d % 4) == 0 &&
                    (reinterpret_cast<uintptr_t>(g.emb) & 15) == 0;
  if (vec4)
    hipLaunchKernelGGL(k_le_edges<true>, dim3(grid_for(ns)), dim3(kLeNT), 0,
                       st, g.emb, g.n, g.d, g.nbr, g.k, status, g.word,
                       (float)g.tau, ctl, g.affinity, g.grad, g.sampled, ctl);
  else
    hipLaunchKernelGGL(k_le_edges<false>, dim3(grid_for(ns)), dim3(kLeNT), 0,
                       st, g.emb, g.n, g.d, g.nbr, g.k, status, g.word,
                       (float)g.tau, ctl, g.affinity, g.grad, g.sampled, ctl);
  prof_end(st);
  int rc = read_ctl(ctl, hc, st);
  if (rc) return rc;
  // algorithmic bytes: the table, the words and the classes read once, each
  // pair's two embedding rows, the per-slot outputs and the gradient
  prof_bytes("edge_loss",
             ns * 8.0 + 4.0 * g.n + 8.0 * g.d * (double)hc->le_edges +
                 (g.affinity ? 4.0 * ns : 0.0) + (g.sampled ? 1.0 * ns : 0.0) +
                 (g.grad ? 4.0 * g.n * g.d : 0.0));
  if (hc->err & kErrNonFinite) {
    set_error("non-finite value in emb");
    return -2;
  }
  if (hc->err & kErrBadIndex) {
    set_error("neighbour id outside [-1, n)");
    return -1;
  }
  if (hc->err) {
    set_error("internal check failed in the edge loss (0x%x)", hc->err);
    return -5;
  }
  res->loss = hc->le_loss;
  res->n_edges = (int64_t)hc->le_edges;
  res->n_intra = (int64_t)hc->le_intra;
  res->n_inter = res->n_edges - res->n_intra;
  res->n_intra_kept = (int64_t)hc->le_keep;
  return 0;
}

}  // namespace ezsp
