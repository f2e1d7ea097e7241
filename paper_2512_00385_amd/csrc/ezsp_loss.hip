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
//
// Layout: a group of G lanes (the power of two >= max(D, k), at most 64) owns
// one row p of the table, lane i holding embedding dimensions i, i + G, ...;
// every e_q gather is then one contiguous segment.  The row accumulates the
// gradient on its own side of every sampled pair it lists in registers; the
// other end q gets its side from its own row when q lists p too (a mutual
// pair), and by atomics from the owner slot otherwise.  A slot's 16-bit
// status carries the pair type, whether it owns the pair, whether the pair is
// mutual, and where row q lists p, so a mirror slot can read the owner's
// random word.
#include "ezsp_internal.h"

namespace ezsp {

namespace {

// Slot status: bits 0-1 pair type, bit 2 owner, bit 3 mutual, bits 8-15
// the position of p in row q (mutual pairs).
enum : uint16_t {
  kSlotNone = 0,
  kSlotInter = 1,
  kSlotIntra = 2,
  kSlotOwner = 4,
  kSlotMutual = 8
};

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
// Position of p in row r (k entries), or -1; rows of 4k ids are read as
// int4 (the table is 16-byte aligned then).
template <bool VEC4>
__device__ __forceinline__ int32_t find_in_row(const int32_t *r, int32_t k,
                                               int32_t p) {
  if (VEC4) {
    const int4 *r4 = reinterpret_cast<const int4 *>(r);
    for (int32_t t = 0; t < k / 4; ++t) {
      const int4 x = r4[t];
      if (x.x == p) return 4 * t;
      if (x.y == p) return 4 * t + 1;
      if (x.z == p) return 4 * t + 2;
      if (x.w == p) return 4 * t + 3;
    }
    return -1;
  }
  for (int32_t t = 0; t < k; ++t)
    if (r[t] == p) return t;
  return -1;
}

template <bool VEC4>
__global__ __launch_bounds__(kLeNT) void k_le_classify(
    const int32_t *__restrict__ nbr, int32_t n, int32_t k,
    const int32_t *__restrict__ cls, uint16_t *__restrict__ status,
    Ctl *ctl) {
  __shared__ unsigned long long sh[kLeNT / kWave];
  const int64_t ns = (int64_t)n * k;
  unsigned long long edges = 0, intra = 0;
  for (int64_t s = blockIdx.x * (int64_t)kLeNT + threadIdx.x; s < ns;
       s += (int64_t)gridDim.x * kLeNT) {
    const int32_t p = (int32_t)(s / k);
    const int32_t j = (int32_t)(s - (int64_t)p * k);
    const int32_t q = nbr[s];
    uint16_t v = kSlotNone;
    if (q < -1 || q >= n) {
      raise_err(ctl, kErrBadIndex);
    } else if (q >= 0 && q != p) {
      bool first = true;  // no earlier slot of row p lists q
      const int32_t *row = nbr + (int64_t)p * k;
      for (int32_t t = 0; t < j && first; ++t) first = row[t] != q;
      if (first) {
        const int32_t jq = find_in_row<VEC4>(nbr + (int64_t)q * k, k, p);
        const bool mutual = jq >= 0;
        const bool owner = p < q || !mutual;
        v = (cls[p] == cls[q]) ? kSlotIntra : kSlotInter;
        if (owner) v |= kSlotOwner;
        if (mutual) v |= kSlotMutual | (uint16_t)(jq << 8);
        if (owner) {
          edges += 1;
          intra += ((v & 3) == kSlotIntra);
        }
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
    const uint16_t *__restrict__ status, const uint32_t *__restrict__ word,
    int64_t ns, int shift, const Ctl *ctl, uint32_t *hist) {
  if (ctl->sel_mode != 2) return;
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t prefix = ctl->sel_prefix, mask = ctl->sel_mask;
  for (int64_t s = blockIdx.x * (int64_t)kLeNT + threadIdx.x; s < ns;
       s += (int64_t)gridDim.x * kLeNT) {
    if ((status[s] & (3 | kSlotOwner)) != (kSlotIntra | kSlotOwner)) continue;
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

// Affinity of every slot; loss and gradient of every sampled pair.  G lanes
// per row (G >= k), NV dimensions per lane (D <= G * NV).  Lane t first reads
// slot t of the row (id and status, one coalesced load), then the group walks
// the slots U at a time, with the U embedding gathers issued together.
constexpr int kLeU = 4;

template <int G, int NV>
__global__ __launch_bounds__(kLeNT) void k_le_rows(
    const float *__restrict__ emb, int32_t n, int32_t d,
    const int32_t *__restrict__ nbr, int32_t k,
    const uint16_t *__restrict__ status, const uint32_t *__restrict__ word,
    float tau, const Ctl *sel, float *__restrict__ affinity,
    float *__restrict__ grad, uint8_t *__restrict__ sampled, Ctl *ctl) {
  __shared__ double sh[kLeNT / kWave];
  constexpr int kRows = kLeNT / G;  // rows per block and step
  const int lane = threadIdx.x & (G - 1);
  const int mode = sel->sel_mode;
  const uint64_t thr = sel->sel_prefix;
  const float inv_tau = 1.0f / tau;
  double lsum = 0.0;
  for (int64_t p = (int64_t)blockIdx.x * kRows + threadIdx.x / G; p < n;
       p += (int64_t)gridDim.x * kRows) {
    const int32_t my_q = lane < k ? nbr[p * k + lane] : -1;
    const int32_t my_st = lane < k ? (int32_t)status[p * k + lane] : 0;
    float ep[NV], acc[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int i = lane + v * G;
      ep[v] = i < d ? emb[p * d + i] : 0.0f;
      acc[v] = 0.0f;
    }
    for (int32_t j0 = 0; j0 < k; j0 += kLeU) {
      int32_t qs[kLeU];
      float eq[kLeU][NV];
#pragma unroll
      for (int u = 0; u < kLeU; ++u) {
        const int32_t q = __shfl(my_q, j0 + u, G);
        qs[u] = (j0 + u < k && q >= 0 && q < n) ? q : -1;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int i = lane + v * G;
          eq[u][v] = (qs[u] >= 0 && i < d) ? emb[(int64_t)qs[u] * d + i] : 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < kLeU; ++u) {
        const int32_t j = j0 + u;
        if (j >= k) break;
        const int64_t s = p * k + j;
        const int32_t q = qs[u];
        const uint16_t st = (uint16_t)__shfl(my_st, j, G);
        if (q < 0) {  // empty slot (bad ids were reported already)
          if (lane == 0) {
            if (affinity) affinity[s] = 0.0f;
            if (sampled) sampled[s] = 0;
          }
          continue;
        }
        float df[NV];
        float part = 0.0f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          df[v] = ep[v] - eq[u][v];
          part += df[v] * df[v];
        }
#pragma unroll
        for (int off = G / 2; off > 0; off >>= 1)
          part += __shfl_xor(part, off, G);
        const float dist = sqrtf(part);
        const float x = dist * inv_tau;
        bool take = false;
        const int type = st & 3;
        if (type == kSlotInter) {
          take = true;
        } else if (type == kSlotIntra) {
          const int64_t os =
              (st & kSlotOwner) ? s : (int64_t)q * k + (st >> 8);
          take = mode == 1 || (mode == 2 && draw_key(word, os) <= thr);
        }
        const bool owner = (st & kSlotOwner) != 0;
        if (lane == 0) {
          if (affinity) affinity[s] = expf(-x);
          if (sampled) sampled[s] = (take && owner) ? 1 : 0;
        }
        if (!take) continue;
        float term, coef;
        if (type == kSlotIntra) {
          term = x;
          coef = dist > 0.0f ? inv_tau / dist : 0.0f;
        } else {
          term = -logf(-expm1f(-x));
          coef = dist > 0.0f ? -inv_tau / (expm1f(x) * dist) : 0.0f;
        }
        if (owner && lane == 0) lsum += (double)term;
        if (grad) {
#pragma unroll
          for (int v = 0; v < NV; ++v) acc[v] += coef * df[v];
          if (!(st & kSlotMutual) && coef != 0.0f) {
            // q does not list p: the owner slot gives q its side
#pragma unroll
            for (int v = 0; v < NV; ++v) {
              const int i = lane + v * G;
              if (i < d)
                unsafeAtomicAdd(grad + (int64_t)q * d + i, -coef * df[v]);
            }
          }
        }
      }
    }
    if (grad) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int i = lane + v * G;
        if (i < d && acc[v] != 0.0f) unsafeAtomicAdd(grad + p * d + i, acc[v]);
      }
    }
  }
  const double t = block_sum(lsum, sh);
  if (threadIdx.x == 0 && t != 0.0) atomicAdd(&ctl->le_loss, t);
}

template <int G, int NV>
void launch_rows(const LossArgs &g, const uint16_t *status, Ctl *ctl,
                 hipStream_t st) {
  constexpr int kRows = kLeNT / G;
  int64_t blocks = ((int64_t)g.n + kRows - 1) / kRows;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL((k_le_rows<G, NV>), dim3((unsigned)blocks), dim3(kLeNT),
                     0, st, g.emb, g.n, g.d, g.nbr, g.k, status, g.word,
                     (float)g.tau, ctl, g.affinity, g.grad, g.sampled, ctl);
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
  a.take<uint16_t>((size_t)n * k);
  a.take<uint32_t>(256);
}

int loss_run(const LossArgs &g, LossResult *res, Ctl *ctl, Arena &a,
             hipStream_t st) {
  const int64_t ns = (int64_t)g.n * g.k;
  uint16_t *status = a.take<uint16_t>((size_t)ns);
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
  hipLaunchKernelGGL(k_maxabs, dim3(2048), dim3(256), 0, st, g.emb,
                     (int64_t)g.n * g.d, ctl);
  if (g.k % 4 == 0 && (reinterpret_cast<uintptr_t>(g.nbr) & 15) == 0)
    hipLaunchKernelGGL(k_le_classify<true>, dim3(grid_for(ns)), dim3(kLeNT),
                       0, st, g.nbr, g.n, g.k, g.cls, status, ctl);
  else
    hipLaunchKernelGGL(k_le_classify<false>, dim3(grid_for(ns)), dim3(kLeNT),
                       0, st, g.nbr, g.n, g.k, g.cls, status, ctl);
  hipLaunchKernelGGL(k_le_quota, dim3(1), dim3(64), 0, st, ctl, g.rho);
  for (int shift = 56; shift >= 0; shift -= 8) {
    hipLaunchKernelGGL(k_le_hist, dim3(grid_for(ns)), dim3(kLeNT), 0, st,
                       status, g.word, ns, shift, ctl, hist);
    hipLaunchKernelGGL(k_le_pick, dim3(1), dim3(256), 0, st, ctl, hist, shift);
  }
  // lanes per row: the power of two covering both D (up to 64) and k
  const int32_t span = g.d < 64 ? (g.d > g.k ? g.d : g.k) : 64;
  if (span <= 4) launch_rows<4, 1>(g, status, ctl, st);
  else if (span <= 8) launch_rows<8, 1>(g, status, ctl, st);
  else if (span <= 16) launch_rows<16, 1>(g, status, ctl, st);
  else if (span <= 32) launch_rows<32, 1>(g, status, ctl, st);
  else if (g.d <= 64) launch_rows<64, 1>(g, status, ctl, st);
  else if (g.d <= 128) launch_rows<64, 2>(g, status, ctl, st);
  else if (g.d <= 256) launch_rows<64, 4>(g, status, ctl, st);
  else if (g.d <= 512) launch_rows<64, 8>(g, status, ctl, st);
  else launch_rows<64, 16>(g, status, ctl, st);
  prof_end(st);
  int rc = read_ctl(ctl, hc, st);
  if (rc) return rc;
  // algorithmic bytes: every input read once (embeddings, table, words,
  // classes) and every output written once
  prof_bytes("edge_loss",
             4.0 * g.n * g.d + 8.0 * ns + 4.0 * g.n +
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
