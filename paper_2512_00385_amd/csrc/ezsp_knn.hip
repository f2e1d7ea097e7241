// ezsp_knn.hip -- exact k-nearest-neighbour adjacency (Sec. 3.1: every point
// linked to its k nearest neighbours; Sec. 4.1: k and unit weights).
//
// Grid build: each point gets a 39-bit Morton key of its 13-bit-per-axis
// voxel in the bounding box (cubic voxels of 1/8191 of the largest extent:
// a 100 m tile gets 1.2 cm voxels, which hold about one point each in the
// test scenes); a radix sort of five 8-bit passes lays the points out in
// Morton order.  Consecutive runs of 16 sorted points form buckets, and an
// implicit 8-ary tree of axis-aligned boxes sits over the buckets, so the
// voxel hierarchy adapts to any density.
//
// Query: one query point per lane, one wavefront per four consecutive
// buckets (64 points).  Each lane keeps its own sorted top-k of 64-bit keys
// (d2 bits, original index) in registers.  A wave scans its own buckets and
// the two next to them in Morton order first, then walks the tree depth
// first; the walk is the wave's, so its state is uniform and runs on the
// scalar unit, with box loads through the scalar cache.  When a node is
// entered, its eight children are tested at once, one child per lane,
// against the box of the wave's own points widened by the wave's largest
// current k-th distance; the children that pass are kept as bits of a
// per-level mask (the lowest set bit is the next to take).  When a child is
// taken, every lane tests its box against its own point and its own current
// k-th distance, and the child is entered (or, for a bucket, scanned) only
// if some lane needs it.  A scanned bucket is loaded by each 16-lane DPP row
// and its points broadcast within the row.  Both box distances are built
// from the same IEEE operations as d2 and rounding is monotone, so neither
// exceeds the d2 of a query and a point inside the box: no neighbour, and no
// tie with a smaller index, can be skipped.
#include "ezsp_internal.h"

namespace ezsp {

__device__ __forceinline__ void bbox_take(float v, int a, float (&mn)[3],
                                          float (&mx)[3], bool &bad) {
  if (!isfinite(v)) {
    bad = true;
  } else {
    mn[a] = fminf(mn[a], v);
    mx[a] = fmaxf(mx[a], v);
  }
}

// Coordinate-wise min / max of the cloud and the non-finite check.  With a
// 16-byte aligned array, a thread takes 4 points at a time as 3 float4
// (x0 y0 z0 x1 | y1 z1 x2 y2 | z2 x3 y3 z3), the last n % 4 points singly.
__global__ __launch_bounds__(256) void k_bbox(const float *xyz, int32_t n,
                                              Ctl *ctl) {
  float mn[3] = {INFINITY, INFINITY, INFINITY};
  float mx[3] = {-INFINITY, -INFINITY, -INFINITY};
  bool bad = false;
  const int32_t tid = blockIdx.x * blockDim.x + threadIdx.x;
  const int32_t stride = gridDim.x * blockDim.x;
  int32_t done = 0;  // points covered by the vector loop
  if ((reinterpret_cast<uintptr_t>(xyz) & 15) == 0) {
    const float4 *v = reinterpret_cast<const float4 *>(xyz);
    const int32_t groups = n / 4;
    // four groups a thread in flight per step; indices past the end are
    // clamped to the last group, whose second reading changes neither a
    // minimum, a maximum nor the finiteness check
    constexpr int kG = 4;
    for (int32_t g0 = tid; g0 < groups; g0 += kG * stride) {
      float4 a[kG], b[kG], c[kG];
#pragma unroll
      for (int e = 0; e < kG; ++e) {
        const int64_t g = min(g0 + e * stride, groups - 1);
        a[e] = v[3 * g];
        b[e] = v[3 * g + 1];
        c[e] = v[3 * g + 2];
      }
#pragma unroll
      for (int e = 0; e < kG; ++e) {
        bbox_take(a[e].x, 0, mn, mx, bad);
        bbox_take(a[e].y, 1, mn, mx, bad);
        bbox_take(a[e].z, 2, mn, mx, bad);
        bbox_take(a[e].w, 0, mn, mx, bad);
        bbox_take(b[e].x, 1, mn, mx, bad);
        bbox_take(b[e].y, 2, mn, mx, bad);
        bbox_take(b[e].z, 0, mn, mx, bad);
        bbox_take(b[e].w, 1, mn, mx, bad);
        bbox_take(c[e].x, 2, mn, mx, bad);
        bbox_take(c[e].y, 0, mn, mx, bad);
        bbox_take(c[e].z, 1, mn, mx, bad);
        bbox_take(c[e].w, 2, mn, mx, bad);
      }
    }
    done = groups * 4;
  }
  for (int32_t i = done + tid; i < n; i += stride) {
#pragma unroll
    for (int a = 0; a < 3; ++a) bbox_take(xyz[3 * (int64_t)i + a], a, mn, mx, bad);
  }
#pragma unroll
  for (int a = 0; a < 3; ++a) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      mn[a] = fminf(mn[a], __shfl_xor(mn[a], off, kWave));
      mx[a] = fmaxf(mx[a], __shfl_xor(mx[a], off, kWave));
    }
  }
  __shared__ float smn[3][256 / kWave], smx[3][256 / kWave];
  __shared__ int sbad;
  const int wid = threadIdx.x / kWave;
  if (threadIdx.x == 0) sbad = 0;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) {
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      smn[a][wid] = mn[a];
      smx[a][wid] = mx[a];
    }
  }
  if (__ballot(bad) && (threadIdx.x & (kWave - 1)) == 0) sbad = 1;
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      float lo = smn[a][0], hi = smx[a][0];
      for (int q = 1; q < 256 / kWave; ++q) {
        lo = fminf(lo, smn[a][q]);
        hi = fmaxf(hi, smx[a][q]);
      }
      // striped: device-scope atomics on one address are serialised at the
      // memory side (256 blocks x 6 of them took most of this kernel)
      atomicMin(&ctl->bbox_s[a][blockIdx.x % kStripes].v, f2ord(lo));
      atomicMax(&ctl->bbox_s[3 + a][blockIdx.x % kStripes].v, f2ord(hi));
    }
    if (sbad) raise_err(ctl, kErrNonFinite);
  }
}

// The box from its stripes, one wave: bbox_enc = min / max over them.
__global__ __launch_bounds__(64) void k_bbox_fold(Ctl *ctl) {
  const int lane = threadIdx.x;
#pragma unroll
  for (int a = 0; a < 6; ++a) {
    int32_t v = lane < kStripes ? ctl->bbox_s[a][lane].v
                                : f2ord(a < 3 ? INFINITY : -INFINITY);
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      const int32_t o = __shfl_xor(v, off, kWave);
      v = a < 3 ? min(v, o) : max(v, o);
    }
    if (lane == 0) ctl->bbox_enc[a] = v;
  }
}

constexpr int kMortonBits = 13;  // per axis
constexpr float kMortonMax = (float)((1 << kMortonBits) - 1);

// 16 bits -> every third bit of 48 (only the low kMortonBits are set).
__device__ __forceinline__ uint64_t spread3(uint32_t v) {
  uint64_t x = v & 0xffffu;
  x = (x | (x << 16)) & 0x0000ff0000ffull;
  x = (x | (x << 8)) & 0x00f00f00f00full;
  x = (x | (x << 4)) & 0x0c30c30c30c3ull;
  x = (x | (x << 2)) & 0x249249249249ull;
  return x;
}

// The point's index either goes to vals, or (vals null, n <= 2^kPackBits)
// into the key's low kPackBits bits below the code, so that a key-only sort
// of the code bits carries it.
constexpr int kPackBits = 25;
__global__ __launch_bounds__(256) void k_morton(const float *xyz, int32_t n,
                                                const Ctl *ctl, uint64_t *keys,
                                                uint32_t *vals) {
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float lo[3], ext = 0.0f;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    lo[a] = ord2f(ctl->bbox_enc[a]);
    ext = fmaxf(ext, ord2f(ctl->bbox_enc[3 + a]) - lo[a]);
  }
  const float scale = (ext > 0.0f) ? kMortonMax / ext : 0.0f;
  uint32_t q[3];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    float t = (xyz[3 * (int64_t)i + a] - lo[a]) * scale;
    t = fminf(fmaxf(t, 0.0f), kMortonMax);  // NaN maps to 0
    q[a] = (uint32_t)t;
  }
  const uint64_t code =
      spread3(q[0]) | (spread3(q[1]) << 1) | (spread3(q[2]) << 2);
  if (vals) {
    keys[i] = code;
    vals[i] = (uint32_t)i;
  } else {
    keys[i] = (code << kPackBits) | (uint64_t)i;
  }
}

// Min and max along each 16-lane DPP row (a bucket of points): after the
// four shifted steps lane 15 of the row holds the row's value (lanes whose
// source is outside the row keep their own value).
__device__ __forceinline__ float row_min15(float v) {
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x111, 0xF, 0xF, false)));
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x112, 0xF, 0xF, false)));
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x114, 0xF, 0xF, false)));
  v = fminf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x118, 0xF, 0xF, false)));
  return v;
}
__device__ __forceinline__ float row_max15(float v) {
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x111, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x112, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x114, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(
                   __float_as_int(v), __float_as_int(v), 0x118, 0xF, 0xF, false)));
  return v;
}

__device__ __forceinline__ void box_join(float4 &lo, float4 &hi,
                                         const float4 &a, const float4 &b) {
  lo.x = fminf(lo.x, a.x);
  lo.y = fminf(lo.y, a.y);
  lo.z = fminf(lo.z, a.z);
  hi.x = fmaxf(hi.x, b.x);
  hi.y = fmaxf(hi.y, b.y);
  hi.z = fmaxf(hi.z, b.z);
}

// Sorted points as float4 (x, y, z, original index bits) plus both maps;
// the array runs to a whole number of buckets.  The same pass builds the
// tree's two lowest levels: each bucket's box (16 consecutive points, one
// DPP row) and the box of every 8 buckets (16 buckets per block).
__global__ __launch_bounds__(256) void k_gather_points(
    const float *xyz, int32_t n, const uint32_t *order,
    const uint64_t *packed, float4 *pts, int32_t *perm, int32_t *inv,
    float4 *blo, float4 *bhi, Tree tree, Ctl *ctl) {
  __shared__ float4 s_lo[256 / kBucket], s_hi[256 / kBucket];
  const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  // points past the end (the last bucket's missing ones) are infinitely
  // far, with an index above every real one, so a bucket scan needs no
  // bounds check; they take no part in the boxes
  float4 p = make_float4(INFINITY, INFINITY, INFINITY,
                         __int_as_float(kPadIndex));
  bool real = false;
  if (i < n) {
    const uint32_t o =
        packed ? (uint32_t)(packed[i] & ((1ull << kPackBits) - 1)) : order[i];
    if (o >= (uint32_t)n) {
      raise_err(ctl, kErrInternal);
    } else {
      const float *q = xyz + 3 * (int64_t)o;
      p = make_float4(q[0], q[1], q[2], __int_as_float((int32_t)o));
      perm[i] = (int32_t)o;
      inv[o] = i;
      real = true;
    }
  }
  if (i < pad_bucket(n)) pts[i] = p;
  float4 lo = real ? p : make_float4(INFINITY, INFINITY, INFINITY, 0.f);
  float4 hi = real ? p : make_float4(-INFINITY, -INFINITY, -INFINITY, 0.f);
  lo.x = row_min15(lo.x);
  lo.y = row_min15(lo.y);
  lo.z = row_min15(lo.z);
  hi.x = row_max15(hi.x);
  hi.y = row_max15(hi.y);
  hi.z = row_max15(hi.z);
  lo.w = hi.w = 0.f;
  const int32_t nb0 = tree.cnt[0];
  const int32_t b = i / kBucket;
  if ((threadIdx.x & (kBucket - 1)) == kBucket - 1) {
    s_lo[threadIdx.x / kBucket] = lo;
    s_hi[threadIdx.x / kBucket] = hi;
    if (b < nb0) {
      blo[b] = lo;
      bhi[b] = hi;
    }
  }
  __syncthreads();
  constexpr int kPer = 256 / kBucket / kFan;  // level-1 nodes per block
  if (tree.top >= 1 && threadIdx.x < kPer) {
    const int32_t j = blockIdx.x * kPer + (int32_t)threadIdx.x;
    if (j < tree.cnt[1]) {
      float4 l1 = make_float4(INFINITY, INFINITY, INFINITY, 0.f);
      float4 h1 = make_float4(-INFINITY, -INFINITY, -INFINITY, 0.f);
      for (int c = 0; c < kFan; ++c)
        if (j * kFan + c < nb0)
          box_join(l1, h1, s_lo[threadIdx.x * kFan + c],
                   s_hi[threadIdx.x * kFan + c]);
      blo[tree.off[1] + j] = l1;
      bhi[tree.off[1] + j] = h1;
    }
  }
}

__global__ __launch_bounds__(256) void k_up_boxes(float4 *blo, float4 *bhi,
                                                  int32_t child_off,
                                                  int32_t child_cnt,
                                                  int32_t off, int32_t cnt) {
  const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= cnt) return;
  const int32_t s = j * kFan;
  const int32_t e = min(child_cnt, s + kFan);
  float4 lo = make_float4(INFINITY, INFINITY, INFINITY, 0.f);
  float4 hi = make_float4(-INFINITY, -INFINITY, -INFINITY, 0.f);
  for (int32_t c = s; c < e; ++c)
    box_join(lo, hi, blo[child_off + c], bhi[child_off + c]);
  blo[off + j] = lo;
  bhi[off + j] = hi;
}

// Levels l0 .. top in one block, a barrier between levels (the upper
// levels are small: a launch per level would cost more than its work).
__global__ __launch_bounds__(1024) void k_top_boxes(float4 *blo, float4 *bhi,
                                                    Tree tree, int l0) {
  for (int l = l0; l <= tree.top; ++l) {
    const int32_t cnt = tree.cnt[l], child_cnt = tree.cnt[l - 1];
    for (int32_t j = threadIdx.x; j < cnt; j += blockDim.x) {
      const int32_t s = j * kFan;
      const int32_t e = min(child_cnt, s + kFan);
      float4 lo = make_float4(INFINITY, INFINITY, INFINITY, 0.f);
      float4 hi = make_float4(-INFINITY, -INFINITY, -INFINITY, 0.f);
      for (int32_t c = s; c < e; ++c)
        box_join(lo, hi, blo[tree.off[l - 1] + c], bhi[tree.off[l - 1] + c]);
      blo[tree.off[l] + j] = lo;
      bhi[tree.off[l] + j] = hi;
    }
    __threadfence_block();
    __syncthreads();
  }
}

// A candidate is the 64-bit key (fp32 bits of d2) << 32 | original index.
// d2 >= 0, so the bits of d2 are ordered like d2 and the key order is the
// order (d2, index).  An empty slot of the output holds ~0 (kNoKey); the
// lists being built use kEmpty instead, the largest finite fp64 pattern:
// above every real key (d2 bits <= 0x7f800000 for the padding's infinity),
// its upper half above every d2 (so it admits every box) and its lower
// half above every index.
constexpr uint64_t kNoKey = ~0ull;
constexpr uint64_t kEmpty = 0x7fefffffffffffffull;

__device__ __forceinline__ uint64_t cand_key(float d2, int32_t o) {
  return ((uint64_t)__float_as_uint(d2) << 32) | (uint32_t)o;
}

// A key read as an fp64 value: its sign bit is clear and its exponent
// field below 0x7ff (at most kEmpty), so it is a non-negative finite number
// (denormal when d2 < 2^-126) and the fp64 order is the integer order.
// v_min_f64 / v_max_f64 then return the bits of the smaller / larger key
// (fp64 denormals are kept in these kernels, and no key is a NaN).  They
// are written out because the compiler's fmin / fmax first quiet each
// operand with a further instruction, which no key needs.
__device__ __forceinline__ uint64_t key_min(uint64_t a, uint64_t b) {
  uint64_t r;
  asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ uint64_t key_max(uint64_t a, uint64_t b) {
  uint64_t r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Insert nk into the sorted top-K (a no-op when nk is not below the last
// entry): the new entry t is min(key[t], max(key[t-1], nk)), which keeps
// key[t] when nk >= key[t], takes nk when key[t-1] <= nk < key[t], and
// shifts key[t-1] up when nk < key[t-1].
template <int K>
__device__ __forceinline__ void topk_insert(uint64_t (&key)[K], uint64_t nk) {
#pragma unroll
  for (int t = K - 1; t > 0; --t) key[t] = key_min(key[t], key_max(key[t - 1], nk));
  key[0] = key_min(key[0], nk);
}

// Broadcast lane J of every 16-lane row (one DPP row = one query group).
template <int J>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(
      0, __float_as_int(v), 0x150 + J, 0xF, 0xF, false));
}
template <int J>
__device__ __forceinline__ int32_t row_bcast_i(int32_t v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x150 + J, 0xF, 0xF, true);
}

// Key of candidate J of the bucket held one point per lane in q: d2 in the
// fixed order fma(dz, dz, fma(dy, dy, dx*dx)), dx = x_q - x_p.  Only the
// query's own bucket can hold the query itself (SELF), which gives kNoKey.
// Padding points past the end give an infinite d2 and an index above every
// real one, so they never displace a real point.
template <int J, bool SELF>
__device__ __forceinline__ uint64_t bucket_key(const float4 &q, float px,
                                               float py, float pz,
                                               int32_t me) {
  const float dx = row_bcast<J>(q.x) - px;
  const float dy = row_bcast<J>(q.y) - py;
  const float dz = row_bcast<J>(q.z) - pz;
  const int32_t qo = row_bcast_i<J>(__float_as_int(q.w));
  const float d2 = fmaf(dz, dz, fmaf(dy, dy, dx * dx));
  if (SELF) return qo != me ? cand_key(d2, qo) : kEmpty;
  return cand_key(d2, qo);
}

template <int K, int J, bool SELF>
struct BucketStep {
  __device__ __forceinline__ static void run(const float4 &q, float px,
                                             float py, float pz, int32_t me,
                                             uint64_t (&key)[K]) {
    const uint64_t nk = bucket_key<J, SELF>(q, px, py, pz, me);
    if (nk < key[K - 1]) topk_insert<K>(key, nk);
    BucketStep<K, J + 1, SELF>::run(q, px, py, pz, me, key);
  }
};
template <int K, bool SELF>
struct BucketStep<K, kBucket, SELF> {
  __device__ __forceinline__ static void run(const float4 &, float, float,
                                             float, int32_t,
                                             uint64_t (&)[K]) {}
};

// All 16 lanes of a group scan bucket b together (group-uniform call); the
// points array is padded to whole buckets.  Lanes of an inactive query
// (me = -1) carry keys too, they are not written.
template <int K, bool SELF>
__device__ __forceinline__ void scan_bucket(const float4 *__restrict__ pts,
                                            int32_t b, int lane16, float px,
                                            float py, float pz, int32_t me,
                                            uint64_t (&key)[K]) {
  const float4 q = pts[b * kBucket + lane16];
  BucketStep<K, 0, SELF>::run(q, px, py, pz, me, key);
}

// Largest k-th d2 (as bits) over the active lanes of the wave, the same
// value in every lane: a prefix max along each 16-lane DPP row, then the
// four rows' last lanes.  An empty list (kEmpty) gives 0x7fefffff, above
// every d2's bits, which admits every box.
__device__ __forceinline__ uint32_t wave_max_kth(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF,
                                                   false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF,
                                                   false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF,
                                                   false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF,
                                                   false));
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 47);
  const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
  return max(max(r0, r1), max(r2, r3));
}

// Squared distance from point p to box [lo, hi], from the same IEEE
// operations as d2 (per axis the gap max(lo - p, p - hi, 0)); it never
// exceeds the d2 of p and a point inside the box.
__device__ __forceinline__ float box_d2(const float4 &lo, const float4 &hi,
                                        float px, float py, float pz) {
  const float ex = fmaxf(fmaxf(lo.x - px, px - hi.x), 0.f);
  const float ey = fmaxf(fmaxf(lo.y - py, py - hi.y), 0.f);
  const float ez = fmaxf(fmaxf(lo.z - pz, pz - hi.z), 0.f);
  return fmaf(ez, ez, fmaf(ey, ey, ex * ex));
}

// Coarse test of the children first .. first+7 (level lc) of one node,
// one child per lane (lane c and every lane c mod 8 take child c): bit c is
// set when the child's box is within the wave's largest k-th distance of
// the box of the wave's own points (qlo, qhi).  Per axis the gap to the
// query box is at most the gap to any query point in it (same IEEE
// operations, rounding is monotone), so a child that some lane's own test
// would admit is always admitted here.
__device__ __forceinline__ uint32_t coarse_mask(
    const float4 *__restrict__ blo, const float4 *__restrict__ bhi,
    int32_t lv_off, int32_t lv_cnt, int32_t first, const float4 &qlo,
    const float4 &qhi, uint32_t gkth, int lane) {
  const int32_t nchild = min(kFan, lv_cnt - first);
  const int c = lane & (kFan - 1);
  const int32_t j = lv_off + first + min(c, nchild - 1);
  const float4 lo = blo[j], hi = bhi[j];
  const float ex = fmaxf(fmaxf(lo.x - qhi.x, qlo.x - hi.x), 0.f);
  const float ey = fmaxf(fmaxf(lo.y - qhi.y, qlo.y - hi.y), 0.f);
  const float ez = fmaxf(fmaxf(lo.z - qhi.z, qlo.z - hi.z), 0.f);
  const float d2b = fmaf(ez, ez, fmaf(ey, ey, ex * ex));
  const bool need = c < nchild && __float_as_uint(d2b) <= gkth;
  return (uint32_t)__ballot(need) & 0xffu;
}

__device__ __forceinline__ void set_level_bits(uint64_t &mlo, uint64_t &mhi,
                                               int l, uint32_t m8) {
  if (l < 8)
    mlo |= (uint64_t)m8 << (8 * l);
  else
    mhi |= (uint64_t)m8 << (8 * (l - 8));
}

// One query group = one wavefront = the 64 points of four consecutive
// buckets, one query per lane.  The walk is the wave's own, so its state
// (pending children, path, bucket to scan) is uniform and lives in scalar
// registers; only the distance tests and the bucket scans are per lane.
// The wave scans its own buckets and the two next to them in Morton order
// first.  A node is entered when some lane's box distance does not exceed
// that lane's current k-th distance.  ST: also count, per wave, the
// buckets it scans (its own included) and the inner nodes it enters
// (st_scan, st_node; the walk statistics, a separate instantiation).
template <int K, bool ST = false>
__global__ __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(8, 8))) void k_knn_query(
    const float4 *__restrict__ pts, const int32_t *__restrict__ inv,
    int32_t n, const float4 *__restrict__ blo, const float4 *__restrict__ bhi,
    Tree tree, int32_t k, int32_t *__restrict__ nbr_int,
    int32_t *__restrict__ nbr_out, float *__restrict__ d2_out,
    uint64_t *__restrict__ kth_out, int32_t n_waves,
    const float4 *__restrict__ emb, int32_t d4, float4 *__restrict__ emb_out,
    Ctl *ctl, int32_t *__restrict__ st_scan, int32_t *__restrict__ st_node) {
  constexpr int kOwn = kWave / kBucket;  // buckets per wave
  const int32_t wv = __builtin_amdgcn_readfirstlane(
      xcd_block() * (256 / kWave) + (int32_t)(threadIdx.x / kWave));
  if (wv >= n_waves) return;  // whole waves only
  const int lane = threadIdx.x & (kWave - 1);
  const int lane16 = lane & (kBucket - 1);
  const int32_t nb0 = tree.cnt[0];
  const int32_t b0 = wv * kOwn;               // first own bucket
  const int32_t nown = min(kOwn, nb0 - b0);   // 1 .. 4
  const int32_t i = b0 * kBucket + lane;
  const bool act = i < n;
  const float4 p = act ? pts[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  const int32_t me = act ? __float_as_int(p.w) : -1;
  // For the merge, optionally: the point's embedding row (d4 <= 4 float4)
  // copied into internal order, with Step 0's max |e| and the non-finite
  // check.  The loads are issued here and the stores made after the own
  // buckets' scans, whose instructions cover their latency.
  float4 row[4];
  if (emb && act) {
    const float4 *src = emb + (int64_t)me * d4;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < d4) row[q] = src[q];
  }
  uint64_t key[K];
#pragma unroll
  for (int t = 0; t < K; ++t) key[t] = kEmpty;
  // own buckets first: a tight k-th distance early (the two Morton
  // neighbours are the first buckets of the scan loop below)
  for (int32_t j = 0; j < nown; ++j)
    scan_bucket<K, true>(pts, b0 + j, lane16, p.x, p.y, p.z, me, key);
  int32_t c_scan = nown, c_node = 0;  // walk statistics (ST only)
  if (emb) {  // every lane of the wave is here
    uint32_t m = 0;
    bool bad = false;
    if (act) {
      float4 *dst = emb_out + (int64_t)i * d4;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (q >= d4) break;
        dst[q] = row[q];
        const float v[4] = {row[q].x, row[q].y, row[q].z, row[q].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (!isfinite(v[j])) bad = true;
          else m = max(m, __float_as_uint(fabsf(v[j])));
        }
      }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1)
      m = max(m, (uint32_t)__shfl_xor((int)m, off, kWave));
    const bool any_bad = __ballot(bad) != 0;
    if (lane == 0) {
      stripe_max(ctl->maxabs_s, (int32_t)m);  // |e| bits < 2^31
      if (any_bad) raise_err(ctl, kErrNonFinite);
    }
  }

  // Depth-first walk with the pending children of every level of the
  // current path as bits: bit 8*l + c = child c (level l) of the path node
  // at level l+1.  The lowest set bit is the deepest pending node, and the
  // path node at level l+1 is cur >> 3*(l+1-curl) (cur: last node taken, at
  // level curl), since children of x are 8x..8x+7.  Children are marked by
  // the wave's coarse test when their parent is entered; a node is entered
  // only when, as it is taken, some lane's own test against its current
  // k-th distance still needs it.
  float4 qlo = blo[b0], qhi = bhi[b0];  // the own buckets' box
  for (int32_t j = 1; j < nown; ++j) {
    const float4 lo = blo[b0 + j], hi = bhi[b0 + j];
    qlo.x = fminf(qlo.x, lo.x);
    qlo.y = fminf(qlo.y, lo.y);
    qlo.z = fminf(qlo.z, lo.z);
    qhi.x = fmaxf(qhi.x, hi.x);
    qhi.y = fmaxf(qhi.y, hi.y);
    qhi.z = fmaxf(qhi.z, hi.z);
  }
  uint64_t mlo = 0, mhi = 0;
  int32_t cur = 0;
  int curl = tree.top;
  // the wave's largest k-th distance changes only in a bucket scan
  uint32_t gk = wave_max_kth(act ? (uint32_t)(key[K - 1] >> 32) : 0u);
  if (tree.top > 0) {
    const uint32_t m8 =
        coarse_mask(blo, bhi, tree.off[tree.top - 1], tree.cnt[tree.top - 1],
                    0, qlo, qhi, gk, lane);
    set_level_bits(mlo, mhi, tree.top - 1, m8);
  }
  int pre = 0;  // Morton neighbours taken: b0 - 1, then b0 + nown
  for (;;) {
    int32_t leaf = -1;
    while (pre < 2 && leaf < 0) {
      const int32_t b = pre == 0 ? b0 - 1 : b0 + nown;
      ++pre;
      if (b >= 0 && b < nb0) leaf = b;
    }
    while (leaf < 0) {
      int t;
      if (mlo != 0) {
        t = __builtin_ctzll(mlo);
        mlo &= mlo - 1;
      } else {
        // levels 8 and up (trees over more than 8^8 buckets only)
        if (mhi == 0) break;
        t = 64 + __builtin_ctzll(mhi);
        mhi &= mhi - 1;
      }
      const int l = t >> 3, c = t & 7;
      const int32_t node = ((cur >> (3 * (l + 1 - curl))) << 3) | c;
      cur = node;
      curl = l;
      if (l == 0 && node >= b0 - 1 && node <= b0 + nown) continue;
      const int32_t j = tree.off[l] + node;
      const uint32_t kth = (uint32_t)(key[K - 1] >> 32);
      const float d2b = box_d2(blo[j], bhi[j], p.x, p.y, p.z);
      if (__ballot(act && __float_as_uint(d2b) <= kth) == 0) continue;
      if (l == 0) {
        leaf = node;
        break;
      }
      const uint32_t m8 = coarse_mask(blo, bhi, tree.off[l - 1],
                                      tree.cnt[l - 1], node * kFan, qlo, qhi,
                                      gk, lane);
      set_level_bits(mlo, mhi, l - 1, m8);
      if constexpr (ST) ++c_node;
    }
    if (leaf < 0) break;
    scan_bucket<K, false>(pts, leaf, lane16, p.x, p.y, p.z, me, key);
    gk = wave_max_kth(act ? (uint32_t)(key[K - 1] >> 32) : 0u);
    if constexpr (ST) ++c_scan;
  }
  if constexpr (ST) {
    if (lane == 0) {  // the walk is uniform over the wave
      st_scan[wv] = c_scan;
      st_node[wv] = c_node;
    }
  }

  if (!act) return;
  const int32_t kp = pad4(k);
  // the k-th key (kNoKey when fewer than k points exist): later, q is among
  // p's neighbours exactly when q's key as seen from p does not exceed it.
  // Empty slots and padding points carry an index >= n.
#pragma unroll
  for (int t = 0; t < K; ++t)
    if (t == k - 1) kth_out[i] = (uint32_t)key[t] < (uint32_t)n ? key[t] : kNoKey;
#pragma unroll
  for (int t = 0; t < K; ++t) {
    if (t < k) {
      const bool has = (uint32_t)key[t] < (uint32_t)n;
      const int32_t o = (int32_t)(uint32_t)key[t];
      nbr_int[(int64_t)i * kp + t] = has ? inv[o] : -1;
      if (nbr_out) nbr_out[(int64_t)me * k + t] = has ? o : -1;
      if (d2_out)
        d2_out[(int64_t)me * k + t] =
            has ? __uint_as_float((uint32_t)(key[t] >> 32)) : INFINITY;
    }
  }
  for (int32_t t = k; t < kp; ++t) nbr_int[(int64_t)i * kp + t] = -1;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static int knn_template_k(int32_t k) {
  static const int ks[] = {4, 8, 10, 16, 32, 64};
  for (int v : ks)
    if (k <= v) return v;
  return -1;
}

void knn_reserve(Arena &a, int32_t n, int32_t k, KnnWork *w) {
  const Tree t = make_tree(n);
  w->perm = a.take<int32_t>(n);
  w->inv = a.take<int32_t>(n);
  w->nbr_int = a.take<int32_t>((size_t)n * pad4(k));
  w->keys = a.take<uint64_t>(n);
  w->keys2 = a.take<uint64_t>(n);
  w->vals = a.take<uint32_t>(n);
  w->vals2 = a.take<uint32_t>(n);
  w->pts = a.take<float4>(pad_bucket(n));
  w->kth = a.take<uint64_t>(n);
  w->blo = a.take<float4>(t.total);
  w->bhi = a.take<float4>(t.total);
  w->hist = a.take<int32_t>(radix_hist_ints(n));
  w->bsum = a.take<int32_t>(scan_blocks(radix_hist_ints(n)) + 1);
  w->total = a.take<int32_t>(4);
}

// the largest level left to the single-block kernel
constexpr int32_t kTopBoxes = 512;

static hipError_t knn_impl(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                           const KnnWork &s, int32_t *nbr_out, float *d2_out,
                           const float *emb, int32_t d, float *emb_out,
                           int32_t *st_scan, int32_t *st_node,
                           hipStream_t st) {
  const KnnWork &w = s;
  const Tree tree = make_tree(n);
  const int nt = 256;
  const int gb = (n + nt - 1) / nt;
  hipLaunchKernelGGL(k_bbox, dim3(min(gb, 256)), dim3(nt), 0, st, xyz, n,
                     ctl);
  hipLaunchKernelGGL(k_bbox_fold, dim3(1), dim3(64), 0, st, ctl);
  // the index packed under the code when it fits in 64 bits: the sort then
  // moves 8 bytes a key instead of 12
  const bool pack = n <= (1 << kPackBits);
  static_assert(3 * kMortonBits + kPackBits <= 64, "code and index in a key");
  hipLaunchKernelGGL(k_morton, dim3(gb), dim3(nt), 0, st, xyz, n, ctl, s.keys,
                     pack ? (uint32_t *)nullptr : s.vals);
  prof_begin("morton_sort", st);
  const bool alt =
      pack ? radix_sort_keys(s.keys, s.keys2, n, kPackBits, 3 * kMortonBits,
                             s.hist, s.bsum, s.total, ctl, st)
           : radix_sort_pairs(s.keys, s.vals, s.keys2, s.vals2, n,
                              3 * kMortonBits, s.hist, s.bsum, s.total, ctl,
                              st);
  prof_end(st);
  const uint32_t *order = pack ? nullptr : (alt ? s.vals2 : s.vals);
  const uint64_t *packed = pack ? (alt ? s.keys2 : s.keys) : nullptr;
  // points in Morton order with the two lowest box levels, then a launch
  // per level while a level is large, the rest in one block
  hipLaunchKernelGGL(k_gather_points, dim3(gb), dim3(nt), 0, st, xyz, n, order,
                     packed, s.pts, w.perm, w.inv, s.blo, s.bhi, tree, ctl);
  int l = 2;
  for (; l <= tree.top && tree.cnt[l] > kTopBoxes; ++l)
    hipLaunchKernelGGL(k_up_boxes, dim3((tree.cnt[l] + nt - 1) / nt), dim3(nt),
                       0, st, s.blo, s.bhi, tree.off[l - 1], tree.cnt[l - 1],
                       tree.off[l], tree.cnt[l]);
  if (l <= tree.top)
    hipLaunchKernelGGL(k_top_boxes, dim3(1), dim3(1024), 0, st, s.blo, s.bhi,
                       tree, l);
  // a wave per four buckets, four waves per block
  constexpr int kOwn = kWave / kBucket;
  const int32_t n_waves = (tree.cnt[0] + kOwn - 1) / kOwn;
  const int32_t qblocks = (n_waves + (nt / kWave) - 1) / (nt / kWave);
  const dim3 grid(xcd_grid(qblocks));
  const float4 *emb4 = reinterpret_cast<const float4 *>(emb);
  float4 *emb_out4 = reinterpret_cast<float4 *>(emb_out);
  prof_begin("knn_query", st);
  switch (knn_template_k(k)) {
#define EZSP_KNN_CASE(KK)                                                    \
  case KK:                                                                   \
    if (st_scan)                                                             \
      hipLaunchKernelGGL((k_knn_query<KK, true>), grid, dim3(nt), 0, st,     \
                         s.pts, w.inv, n, s.blo, s.bhi, tree, k, w.nbr_int,  \
                         nbr_out, d2_out, w.kth, n_waves, emb4, d / 4,       \
                         emb_out4, ctl, st_scan, st_node);                   \
    else                                                                     \
      hipLaunchKernelGGL(k_knn_query<KK>, grid, dim3(nt), 0, st, s.pts,      \
                         w.inv, n, s.blo, s.bhi, tree, k, w.nbr_int,         \
                         nbr_out, d2_out, w.kth, n_waves, emb4, d / 4,       \
                         emb_out4, ctl, (int32_t *)nullptr,                  \
                         (int32_t *)nullptr);                                \
    break;
    EZSP_KNN_CASE(4)
    EZSP_KNN_CASE(8)
    EZSP_KNN_CASE(10)
    EZSP_KNN_CASE(16)
    EZSP_KNN_CASE(32)
    EZSP_KNN_CASE(64)
#undef EZSP_KNN_CASE
    default:
      prof_end(st);
      return hipErrorInvalidValue;
  }
  prof_end(st);
  // algorithmic bytes: read xyz, write the n*k neighbour table (the
  // embedding copy is a reordering for the merge, not counted)
  prof_bytes("knn_query", (12.0 + 4.0 * k) * n);
  return hipGetLastError();
}

hipError_t knn_launch(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                      const KnnWork &s, int32_t *nbr_out, float *d2_out,
                      hipStream_t st) {
  return knn_impl(xyz, n, k, ctl, s, nbr_out, d2_out, nullptr, 0, nullptr,
                  nullptr, nullptr, st);
}

hipError_t knn_launch_stats(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                            const KnnWork &s, int32_t *nbr_out,
                            int32_t *st_scan, int32_t *st_node,
                            hipStream_t st) {
  return knn_impl(xyz, n, k, ctl, s, nbr_out, nullptr, nullptr, 0, nullptr,
                  st_scan, st_node, st);
}

hipError_t knn_launch_emb(const float *xyz, int32_t n, int32_t k, Ctl *ctl,
                          const KnnWork &s, const float *emb, int32_t d,
                          float *emb_out, hipStream_t st) {
  if (d % 4 != 0 || d > 16 || (reinterpret_cast<uintptr_t>(emb) & 15) != 0 ||
      (reinterpret_cast<uintptr_t>(emb_out) & 15) != 0)
    return hipErrorInvalidValue;
  return knn_impl(xyz, n, k, ctl, s, nullptr, nullptr, emb, d, emb_out,
                  nullptr, nullptr, st);
}

}  // namespace ezsp
