// ezsp_stats.hip -- per-superpoint size, mean embedding and centroid of a
// labelling (Sec. 3.2: the mean embedding Y_P of a superpoint; App. Alg. A-2,
// component_attributes).  Sums are exact int64 fixed point, so the result
// does not depend on the order in which points are added.
#include "ezsp_internal.h"

namespace ezsp {

__global__ __launch_bounds__(256) void k_cs_zero(int32_t nc, int32_t d,
                                                 bool with_xyz, int64_t *size,
                                                 int64_t *Se, int64_t *Sx) {
  const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nc) return;
  size[c] = 0;
  for (int32_t i = 0; i < d; ++i) Se[(int64_t)c * d + i] = 0;
  if (with_xyz)
    for (int a = 0; a < 3; ++a) Sx[(int64_t)c * 3 + a] = 0;
}

__global__ __launch_bounds__(256) void k_cs_add(
    int32_t n, const int32_t *__restrict__ labels, int32_t nc,
    const float *__restrict__ emb, int32_t d, const float *__restrict__ xyz,
    const Ctl *ce, const Ctl *cx, int64_t *size, int64_t *Se, int64_t *Sx,
    Ctl *ctl) {
  const int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t c = labels[p];
  if ((uint32_t)c >= (uint32_t)nc) {
    raise_err(ctl, kErrBadIndex);
    return;
  }
  atomicAdd(reinterpret_cast<unsigned long long *>(&size[c]), 1ull);
  const double sF = ldexp(1.0, ce->F);
  for (int32_t i = 0; i < d; ++i) {
    const int64_t q = (int64_t)rint((double)emb[(int64_t)p * d + i] * sF);
    atomicAdd(reinterpret_cast<unsigned long long *>(&Se[(int64_t)c * d + i]),
              (unsigned long long)q);
  }
  if (xyz) {
    const double sX = ldexp(1.0, cx->F);
    for (int a = 0; a < 3; ++a) {
      const int64_t q = (int64_t)rint((double)xyz[(int64_t)p * 3 + a] * sX);
      atomicAdd(reinterpret_cast<unsigned long long *>(&Sx[(int64_t)c * 3 + a]),
                (unsigned long long)q);
    }
  }
}

// out = (float)(((double)S / size) * 2^-F), 0 for an empty superpoint.
__global__ __launch_bounds__(256) void k_cs_mean(int32_t nc, int32_t d,
                                                 const int64_t *size,
                                                 const int64_t *S,
                                                 const Ctl *cf, float *out) {
  const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (t >= (int64_t)nc * d) return;
  const int64_t c = t / d;
  const double sIF = ldexp(1.0, -cf->F);
  const double q = size[c] > 0 ? (double)S[t] / (double)size[c] : 0.0;
  out[t] = (float)(q * sIF);
}

__global__ void k_cs_merge_err(Ctl *ctl, const Ctl *other) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && other->err)
    atomicOr(&ctl->err, other->err);
}

void stats_reserve(Arena &a, int32_t n, int64_t n_comp, int32_t d) {
  (void)n;
  a.take<Ctl>(1);
  a.take<int64_t>((size_t)n_comp * d);
  a.take<int64_t>((size_t)n_comp * 3);
}

int stats_run(const int32_t *labels, int32_t n, int32_t nc, const float *emb,
              int32_t d, const float *xyz, int64_t *size, float *emb_mean,
              float *centroid, Ctl *ctl, Arena &a, hipStream_t st) {
  Ctl *cx = a.take<Ctl>(1);  // shift of xyz; ctl holds the one of emb
  int64_t *Se = a.take<int64_t>((size_t)nc * d);
  int64_t *Sx = a.take<int64_t>((size_t)nc * 3);
  hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(64), 0, st, cx);
  hipLaunchKernelGGL(k_maxabs, dim3(2048), dim3(256), 0, st, emb,
                     (int64_t)n * d, ctl);
  hipLaunchKernelGGL(k_fixshift, dim3(1), dim3(64), 0, st, ctl, n);
  if (xyz) {
    hipLaunchKernelGGL(k_maxabs, dim3(2048), dim3(256), 0, st, xyz,
                       (int64_t)n * 3, cx);
    hipLaunchKernelGGL(k_fixshift, dim3(1), dim3(64), 0, st, cx, n);
  }
  const int nt = 256;
  hipLaunchKernelGGL(k_cs_zero, dim3((nc + nt - 1) / nt), dim3(nt), 0, st, nc,
                     d, xyz != nullptr, size, Se, Sx);
  hipLaunchKernelGGL(k_cs_add, dim3((n + nt - 1) / nt), dim3(nt), 0, st, n,
                     labels, nc, emb, d, xyz, ctl, cx, size, Se, Sx, ctl);
  const int64_t te = (int64_t)nc * d;
  hipLaunchKernelGGL(k_cs_mean, dim3((unsigned)((te + nt - 1) / nt)), dim3(nt),
                     0, st, nc, d, size, Se, ctl, emb_mean);
  if (xyz && centroid) {
    const int64_t tx = (int64_t)nc * 3;
    hipLaunchKernelGGL(k_cs_mean, dim3((unsigned)((tx + nt - 1) / nt)),
                       dim3(nt), 0, st, nc, 3, size, Sx, cx, centroid);
  }
  hipLaunchKernelGGL(k_cs_merge_err, dim3(1), dim3(64), 0, st, ctl, cx);
  // stream-asynchronous: device-detected errors stay in ctl for
  // ezsp_sync_status
  return check_hip(hipGetLastError(), "component statistics launch");
}

}  // namespace ezsp
