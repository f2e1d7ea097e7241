// ezsp_noalloc.hip -- ezsp_knn_noalloc: the kNN entry point (Sec. 3.1, the
// k-nearest-neighbour graph) for callers that cannot allocate memory, with
// its scratch in a file-scope device array instead of a caller workspace.
//
// The array lives in the library's code object: each GPU the library runs
// on holds its own copy, at its own address, until the process ends.  Host
// code never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol); it looks up the device address once per device
// with hipGetSymbolAddress and passes that.  Every call on one GPU shares
// the array: calls that overlap on one GPU (different streams, or threads)
// race, and each call re-initialises what must start at zero (its control
// block, by a kernel) before using it.
#include <mutex>

#include "../../include/ezsp.h"
#include "ezsp_internal.h"

namespace ezsp {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device

}  // namespace

int noalloc_scratch(void **ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("no usable current HIP device (%d)", dev);
    return EZSP_ERR_DEVICE;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error("hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                hipGetErrorString(e));
      return EZSP_ERR_DEVICE;
    }
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return EZSP_OK;
}

}  // namespace ezsp

using namespace ezsp;

extern "C" int ezsp_knn_noalloc(const float *xyz, int64_t n, int32_t k,
                                int32_t *nbr, float *d2, void *stream) {
  set_error("%s", "");
  if (!xyz || !nbr) {
    set_error("xyz and nbr must not be NULL");
    return EZSP_ERR_INVALID_ARG;
  }
  const size_t need = ezsp_knn_workspace_size(n, k);
  if (need == 0) {
    set_error("n must be in [1, 2^31 - 256] and k in 1..64");
    return EZSP_ERR_INVALID_ARG;
  }
  if (need > kNoallocScratchBytes) {
    set_error("n = %lld, k = %d need %zu bytes of scratch; the static scratch "
              "holds %zu (use ezsp_knn with a workspace)",
              (long long)n, k, need, kNoallocScratchBytes);
    return EZSP_ERR_INVALID_ARG;
  }
  void *ws = nullptr;
  const int rc = noalloc_scratch(&ws);
  if (rc) return rc;
  return ezsp_knn(xyz, n, k, nbr, d2, ws, kNoallocScratchBytes, stream);
}
