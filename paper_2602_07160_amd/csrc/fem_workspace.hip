// Stream-ordered scratch memory for the kernels' intermediate results, and
// the device facts the launchers size their grids by.
//
// Allocations come from a library-owned memory pool per device whose release
// threshold is unbounded, so after the first call a workspace of the same
// size is served from the pool without touching the driver.  Allocation and
// release are ordered on the caller's stream, so calls on different streams
// never share scratch.

#include "fem_internal.h"

#include <mutex>
#include <stdint.h>

namespace fem {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
hipMemPool_t g_pool[kMaxDevices] = {};

hipError_t pool_for_current_device(hipMemPool_t* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_pool[dev]) {
    hipMemPoolProps props = {};
    props.allocType = hipMemAllocationTypePinned;
    props.handleTypes = hipMemHandleTypeNone;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipMemPool_t pool = nullptr;
    e = hipMemPoolCreate(&pool, &props);
    if (e != hipSuccess) return e;
    uint64_t keep = UINT64_MAX;
    e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
    if (e != hipSuccess) {
      (void)hipMemPoolDestroy(pool);
      return e;
    }
    g_pool[dev] = pool;
  }
  *out = g_pool[dev];
  return hipSuccess;
}

}  // namespace

hipError_t workspace_alloc(void** p, size_t bytes, hipStream_t stream) {
  hipMemPool_t pool = nullptr;
  const hipError_t e = pool_for_current_device(&pool);
  if (e != hipSuccess) return e;
  return hipMallocFromPoolAsync(p, bytes, pool, stream);
}

hipError_t workspace_free(void* p, hipStream_t stream) { return hipFreeAsync(p, stream); }

int device_cus() {
  static int cus[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  std::lock_guard<std::mutex> lock(g_mu);
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) n = 0;
    cus[dev] = n;
  }
  return cus[dev];
}

}  // namespace fem
