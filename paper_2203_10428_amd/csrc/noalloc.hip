// The layer forward for callers that cannot allocate device memory (code
// under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc): the same kernels as pgcn_layer_fwd, with the workspace taken
// from a fixed device array of this library instead of the caller.
//
// Each GPU the library runs on holds its own copy of the array (at its own
// address) until the process ends.  Host code never passes the array's name
// to a kernel or a copy: the name is a host-side stand-in, not a device
// address.  Its address on a device is resolved once per device, with that
// device current, by pgcn_partition_setup (or by the first call on a device
// whose partitions were built before), and kept per device.
#include <atomic>
#include <mutex>

#include "internal.h"

static __device__ __align__(256) unsigned char scratch[PGCN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

}  // namespace

namespace pgcn {

int noalloc_scratch_init(int dev) {
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(PGCN_EUNSUPPORTED, "libpgcn: device ordinal above the scratch table's 64 devices");
  if (g_scratch_ptr[dev].load(std::memory_order_acquire)) return PGCN_OK;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch_ptr[dev].load(std::memory_order_relaxed)) return PGCN_OK;
  int cur = -1;
  PGCN_HIP(hipGetDevice(&cur));
  if (cur != dev) return set_error(PGCN_EINVAL, "libpgcn: scratch address resolved with another device current");
  void *ptr = nullptr;
  PGCN_HIP(hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch)));
  if (!ptr) return set_error(PGCN_EHIP, "libpgcn: hipGetSymbolAddress returned a null scratch address");
  g_scratch_ptr[dev].store(ptr, std::memory_order_release);
  return PGCN_OK;
}

}  // namespace pgcn

using namespace pgcn;

extern "C" int pgcn_layer_fwd_noalloc(const pgcn_partition *p, const pgcn_fwd_args *a, hipStream_t s) try {
  PGCN_REQUIRE(p && a, "pgcn_layer_fwd_noalloc: null partition or args");
  PGCN_REQUIRE(!p->host_only, "pgcn_layer_fwd_noalloc: partition was built host-only");
  PGCN_REQUIRE(!a->workspace && a->workspace_bytes == 0,
               "pgcn_layer_fwd_noalloc: workspace must be NULL with 0 bytes (the library's fixed scratch is used)");
  int dev = -1;
  PGCN_HIP(hipGetDevice(&dev));
  PGCN_REQUIRE(dev == p->device, "pgcn_layer_fwd_noalloc: current device differs from set-up device");
  // 0 for arguments pgcn_layer_fwd rejects: it reports them itself before any launch
  const size_t need = layer_fwd_workspace(p, a);
  if (need > (size_t)PGCN_NOALLOC_SCRATCH_BYTES)
    return set_error(PGCN_EWORKSPACE, "pgcn_layer_fwd_noalloc: the layer needs " + std::to_string(need) +
                                          " bytes of scratch, above PGCN_NOALLOC_SCRATCH_BYTES (" +
                                          std::to_string((size_t)PGCN_NOALLOC_SCRATCH_BYTES) + ")");
  void *ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!ptr) {
    int rc = noalloc_scratch_init(dev);
    if (rc) return rc;
    ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  }
  pgcn_fwd_args b = *a;
  b.workspace = ptr;
  b.workspace_bytes = (size_t)PGCN_NOALLOC_SCRATCH_BYTES;
  return pgcn_layer_fwd(p, &b, s);
} catch (...) {
  return exception_status("pgcn_layer_fwd_noalloc");
}
