// gts_noalloc.hip — gts_simulate_hwset_noalloc: gts_simulate_hwset with the
// simulations' scratch taken from a file-scope device array instead of a
// caller buffer, for callers that cannot allocate device memory.
//
// The array is a static device symbol of GTS_NOALLOC_SCRATCH_BYTES; every GPU
// the library runs on holds its own copy until the process ends.  Host code
// never passes the symbol's name to a kernel (in host code it names a host
// stand-in, not device memory): on the first call on a device, with that
// device current, its device address is looked up once with
// hipGetSymbolAddress and kept per device, and that address is what the
// kernels receive.  Nothing is allocated here: the call validates, then
// enqueues the same kernels as gts_simulate_hwset.  The kernels initialise
// every part of a simulation's scratch they read, so the array needs no
// clearing between calls (it keeps the last call's contents).
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/gts.h"

namespace gts {
int check_fixed_scratch(const gts_graph* g, uint32_t B, uint64_t limit);
int report_hip(hipError_t e, const char* what);
}  // namespace gts

namespace {

__device__ __align__(256) uint8_t scratch[GTS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];  // device address of `scratch` on each device, once looked up

// The array's device address on the current device (NULL on failure, with
// *err set).
void* scratch_on_current_device(hipError_t* err) {
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) return nullptr;
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" int gts_simulate_hwset_noalloc(const gts_graph* g, const gts_hwset* hw, uint32_t first, uint32_t B,
                                          uint32_t* out_cycles, uint32_t* out_makespan, int32_t* out_status,
                                          uint64_t* out_digest, uint32_t flags, void* hip_stream) {
  // B simulations must fit the array (GTS_E_SCRATCH before anything is
  // enqueued); argument errors are reported by gts_simulate_hwset
  const int rc = gts::check_fixed_scratch(g, B, GTS_NOALLOC_SCRATCH_BYTES);
  if (rc) return rc;
  hipError_t e = hipSuccess;
  void* p = scratch_on_current_device(&e);
  if (!p) return gts::report_hip(e, "device address of the no-allocation scratch");
  return gts_simulate_hwset(g, hw, first, B, out_cycles, out_makespan, out_status, out_digest, p,
                            GTS_NOALLOC_SCRATCH_BYTES, flags, hip_stream);
}
