// gts_host_only.cpp — stand-ins for the device side of libgts.so in a CPU-only
// build of the host library (gts_host.cpp), used to run its validation, image
// construction and argument checks under AddressSanitizer and UBSan without
// a GPU or device code.  Every kernel launch, and the no-allocation entry
// point (whose scratch is device memory), reports that there is no device.
#include <hip/hip_runtime.h>

#include "../../include/gts.h"
#include "gts_dev.h"

namespace gts {
hipError_t launch_sim(const Launch&, uint32_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_window(const Launch&, uint32_t, hipStream_t) { return hipErrorNoDevice; }
}  // namespace gts

extern "C" int gts_simulate_hwset_noalloc(const gts_graph*, const gts_hwset*, uint32_t, uint32_t, uint32_t*,
                                          uint32_t*, int32_t*, uint64_t*, uint32_t, void*) {
  return GTS_E_HIP;
}
