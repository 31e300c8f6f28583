// Stand-ins for the kernel launchers of the HIP sources, for the host-only
// sanitizer build: the host layer links against these instead of the device
// code. Every well-formed call reaches the device check first, which fails
// without a usable gfx950 device, so these only report that no device work
// can be enqueued.
#include "sgdkv_internal.h"

namespace sgdkv {
hipError_t launch_scores(const CompressArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_select(const CompressArgs&, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_gather(const CompressArgs&, int, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_decode(const DecodeArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_append(const DecodeArgs&, const void*, const void*, void*, void*, int64_t, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t decode_scratch(void**) { return hipErrorNoDevice; }
}  // namespace sgdkv
