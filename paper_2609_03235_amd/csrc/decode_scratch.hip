// Static device scratch for the decode entry point that allocates nothing
// (sgdkv_decode_attention_noalloc).
//
// `scratch` is a file-scope device array: every GPU the library runs on holds
// its own copy, at its own address, from the moment this code object is loaded
// until the process ends. In host code the array's name is only a host-side
// stand-in, so the device address is looked up once per device with
// hipGetSymbolAddress, with that device current, and kept; kernels receive
// that address, never the name. Calls on one GPU share its copy: their split
// partials overwrite each other, so calls that overlap in time on one GPU race.
// Every partial the combine reads is written by the split kernel of the same
// call, so nothing needs clearing between calls.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "sgdkv_internal.h"

namespace sgdkv {

static __device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];

hipError_t decode_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  static std::mutex mu;
  static std::vector<void*> addr;  // per device; nullptr until looked up
  std::lock_guard<std::mutex> lock(mu);
  if ((int)addr.size() <= dev) addr.resize(dev + 1, nullptr);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace sgdkv
