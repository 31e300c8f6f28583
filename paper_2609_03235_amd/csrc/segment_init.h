// Per-segment set-up of the selection, run by the first workgroup of each segment in a
// kernel that precedes the selection (the column-sum pass, or select_init_kernel when that
// pass does not run): clears the segment's four radix histograms and, when the caller asked
// for the compressed cache, writes the segment's offset (and, for the last segment, the
// total) into offsets_out.
#pragma once

#include "device_common.h"
#include "sgdkv_internal.h"

namespace sgdkv {

__device__ __forceinline__ void init_segment(const CompressArgs& a, int seg) {
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int nseg = a.B * a.Hkv;
  const rsrc_t hr = make_rsrc(a.hist + (int64_t)seg * 4 * 256, 4 * 256 * 4);
  for (int i = threadIdx.x; i < 4 * 256; i += blockDim.x) st32(hr, (uint32_t)i * 4u, 0u);
  if (threadIdx.x == 0 && a.offsets != nullptr) {
    const rsrc_t orr = make_rsrc(a.offsets, (uint64_t)(nseg + 1) * 8);
    st64(orr, (uint32_t)seg * 8, (uint64_t)((int64_t)b * a.T_layer + a.prefix[h]));
    if (seg == nseg - 1) st64(orr, (uint32_t)nseg * 8, (uint64_t)((int64_t)a.B * a.T_layer));
  }
}

}  // namespace sgdkv
