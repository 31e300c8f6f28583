// Device helpers shared by the SGD-KV kernels (gfx950 only).
//
// Every global-memory access in these kernels goes through a buffer resource
// descriptor whose byte bound is the extent of the tensor slice the
// workgroup owns (one KV head's keys, one segment of the compressed cache,
// ...). The hardware range-checks each access against that bound: an
// out-of-range load returns zero and an out-of-range store is dropped, so an
// indexing slip yields wrong numbers instead of a memory fault. Zero-filled
// loads are also used on purpose for padding (rows past the last query row,
// keys past the end of a pooling window).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sgdkv {

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Word 3 of a raw (untyped, stride 0) buffer descriptor on the gfx9 family.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  // Bounds beyond 4 GiB cannot be expressed; callers keep slices below that.
  uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, kRsrcWord3);
}

__device__ __forceinline__ u32x4 ld128(rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 0);
}
__device__ __forceinline__ uint32_t ld32(rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, 0);
}
__device__ __forceinline__ float ldf(rsrc_t r, uint32_t byte_off) {
  return __uint_as_float(ld32(r, byte_off));
}
__device__ __forceinline__ void st128(rsrc_t r, uint32_t byte_off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)byte_off, 0, 0);
}
__device__ __forceinline__ void st32(rsrc_t r, uint32_t byte_off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)byte_off, 0, 0);
}
__device__ __forceinline__ void stf(rsrc_t r, uint32_t byte_off, float v) {
  st32(r, byte_off, __float_as_uint(v));
}
__device__ __forceinline__ void st64(rsrc_t r, uint32_t byte_off, uint64_t v) {
  u32x2 w;
  w.x = (uint32_t)v;
  w.y = (uint32_t)(v >> 32);
  __builtin_amdgcn_raw_buffer_store_b64(w, r, (int)byte_off, 0, 0);
}
__device__ __forceinline__ uint64_t ld64(rsrc_t r, uint32_t byte_off) {
  u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(r, (int)byte_off, 0, 0);
  return (uint64_t)w.x | ((uint64_t)w.y << 32);
}

// Non-temporal accesses (the cache-policy nt bit): for data streamed once, so that it does not
// displace what the caches hold for others.
constexpr int kNonTemporal = 2;
__device__ __forceinline__ u32x4 ld128_nt(rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, kNonTemporal);
}
__device__ __forceinline__ uint64_t ld64_nt(rsrc_t r, uint32_t byte_off) {
  u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(r, (int)byte_off, 0, kNonTemporal);
  return (uint64_t)w.x | ((uint64_t)w.y << 32);
}
__device__ __forceinline__ void st128_nt(rsrc_t r, uint32_t byte_off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)byte_off, 0, kNonTemporal);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// bf16 <-> fp32. bf16 -> fp32 is exact; fp32 -> bf16 rounds to nearest even
// (NaN kept quiet).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// Full-wave reductions (wave64) through cross-lane permutes.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// Sum over the four 16-lane groups: every lane ends with the total of its
// column (lane % 16). Two cross-lane swaps on the vector ALU, no LDS traffic.
__device__ __forceinline__ float sum_lane_groups(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float h = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(h), __float_as_uint(h), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
// Maximum over the four 16-lane groups, as sum_lane_groups.
__device__ __forceinline__ float max_lane_groups(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float h = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(h), __float_as_uint(h), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
// Maximum over the 16 lanes of a row (lanes 16r .. 16r+15), by DPP rotations.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x122, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x121, 0xF, 0xF, false)));
  return x;
}
__device__ __forceinline__ float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x122, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x121, 0xF, 0xF, false));
  return x;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace sgdkv
