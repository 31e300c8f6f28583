// MFMA operand fragments shared by the score and decode kernels (gfx950).
//
// A fragment is the 8 consecutive elements k = 8*(lane/16) .. +7 of one row
// (lane%16) of a 32-wide k chunk. bf16 rows feed v_mfma_f32_16x16x32_bf16
// directly; fp32 rows feed eight v_mfma_f32_16x16x4_f32 steps, where slot t
// of lane group lane/16 carries k = 8*(lane/16)+t in both operands, so the
// contraction covers the same 32 k values. The 16x16 fp32 result: lane l
// holds rows 4*(l/16)+0..3 of column l%16.
#pragma once

#include "device_common.h"

namespace sgdkv {

template <typename T>
struct Frag;
template <>
struct Frag<__bf16> {
  u32x4 v;
};
template <>
struct Frag<float> {
  u32x4 v0, v1;
};

template <typename T>
constexpr int elt_bytes() {
  return sizeof(T);
}

template <typename T>
__device__ __forceinline__ Frag<T> gload_frag(rsrc_t r, uint32_t off);
template <>
__device__ __forceinline__ Frag<__bf16> gload_frag<__bf16>(rsrc_t r, uint32_t off) {
  Frag<__bf16> f;
  f.v = ld128(r, off);
  return f;
}
template <>
__device__ __forceinline__ Frag<float> gload_frag<float>(rsrc_t r, uint32_t off) {
  Frag<float> f;
  f.v0 = ld128(r, off);
  f.v1 = ld128(r, off + 16);
  return f;
}
// The same with the non-temporal hint (keys streamed once).
template <typename T>
__device__ __forceinline__ Frag<T> gload_frag_nt(rsrc_t r, uint32_t off);
template <>
__device__ __forceinline__ Frag<__bf16> gload_frag_nt<__bf16>(rsrc_t r, uint32_t off) {
  Frag<__bf16> f;
  f.v = ld128_nt(r, off);
  return f;
}
template <>
__device__ __forceinline__ Frag<float> gload_frag_nt<float>(rsrc_t r, uint32_t off) {
  Frag<float> f;
  f.v0 = ld128_nt(r, off);
  f.v1 = ld128_nt(r, off + 16);
  return f;
}

template <typename T>
__device__ __forceinline__ Frag<T> lds_frag(const char* base, uint32_t off);
template <>
__device__ __forceinline__ Frag<__bf16> lds_frag<__bf16>(const char* base, uint32_t off) {
  Frag<__bf16> f;
  f.v = *reinterpret_cast<const u32x4*>(base + off);
  return f;
}
template <>
__device__ __forceinline__ Frag<float> lds_frag<float>(const char* base, uint32_t off) {
  Frag<float> f;
  f.v0 = *reinterpret_cast<const u32x4*>(base + off);
  f.v1 = *reinterpret_cast<const u32x4*>(base + off + 16);
  return f;
}

// acc += A(16 rows x 32 k) * B(32 k x 16 cols); both fragments hold k = 8*(lane/16)+0..7.
__device__ __forceinline__ f32x4 mma(const Frag<__bf16>& a, const Frag<__bf16>& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a.v),
                                                 __builtin_bit_cast(bf16x8, b.v), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma(const Frag<float>& a, const Frag<float>& b, f32x4 c) {
  // Eight k=4 products; slot t of every lane group carries k = 8*(lane/16)+t in both operands.
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v0.x), __uint_as_float(b.v0.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v0.y), __uint_as_float(b.v0.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v0.z), __uint_as_float(b.v0.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v0.w), __uint_as_float(b.v0.w), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v1.x), __uint_as_float(b.v1.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v1.y), __uint_as_float(b.v1.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v1.z), __uint_as_float(b.v1.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v1.w), __uint_as_float(b.v1.w), c, 0, 0, 0);
  return c;
}

}  // namespace sgdkv
