// Small device helpers for gfx950 (wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mira {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef short v8s __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// Round a finite fp32 to the nearest bf16, ties to even.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ float load_act(const T* p, size_t i);
template <>
__device__ __forceinline__ float load_act<float>(const float* p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_act<uint16_t>(const uint16_t* p, size_t i) {
  return bf16_to_f32(p[i]);
}

// four consecutive activations (16-byte or 8-byte aligned) widened to fp32
__device__ __forceinline__ void load4_act(const float* p, float v[4]) {
  const v4f q = *(const v4f*)p;
  v[0] = q[0]; v[1] = q[1]; v[2] = q[2]; v[3] = q[3];
}
__device__ __forceinline__ void load4_act(const uint16_t* p, float v[4]) {
  const uint2 q = *(const uint2*)p;
  v[0] = __uint_as_float(q.x << 16);
  v[1] = __uint_as_float(q.x & 0xFFFF0000u);
  v[2] = __uint_as_float(q.y << 16);
  v[3] = __uint_as_float(q.y & 0xFFFF0000u);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// 16-byte global load / zero.
__device__ __forceinline__ v4i ld16(const void* p) { return *(const v4i*)p; }
__device__ __forceinline__ v4i zero16() { return v4i{0, 0, 0, 0}; }

// Non-temporal 16-byte load for data streamed once (packed expert bytes).
__device__ __forceinline__ v4i ld16_stream(const void* p) {
  return __builtin_nontemporal_load((const v4i*)p);
}

// D = A(16x64 int8) * B(64x16 int8) + C, int32.  Lane l holds A row l%16 and
// B column l%16, 16 k-values each (k-group l/16); D row 4*(l/16)+i, column l%16.
__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// D = A(16x32 bf16) * B(32x16 bf16) + C, fp32 (same lane layout, 8 k-values).
__device__ __forceinline__ v4f mfma_bf16(v4i a, v4i b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a),
                                                __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// Exponent e with |m| < 2^e for m > 0 (frexp convention); 0 for m == 0.
__device__ __forceinline__ int exp_bound(float m) {
  int e = 0;
  if (m > 0.f) (void)frexpf(m, &e);
  return e;
}

// Split an integer |v| < 2^23 into three balanced base-256 digits,
// v = d0 + 256*d1 + 65536*d2 with d0, d1 in [-128, 127].
__device__ __forceinline__ void split_digits(int v, int& d0, int& d1, int& d2) {
  d0 = (int)(int8_t)(v & 0xFF);
  int v1 = (v - d0) >> 8;
  d1 = (int)(int8_t)(v1 & 0xFF);
  d2 = (v1 - d1) >> 8;
}

// Order-preserving map of a finite fp32 onto uint32 (-0 is treated as +0).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  f = f + 0.0f;
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace mira
