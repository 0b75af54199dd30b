// Device helpers shared by the libtsr kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace tsr {

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two fp32 values -> packed bf16 pair (lo in bits 0..15), round to nearest
// even in hardware (v_cvt_pk_bf16_f32): one instruction per pair, the same
// bits as f32_to_bf16 for every finite input.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t h = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, h);
}

// Rotate n pairs (lo[i], hi[i]) by angles with cosine c[i] and sine s[i]:
//   lo' = lo*c - hi*s,  hi' = hi*c + lo*s
// Each product is rounded to fp32 and then added once (no fused
// multiply-add), so results match a plain fp32 evaluation bit for bit.
template <int N>
__device__ __forceinline__ void rope_rotate(float* lo, float* hi, const float* c,
                                            const float* s) {
#pragma clang fp contract(off)
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const float a = lo[i], b = hi[i];
    const float ac = a * c[i];
    const float bs = b * s[i];
    const float bc = b * c[i];
    const float as = a * s[i];
    lo[i] = ac - bs;
    hi[i] = bc + as;
  }
}

// Load 8 consecutive elements as fp32.
__device__ __forceinline__ void load8(const float* p, float* o) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
__device__ __forceinline__ void load8(const uint16_t* p, float* o) {
  const uint4 a = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = bf16_to_f32(w[i] & 0xffffu);
    o[2 * i + 1] = bf16_to_f32(w[i] >> 16);
  }
}
__device__ __forceinline__ void store8(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void store8(uint16_t* p, const float* v) {
  uint4 a;
  a.x = f32_to_bf16(v[0]) | (f32_to_bf16(v[1]) << 16);
  a.y = f32_to_bf16(v[2]) | (f32_to_bf16(v[3]) << 16);
  a.z = f32_to_bf16(v[4]) | (f32_to_bf16(v[5]) << 16);
  a.w = f32_to_bf16(v[6]) | (f32_to_bf16(v[7]) << 16);
  *reinterpret_cast<uint4*>(p) = a;
}

// Raw 8-element copies (bit exact, no conversion).
__device__ __forceinline__ void copy8(float* d, const float* s) {
  *reinterpret_cast<float4*>(d) = *reinterpret_cast<const float4*>(s);
  *reinterpret_cast<float4*>(d + 4) = *reinterpret_cast<const float4*>(s + 4);
}
__device__ __forceinline__ void copy8(uint16_t* d, const uint16_t* s) {
  *reinterpret_cast<uint4*>(d) = *reinterpret_cast<const uint4*>(s);
}

}  // namespace tsr
