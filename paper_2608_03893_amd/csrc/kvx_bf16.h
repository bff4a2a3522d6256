// bf16 / fp16 helpers shared by the bf16 map kernels (device code only).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace kvx {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// The two bf16 values packed in a 32-bit word, widened exactly to fp32.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Round two fp32 values to bf16 (round to nearest even) and pack them; one
// v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const bf16x2_t r = __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

// Inverse rotation of plane (u, v) by the angle whose (cos, sin) is the fp16
// pair cs.  fma(x, y, 0) keeps the fp16 operand inside a mixed-precision FMA.
__device__ __forceinline__ void strip(float& u, float& v, uint32_t cs) {
  const __half2 h = __builtin_bit_cast(__half2, cs);
  const float c = __low2float(h), s = __high2float(h);
  const float u0 = u, v0 = v;
  u = __builtin_fmaf(u0, c, __builtin_fmaf(v0, s, 0.0f));
  v = __builtin_fmaf(v0, c, -__builtin_fmaf(u0, s, 0.0f));
}

// Forward rotation of plane (u, v) by the angle whose (cos, sin) is cs.
__device__ __forceinline__ void rot_fwd16(float& u, float& v, uint32_t cs) {
  const __half2 h = __builtin_bit_cast(__half2, cs);
  const float c = __low2float(h), s = __high2float(h);
  const float u0 = u, v0 = v;
  u = __builtin_fmaf(u0, c, -__builtin_fmaf(v0, s, 0.0f));
  v = __builtin_fmaf(v0, c, __builtin_fmaf(u0, s, 0.0f));
}

// Strip 8 planes whose first channels are packed in a and second channels in
// b (half-split layout: channels j and j+64 in matching positions).
__device__ __forceinline__ void strip_halfsplit(uint4& a, uint4& b, const uint32_t* cs) {
  uint32_t* pa = reinterpret_cast<uint32_t*>(&a);
  uint32_t* pb = reinterpret_cast<uint32_t*>(&b);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float u0 = lo_bf16(pa[w]), u1 = hi_bf16(pa[w]);
    float v0 = lo_bf16(pb[w]), v1 = hi_bf16(pb[w]);
    strip(u0, v0, cs[2 * w]);
    strip(u1, v1, cs[2 * w + 1]);
    pa[w] = pack2(u0, u1);
    pb[w] = pack2(v0, v1);
  }
}

// Strip the 4 interleaved planes (2m, 2m+1) held in one 8-channel group.
__device__ __forceinline__ void strip_interleaved(uint4& a, const uint32_t* cs) {
  uint32_t* pa = reinterpret_cast<uint32_t*>(&a);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float u = lo_bf16(pa[w]), v = hi_bf16(pa[w]);
    strip(u, v, cs[w]);
    pa[w] = pack2(u, v);
  }
}

__device__ __forceinline__ void unpack4(const uint4& q, uint32_t* out) {
  out[0] = q.x; out[1] = q.y; out[2] = q.z; out[3] = q.w;
}

// The same operations on native 4 x 32-bit vectors (struct copies of uint4
// lower to memcpy, which can keep arrays of them out of registers).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void strip_halfsplit(u32x4_t& a, u32x4_t& b, const uint32_t* cs) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float u0 = lo_bf16(a[w]), u1 = hi_bf16(a[w]);
    float v0 = lo_bf16(b[w]), v1 = hi_bf16(b[w]);
    strip(u0, v0, cs[2 * w]);
    strip(u1, v1, cs[2 * w + 1]);
    a[w] = pack2(u0, u1);
    b[w] = pack2(v0, v1);
  }
}

__device__ __forceinline__ void strip_interleaved(u32x4_t& a, const uint32_t* cs) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float u = lo_bf16(a[w]), v = hi_bf16(a[w]);
    strip(u, v, cs[w]);
    a[w] = pack2(u, v);
  }
}

__device__ __forceinline__ void unpack4(const u32x4_t& q, uint32_t* out) {
  out[0] = q[0]; out[1] = q[1]; out[2] = q[2]; out[3] = q[3];
}

}  // namespace kvx
