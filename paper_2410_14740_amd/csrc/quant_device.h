// Group-128 symmetric quantization of one 128-element group by one wave,
// shared by the create-time record builder and the fill's in-place derive
// (so both produce the same bytes). Lane l holds elements 2l and 2l + 1 as
// one fp16 pair. Per tier: s = fp16_rne(fp32(amax) / qmax),
// q = clamp(rne(w / s), -qmax, qmax), q = 0 when s == 0.
#pragma once

#include <hip/hip_fp16.h>

#include "m2c_internal.h"

namespace m2c {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

__device__ __forceinline__ int quant_code(float w, float s, float qmax) {
  if (s == 0.0f) return 0;
  float r = rintf(__fdiv_rn(w, s));
  r = fminf(fmaxf(r, -qmax), qmax);
  return (int)r;
}

// amax of the group (every lane gets it)
__device__ __forceinline__ float group_amax(uint32_t pair) {
  const float w0 = h2f((uint16_t)(pair & 0xffffu)), w1 = h2f((uint16_t)(pair >> 16));
  return wave_max(fmaxf(fabsf(w0), fabsf(w1)));
}

// INT8: the lane's two codes (low byte first) and the group's scale bits
__device__ __forceinline__ uint16_t int8_codes(uint32_t pair, float amax, uint16_t& scale) {
  const __half sh = __float2half_rn(__fdiv_rn(amax, 127.0f));
  const float s = __half2float(sh);
  const int q0 = quant_code(h2f((uint16_t)(pair & 0xffffu)), s, 127.0f);
  const int q1 = quant_code(h2f((uint16_t)(pair >> 16)), s, 127.0f);
  scale = __half_as_ushort(sh);
  return (uint16_t)((uint8_t)(int8_t)q0 | ((uint16_t)(uint8_t)(int8_t)q1 << 8));
}

// INT4: the lane's two codes in one byte (element 2l in the low nibble)
__device__ __forceinline__ uint8_t int4_codes(uint32_t pair, float amax, uint16_t& scale) {
  const __half sh = __float2half_rn(__fdiv_rn(amax, 7.0f));
  const float s = __half2float(sh);
  const int q0 = quant_code(h2f((uint16_t)(pair & 0xffffu)), s, 7.0f);
  const int q1 = quant_code(h2f((uint16_t)(pair >> 16)), s, 7.0f);
  scale = __half_as_ushort(sh);
  return (uint8_t)((q0 & 0xf) | ((q1 & 0xf) << 4));
}

}  // namespace m2c
