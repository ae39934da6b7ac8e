// Device helpers shared by the sparse FFN kernels (gather-dequant GEMV).
#pragma once

#include "m2c_internal.h"

namespace m2c {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));


__device__ __forceinline__ half2v as_h2(uint32_t u) { return __builtin_bit_cast(half2v, u); }

__device__ __forceinline__ float dot8_f16(const uint4 w, const uint4 x, float acc) {
  acc = __builtin_amdgcn_fdot2(as_h2(w.x), as_h2(x.x), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(w.y), as_h2(x.y), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(w.z), as_h2(x.z), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(w.w), as_h2(x.w), acc, false);
  return acc;
}

// Four int8 codes (one word) -> two fp16 pairs holding the exact code values.
// Byte b becomes offset-binary b ^ 0x80 = q + 128, is placed under the fp16
// exponent byte 0x64 (value 1024 + byte), and 1152 is subtracted.
__device__ __forceinline__ void i8x4_to_h2(uint32_t w, half2v& lo, half2v& hi) {
  const uint32_t ob = w ^ 0x80808080u;
  const uint32_t l = __builtin_amdgcn_perm(0x64646464u, ob, 0x04010400u);
  const uint32_t h = __builtin_amdgcn_perm(0x64646464u, ob, 0x04030402u);
  const half2v bias = {(_Float16)1152.0f, (_Float16)1152.0f};
  lo = as_h2(l) - bias;
  hi = as_h2(h) - bias;
}

__device__ __forceinline__ float dot16_i8(const uint4 q, const uint4 x0, const uint4 x1,
                                          float acc) {
  half2v a, b;
  i8x4_to_h2(q.x, a, b);
  acc = __builtin_amdgcn_fdot2(a, as_h2(x0.x), acc, false);
  acc = __builtin_amdgcn_fdot2(b, as_h2(x0.y), acc, false);
  i8x4_to_h2(q.y, a, b);
  acc = __builtin_amdgcn_fdot2(a, as_h2(x0.z), acc, false);
  acc = __builtin_amdgcn_fdot2(b, as_h2(x0.w), acc, false);
  i8x4_to_h2(q.z, a, b);
  acc = __builtin_amdgcn_fdot2(a, as_h2(x1.x), acc, false);
  acc = __builtin_amdgcn_fdot2(b, as_h2(x1.y), acc, false);
  i8x4_to_h2(q.w, a, b);
  acc = __builtin_amdgcn_fdot2(a, as_h2(x1.z), acc, false);
  acc = __builtin_amdgcn_fdot2(b, as_h2(x1.w), acc, false);
  return acc;
}

// Eight int4 codes (one word, element e in bits 4e..4e+3) against x held in
// the pair order (x0,x4), (x1,x5), (x2,x6), (x3,x7).
__device__ __forceinline__ float dot8_i4(uint32_t w, const uint4 xp, float acc) {
  const uint32_t ob = w ^ 0x88888888u;  // q + 8
  const half2v bias = {(_Float16)1032.0f, (_Float16)1032.0f};
  const uint32_t m = 0x000F000Fu, e = 0x64006400u;
  acc = __builtin_amdgcn_fdot2(as_h2((ob & m) | e) - bias, as_h2(xp.x), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(((ob >> 4) & m) | e) - bias, as_h2(xp.y), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(((ob >> 8) & m) | e) - bias, as_h2(xp.z), acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(((ob >> 12) & m) | e) - bias, as_h2(xp.w), acc, false);
  return acc;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Work counts of a plan, clamped so that a buffer that did not come from
// m2c_cache_plan can never index past the plan lists.
__device__ __forceinline__ void work_counts(const int32_t* counts, int cap, int& n3, int& n2,
                                            int& n1) {
  n3 = counts[M2C_CNT_REQ_FP16];
  n2 = counts[M2C_CNT_REQ_INT8];
  n1 = counts[M2C_CNT_REQ_INT4];
  n3 = n3 < 0 ? 0 : n3 > cap ? cap : n3;
  n2 = n2 < 0 ? 0 : n2 > cap - n3 ? cap - n3 : n2;
  n1 = n1 < 0 ? 0 : n1 > cap - n3 - n2 ? cap - n3 - n2 : n1;
}

__device__ __forceinline__ float silu_mul(float a, float b) { return a / (1.0f + expf(-a)) * b; }

}  // namespace m2c
