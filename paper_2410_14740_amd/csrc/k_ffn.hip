// Sparse mixed-precision SwiGLU FFN over the active neurons, each read from
// its cache slot and dequantized at its tier (Sec. 1, Sec. 5.2: only active
// neurons are computed; low-scored ones at INT8 / INT4).
//
//   y = sum_i silu(<g_i, x>) * <u_i, x> * d_i,   i over the plan's work list.
//
// Decode (batch 1) is a memory-bound gather-GEMV, so the design goal is HBM
// bandwidth: every byte of a record is read once with 16-byte loads.
//   up kernel    one wave per neuron (grabbed from a work counter, FP16 work
//                first): gate and up rows stream from the slot, INT8 / INT4
//                codes are unpacked in registers to fp16 pairs
//                (exponent-bias trick) and reduced with v_dot2_f32_f16 against
//                x staged in LDS; the group scale is applied once per 16/32
//                codes; h_i = silu(a_i) * b_i is written in work order.
//   down kernel  grid = (d-slices of 512 columns) x (neuron groups): each
//                workgroup streams the down vectors of its group for its
//                slice and writes one partial row; the partials are summed in
//                a fixed order, so results are deterministic.
#include "m2c_internal.h"

namespace m2c {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

constexpr int kUpThreads = 512;
constexpr int kDnThreads = 256;
constexpr int kDnCols = 512;

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

// Phase 1: h[w] for every work item w.
__global__ __launch_bounds__(kUpThreads) void ffn_up_kernel(
    const uint16_t* __restrict__ x, int d, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ work_slot, const uint8_t* __restrict__ slots, int64_t slot_bytes,
    int cap, int n_slots, float* __restrict__ h, int32_t* __restrict__ ctr, int total_waves) {
  extern __shared__ uint4 xs[];
  const int nc8 = d >> 3;
  uint4* xn = xs;        // x in natural order, 8 halves per entry
  uint4* xp = xs + nc8;  // x in INT4 pair order
  for (int c = threadIdx.x; c < nc8; c += blockDim.x) {
    const uint4 v = reinterpret_cast<const uint4*>(x)[c];
    xn[c] = v;
    uint4 p;
    p.x = (v.x & 0xffffu) | (v.z << 16);
    p.y = (v.x >> 16) | (v.z & 0xffff0000u);
    p.z = (v.y & 0xffffu) | (v.w << 16);
    p.w = (v.y >> 16) | (v.w & 0xffff0000u);
    xp[c] = p;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  const int n = n3 + n2 + n1;
  const int G = d >> 7;
  for (;;) {
    // Grab the next item. Every lane executes the atomic (lane 0 adds 1, the
    // others 0) and the result is broadcast with readfirstlane, so nothing
    // lane-dependent precedes the exit test and the exit is a scalar branch.
    // (A lane-0-only grab broadcast by a shuffle let the compiler split this
    // loop so that lanes 1..63 iterated without lane 0 and never left it.)
    int item = atomicAdd(&ctr[0], lane == 0 ? 1 : 0);
    item = __builtin_amdgcn_readfirstlane(item);
    if (item >= n) break;
    int slot = work_slot[item];
    const bool ok = slot >= 0 && slot < n_slots;
    const uint8_t* rec = slots + (int64_t)(ok ? slot : 0) * slot_bytes;
    float a = 0.0f, b = 0.0f;
    if (!ok) {
      // not a plan from m2c_cache_plan: contribute nothing
    } else if (item < n3) {
      const uint4* g = reinterpret_cast<const uint4*>(rec);
      const uint4* u = reinterpret_cast<const uint4*>(rec + 2 * (int64_t)d);
#pragma unroll 4
      for (int c = lane; c < nc8; c += 64) {
        const uint4 gv = g[c], uv = u[c], xv = xn[c];
        a = dot8_f16(gv, xv, a);
        b = dot8_f16(uv, xv, b);
      }
    } else if (item < n3 + n2) {
      const uint4* g = reinterpret_cast<const uint4*>(rec);
      const uint4* u = reinterpret_cast<const uint4*>(rec + d);
      const uint16_t* gs = reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)d);
      const uint16_t* us = gs + G;
      const int nc16 = d >> 4;
#pragma unroll 2
      for (int c = lane; c < nc16; c += 64) {
        const uint4 gq = g[c], uq = u[c], x0 = xn[2 * c], x1 = xn[2 * c + 1];
        const float pa = dot16_i8(gq, x0, x1, 0.0f);
        const float pb = dot16_i8(uq, x0, x1, 0.0f);
        a = fmaf(h2f(gs[c >> 3]), pa, a);
        b = fmaf(h2f(us[c >> 3]), pb, b);
      }
    } else {
      const uint4* g = reinterpret_cast<const uint4*>(rec);
      const uint4* u = reinterpret_cast<const uint4*>(rec + (d >> 1));
      const uint16_t* gs = reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)(d >> 1));
      const uint16_t* us = gs + G;
      const int nc32 = d >> 5;
#pragma unroll 2
      for (int c = lane; c < nc32; c += 64) {
        const uint4 gq = g[c], uq = u[c];
        const uint4 x0 = xp[4 * c], x1 = xp[4 * c + 1], x2 = xp[4 * c + 2], x3 = xp[4 * c + 3];
        float pa = dot8_i4(gq.x, x0, 0.0f);
        pa = dot8_i4(gq.y, x1, pa);
        pa = dot8_i4(gq.z, x2, pa);
        pa = dot8_i4(gq.w, x3, pa);
        float pb = dot8_i4(uq.x, x0, 0.0f);
        pb = dot8_i4(uq.y, x1, pb);
        pb = dot8_i4(uq.z, x2, pb);
        pb = dot8_i4(uq.w, x3, pb);
        a = fmaf(h2f(gs[c >> 2]), pa, a);
        b = fmaf(h2f(us[c >> 2]), pb, b);
      }
    }
    a = wave_sum(a);
    b = wave_sum(b);
    if (lane == 0) h[item] = silu_mul(a, b);
  }
  // The last wave out resets the work counters for the next launch.
  if (lane == 0) {
    const int done = atomicAdd(&ctr[1], 1);
    if (done == total_waves - 1) {
      atomicExch(&ctr[0], 0);
      atomicExch(&ctr[1], 0);
    }
  }
}

__device__ __forceinline__ void group_range(int n, int g, int ng, int& lo, int& hi) {
  lo = (int)((int64_t)n * g / ng);
  hi = (int)((int64_t)n * (g + 1) / ng);
}

// Phase 2: y_part[g][slice] = sum over group g's items of h_i * d_i[slice].
__global__ __launch_bounds__(kDnThreads) void ffn_down_kernel(
    int d, const int32_t* __restrict__ counts, const int32_t* __restrict__ work_slot,
    const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap, int n_slots,
    const float* __restrict__ h, int n_groups, float* __restrict__ y_part) {
  __shared__ float P[kDnThreads / 64][kDnCols];
  const int slice0 = blockIdx.x * kDnCols;
  const int grp = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int G = d >> 7;
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  float acc16[8], acc8[16], acc4[32];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc16[e] = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc8[e] = 0.0f;
#pragma unroll
  for (int e = 0; e < 32; ++e) acc4[e] = 0.0f;
  int lo, hi;
  {  // FP16: a wave covers 512 columns of one neuron, 8 per lane
    group_range(n3, grp, n_groups, lo, hi);
    const int col = slice0 + 8 * lane;
    if (col < d) {
#pragma unroll 4
      for (int it = lo + w; it < hi; it += 4) {
        const int slot = work_slot[it];
        if (slot < 0 || slot >= n_slots) continue;
        const uint8_t* rec = slots + (int64_t)slot * slot_bytes;
        const float hv = h[it];
        const uint4 v = *reinterpret_cast<const uint4*>(rec + 4 * (int64_t)d + 2 * col);
        const uint32_t ws[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc16[2 * q] = fmaf(hv, h2f((uint16_t)(ws[q] & 0xffffu)), acc16[2 * q]);
          acc16[2 * q + 1] = fmaf(hv, h2f((uint16_t)(ws[q] >> 16)), acc16[2 * q + 1]);
        }
      }
    }
  }
  {  // INT8: a half-wave covers 512 columns, 16 per lane
    group_range(n2, grp, n_groups, lo, hi);
    const int sub = lane >> 5, col = slice0 + 16 * (lane & 31);
    if (col < d) {
#pragma unroll 2
      for (int it = lo + 2 * w + sub; it < hi; it += 8) {
        const int item = n3 + it;
        const int slot = work_slot[item];
        if (slot < 0 || slot >= n_slots) continue;
        const uint8_t* rec = slots + (int64_t)slot * slot_bytes;
        const float s = h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)d + 4 * G +
                                                               2 * (col >> 7)));
        const float c = h[item] * s;
        const uint4 v = *reinterpret_cast<const uint4*>(rec + 2 * (int64_t)d + col);
        const uint32_t ws[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int bb = 0; bb < 4; ++bb) {
            const float qv = (float)(int8_t)((ws[q] >> (8 * bb)) & 0xffu);
            acc8[4 * q + bb] = fmaf(c, qv, acc8[4 * q + bb]);
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) acc8[e] += __shfl_xor(acc8[e], 32);
  }
  {  // INT4: a quarter-wave covers 512 columns, 32 per lane
    group_range(n1, grp, n_groups, lo, hi);
    const int sub = lane >> 4, col = slice0 + 32 * (lane & 15);
    if (col < d) {
#pragma unroll 2
      for (int it = lo + 4 * w + sub; it < hi; it += 16) {
        const int item = n3 + n2 + it;
        const int slot = work_slot[item];
        if (slot < 0 || slot >= n_slots) continue;
        const uint8_t* rec = slots + (int64_t)slot * slot_bytes;
        const float s = h2f(*reinterpret_cast<const uint16_t*>(
            rec + 3 * (int64_t)(d >> 1) + 4 * G + 2 * (col >> 7)));
        const float c = h[item] * s;
        const uint4 v = *reinterpret_cast<const uint4*>(rec + (int64_t)d + (col >> 1));
        const uint32_t ws[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int nb = 0; nb < 8; ++nb) {
            const int nib = (int)((ws[q] >> (4 * nb)) & 0xfu);
            const float qv = (float)(nib >= 8 ? nib - 16 : nib);
            acc4[8 * q + nb] = fmaf(c, qv, acc4[8 * q + nb]);
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      acc4[e] += __shfl_xor(acc4[e], 16);
      acc4[e] += __shfl_xor(acc4[e], 32);
    }
  }
  // per-wave partial rows: FP16 part, then INT8 and INT4 parts added in order
#pragma unroll
  for (int e = 0; e < 8; ++e) P[w][8 * lane + e] = acc16[e];
  __syncthreads();
  if (lane < 32) {
#pragma unroll
    for (int e = 0; e < 16; ++e) P[w][16 * lane + e] += acc8[e];
  }
  __syncthreads();
  if (lane < 16) {
#pragma unroll
    for (int e = 0; e < 32; ++e) P[w][32 * lane + e] += acc4[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < kDnCols; c += kDnThreads) {
    const int col = slice0 + c;
    if (col < d) {
      float v = P[0][c];
#pragma unroll
      for (int q = 1; q < kDnThreads / 64; ++q) v += P[q][c];
      y_part[(int64_t)grp * d + col] = v;
    }
  }
}

__global__ void ffn_reduce_kernel(const float* __restrict__ y_part, int n_groups, int d,
                                  float* __restrict__ y) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= d) return;
  float v = y_part[j];
  for (int g = 1; g < n_groups; ++g) v += y_part[(int64_t)g * d + j];
  y[j] = v;
}

hipError_t launch_ffn(m2c_layer* L, const uint16_t* x, int batch, const uint8_t* plan, float* y,
                      hipStream_t stream) {
  (void)batch;  // batch 1 (checked by the caller)
  const int d = L->desc.d_model;
  const m2c_plan_layout& lay = L->layout;
  const int32_t* counts = reinterpret_cast<const int32_t*>(plan + lay.counts);
  const int32_t* work_slot = reinterpret_cast<const int32_t*>(plan + lay.work_slot);
  const int64_t sb = L->info.slot_bytes;
  int blocks = L->num_cus;
  const int need = (L->cap + kUpThreads / 64 - 1) / (kUpThreads / 64);
  if (blocks > need) blocks = need > 0 ? need : 1;
  const int total_waves = blocks * (kUpThreads / 64);
  const int n_slots = L->desc.cache_slots + L->S;
  hipLaunchKernelGGL(ffn_up_kernel, dim3(blocks), dim3(kUpThreads), (size_t)d * 4, stream, x, d,
                     counts, work_slot, L->slots, sb, L->cap, n_slots, L->h, L->ffn_ctr,
                     total_waves);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int ng = L->ffn_groups;
  float* dst = ng == 1 ? y : L->y_part;
  hipLaunchKernelGGL(ffn_down_kernel, dim3((d + kDnCols - 1) / kDnCols, ng), dim3(kDnThreads), 0,
                     stream, d, counts, work_slot, L->slots, sb, L->cap, n_slots, L->h, ng, dst);
  e = hipGetLastError();
  if (e != hipSuccess || ng == 1) return e;
  hipLaunchKernelGGL(ffn_reduce_kernel, dim3((d + 255) / 256), dim3(256), 0, stream, L->y_part,
                     ng, d, y);
  return hipGetLastError();
}

}  // namespace m2c
