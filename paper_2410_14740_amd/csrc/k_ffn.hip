// Sparse mixed-precision SwiGLU FFN over the active neurons, each read from
// its cache slot and dequantized at its tier (Sec. 1, Sec. 5.2: only active
// neurons are computed; low-scored ones at INT8 / INT4).
//
//   y = sum_i silu(<g_i, x>) * <u_i, x> * d_i,   i over the plan's work list.
//
// Decode (batch 1) is a memory-bound gather-GEMV, so the design goal is HBM
// bandwidth: every byte of a record is read once with 16-byte loads.
//   up kernel    gate and up rows are cut into units of d bytes (see
//                unit_count); waves take units round-robin, unpack INT8 /
//                INT4 codes in registers to exact fp16 pairs (exponent-bias
//                trick), reduce with v_dot2_f32_f16 against x staged in LDS,
//                apply the group scale once per 16 / 32 codes and write one
//                partial (gate, up) pair per unit.
//   down kernel  grid = (d-slices of 512 columns) x (neuron groups): each
//                workgroup forms h_i = silu(a_i) * b_i from the partials,
//                streams its group's down vectors for its slice and writes
//                one partial row; a small kernel sums the partial rows in a
//                fixed order, so results are deterministic.
#include "ffn_device.h"

namespace m2c {

constexpr int kUpThreads = 1024;
constexpr int kDnThreads = 256;
constexpr int kDnCols = 512;

// Work units of the up kernel. Every neuron's gate and up rows are split
// into units of d bytes: an FP16 neuron in 4 quarters (d/4 elements), an
// INT8 neuron in 2 halves (d/2 elements), an INT4 neuron whole. In every
// tier a unit is d/32 chunks of 16 bytes per row. Units are numbered
// tier-major: FP16 item i owns units 4i..4i+3, INT8 item j units
// 4*n3 + 2j, +1, INT4 item m unit 4*n3 + 2*n2 + m.
__device__ __forceinline__ int unit_count(int n3, int n2, int n1) { return 4 * n3 + 2 * n2 + n1; }

// h of work item `it` from its units' partial dot products, summed in
// ascending unit order (deterministic).
__device__ __forceinline__ float item_h(const float2* __restrict__ ab, int it, int n3, int n2) {
  int u, np;
  if (it < n3) {
    u = 4 * it;
    np = 4;
  } else if (it < n3 + n2) {
    u = 4 * n3 + 2 * (it - n3);
    np = 2;
  } else {
    u = 4 * n3 + 2 * n2 + (it - n3 - n2);
    np = 1;
  }
  float a = ab[u].x, b = ab[u].y;
  for (int p = 1; p < np; ++p) {
    a += ab[u + p].x;
    b += ab[u + p].y;
  }
  return silu_mul(a, b);
}

// Phase 1: partial gate / up dot products of every unit. One workgroup per
// CU stages x in LDS; its waves take units round-robin (all units read the
// same number of bytes, so the split is balanced without atomics). K is the
// number of 16-byte chunks per lane and row of a unit (d <= 2048 K).
//
// Loads are issued without branches around them: lanes past the unit and
// units with a bad slot read valid memory (chunk ncu-1 of slot 0) and their
// results are discarded by selects. A load under a per-lane branch becomes
// its own basic block, and the waitcnt pass then drains earlier loads before
// issuing it, which serializes what should be in flight together.
template <int K>
__global__ __launch_bounds__(kUpThreads) void ffn_up_kernel(
    const uint16_t* __restrict__ x, int d, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ work_slot, const uint8_t* __restrict__ slots, int64_t slot_bytes,
    int cap, int n_slots, float2* __restrict__ ab) {
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
  const int U = unit_count(n3, n2, n1);
  const int G = d >> 7;
  const int ncu = d >> 5;  // 16-byte chunks per row of a unit
  const int waves = kUpThreads / 64;
  const int gw = __builtin_amdgcn_readfirstlane(blockIdx.x * waves + (threadIdx.x >> 6));
  const int W = gridDim.x * waves;
  for (int u = gw; u < U; u += W) {
    int tier, item, part;
    if (u < 4 * n3) {
      tier = 3;
      item = u >> 2;
      part = u & 3;
    } else if (u < 4 * n3 + 2 * n2) {
      tier = 2;
      item = n3 + ((u - 4 * n3) >> 1);
      part = (u - 4 * n3) & 1;
    } else {
      tier = 1;
      item = n3 + n2 + (u - 4 * n3 - 2 * n2);
      part = 0;
    }
    const int slot = work_slot[item];
    const bool ok = slot >= 0 && slot < n_slots;  // else not a plan from m2c_cache_plan
    const uint8_t* rec = slots + (int64_t)(ok ? slot : 0) * slot_bytes;
    const int64_t row = tier == 3 ? 2 * (int64_t)d : tier == 2 ? d : (d >> 1);
    const int c0 = part * ncu;  // first chunk of this unit within the row
    const uint4* g = reinterpret_cast<const uint4*>(rec) + c0;
    const uint4* up = reinterpret_cast<const uint4*>(rec + row) + c0;
    // scales of INT8 (group = chunk / 8) and INT4 (group = chunk / 4); read
    // (and ignored) for FP16 too, to keep the loads branch-free
    const uint16_t* gs =
        reinterpret_cast<const uint16_t*>(rec + (tier == 1 ? 3 * (int64_t)(d >> 1) : 3 * (int64_t)d));
    const int sh = tier == 1 ? 2 : 3;
    uint4 gq[K], uq[K];
    uint16_t sgb[K], sub[K];
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int c = min(lane + 64 * i, ncu - 1);
      gq[i] = g[c];
      uq[i] = up[c];
      sgb[i] = gs[(c0 + c) >> sh];
      sub[i] = gs[G + ((c0 + c) >> sh)];
    }
    float a = 0.0f, b = 0.0f;
    if (tier == 3) {
#pragma unroll
      for (int i = 0; i < K; ++i) {
        const int c = min(lane + 64 * i, ncu - 1);
        const uint4 xv = xn[c0 + c];
        const float pa = dot8_f16(gq[i], xv, 0.0f), pb = dot8_f16(uq[i], xv, 0.0f);
        const bool v = ok && lane + 64 * i < ncu;
        a += v ? pa : 0.0f;
        b += v ? pb : 0.0f;
      }
    } else if (tier == 2) {
#pragma unroll
      for (int i = 0; i < K; ++i) {
        const int c = c0 + min(lane + 64 * i, ncu - 1);
        const uint4 x0 = xn[2 * c], x1 = xn[2 * c + 1];
        const float pa = h2f(sgb[i]) * dot16_i8(gq[i], x0, x1, 0.0f);
        const float pb = h2f(sub[i]) * dot16_i8(uq[i], x0, x1, 0.0f);
        const bool v = ok && lane + 64 * i < ncu;
        a += v ? pa : 0.0f;
        b += v ? pb : 0.0f;
      }
    } else {
#pragma unroll
      for (int i = 0; i < K; ++i) {
        const int c = min(lane + 64 * i, ncu - 1);
        const uint4 x0 = xp[4 * c], x1 = xp[4 * c + 1], x2 = xp[4 * c + 2], x3 = xp[4 * c + 3];
        float pa = dot8_i4(gq[i].x, x0, 0.0f);
        pa = dot8_i4(gq[i].y, x1, pa);
        pa = dot8_i4(gq[i].z, x2, pa);
        pa = dot8_i4(gq[i].w, x3, pa);
        float pb = dot8_i4(uq[i].x, x0, 0.0f);
        pb = dot8_i4(uq[i].y, x1, pb);
        pb = dot8_i4(uq[i].z, x2, pb);
        pb = dot8_i4(uq[i].w, x3, pb);
        const bool v = ok && lane + 64 * i < ncu;
        a += v ? h2f(sgb[i]) * pa : 0.0f;
        b += v ? h2f(sub[i]) * pb : 0.0f;
      }
    }
    a = wave_sum(a);
    b = wave_sum(b);
    if (lane == 0) ab[u] = make_float2(a, b);
  }
}

__device__ __forceinline__ void group_range(int n, int g, int ng, int& lo, int& hi) {
  lo = (int)((int64_t)n * g / ng);
  hi = (int)((int64_t)n * (g + 1) / ng);
}

constexpr int kDnWaves = kDnThreads / 64;
constexpr int kDnBatch = 8;          // items whose loads are in flight together, per wave
constexpr int kDnMaxPerTier = 512;   // items staged in LDS at a time
constexpr int kMaxGroups = 64;       // partial rows summed by the reduce kernel

// Phase 2: y[slice] = sum over items of h_i * d_i[slice]. Workgroup
// (slice, group) first stages its group's slots and h_i (formed from the
// unit partials) in LDS, then streams the group's down vectors for its 512
// columns with kDnBatch loads in flight per wave, and writes one partial row
// (or y itself when there is one group).
__global__ __launch_bounds__(kDnThreads) void ffn_down_kernel(
    int d, const int32_t* __restrict__ counts, const int32_t* __restrict__ work_slot,
    const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap, int n_slots,
    const float2* __restrict__ ab, int n_groups, float* __restrict__ y_part,
    float* __restrict__ y) {
  __shared__ float P[kDnWaves][kDnCols];
  __shared__ int s_slot[kDnMaxPerTier];
  __shared__ float s_h[kDnMaxPerTier];
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
  for (int t = 0; t < 3; ++t) {
    int lo, hi;
    group_range(t == 0 ? n3 : t == 1 ? n2 : n1, grp, n_groups, lo, hi);
    lo += t == 0 ? 0 : t == 1 ? n3 : n3 + n2;
    hi += t == 0 ? 0 : t == 1 ? n3 : n3 + n2;
    for (int base = lo; base < hi; base += kDnMaxPerTier) {
      const int nt = hi - base < kDnMaxPerTier ? hi - base : kDnMaxPerTier;
      __syncthreads();  // the previous chunk's lists are no longer read
      for (int i = threadIdx.x; i < nt; i += kDnThreads) {
        const int it = base + i;
        const int slot = work_slot[it];
        const bool ok = slot >= 0 && slot < n_slots;
        s_slot[i] = ok ? slot : -1;  // -1: not a plan from m2c_cache_plan, skipped
        s_h[i] = ok ? item_h(ab, it, n3, n2) : 0.0f;
      }
      __syncthreads();
      if (t == 0) {  // FP16: a wave covers 512 columns of one neuron, 8 per lane
        const int col = slice0 + 8 * lane;
        const int colc = col < d ? col : 0;
        for (int i0 = w; i0 < nt; i0 += kDnBatch * kDnWaves) {
          uint4 v[kDnBatch];
          float hv[kDnBatch];
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {
            const int i = i0 + q * kDnWaves;
            // entries past the list (or with a bad slot) read slot 0 and
            // their data is zeroed below: another tier's bytes read as fp16
            // can be Inf / NaN, and 0 * NaN is NaN
            const bool in = i < nt && s_slot[i] >= 0;
            hv[q] = in ? s_h[i] : 0.0f;
            const uint8_t* rec = slots + (int64_t)(in ? s_slot[i] : 0) * slot_bytes;
            v[q] = *reinterpret_cast<const uint4*>(rec + 4 * (int64_t)d + 2 * colc);
          }
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {  // discard what the padding read
            const bool in = i0 + q * kDnWaves < nt && s_slot[i0 + q * kDnWaves] >= 0;
            v[q] = in ? v[q] : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {
            const uint32_t ws[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              acc16[2 * e] = fmaf(hv[q], h2f((uint16_t)(ws[e] & 0xffffu)), acc16[2 * e]);
              acc16[2 * e + 1] = fmaf(hv[q], h2f((uint16_t)(ws[e] >> 16)), acc16[2 * e + 1]);
            }
          }
        }
      } else if (t == 1) {  // INT8: a half-wave covers 512 columns, 16 per lane
        const int sub = lane >> 5, col = slice0 + 16 * (lane & 31);
        const int colc = col < d ? col : 0;
        const int64_t soff = 3 * (int64_t)d + 4 * G + 2 * (colc >> 7);
        for (int i0 = 2 * w + sub; i0 < nt; i0 += kDnBatch * 2 * kDnWaves) {
          uint4 v[kDnBatch];
          float cv[kDnBatch];
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {
            const int i = i0 + q * 2 * kDnWaves;
            const bool in = i < nt && s_slot[i] >= 0;
            const uint8_t* rec = slots + (int64_t)(in ? s_slot[i] : 0) * slot_bytes;
            cv[q] = (in ? s_h[i] : 0.0f) * h2f(*reinterpret_cast<const uint16_t*>(rec + soff));
            v[q] = *reinterpret_cast<const uint4*>(rec + 2 * (int64_t)d + colc);
          }
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {  // discard what the padding read
            const int i = i0 + q * 2 * kDnWaves;
            const bool in = i < nt && s_slot[i] >= 0;
            cv[q] = in ? cv[q] : 0.0f;
            v[q] = in ? v[q] : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {
            const uint32_t ws[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
#pragma unroll
              for (int bb = 0; bb < 4; ++bb) {
                const float qv = (float)(int8_t)((ws[e] >> (8 * bb)) & 0xffu);
                acc8[4 * e + bb] = fmaf(cv[q], qv, acc8[4 * e + bb]);
              }
            }
          }
        }
      } else {  // INT4: a quarter-wave covers 512 columns, 32 per lane
        const int sub = lane >> 4, col = slice0 + 32 * (lane & 15);
        const int colc = col < d ? col : 0;
        const int64_t soff = 3 * (int64_t)(d >> 1) + 4 * G + 2 * (colc >> 7);
        for (int i0 = 4 * w + sub; i0 < nt; i0 += kDnBatch * 4 * kDnWaves) {
          uint4 v[kDnBatch];
          float cv[kDnBatch];
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {
            const int i = i0 + q * 4 * kDnWaves;
            const bool in = i < nt && s_slot[i] >= 0;
            const uint8_t* rec = slots + (int64_t)(in ? s_slot[i] : 0) * slot_bytes;
            cv[q] = (in ? s_h[i] : 0.0f) * h2f(*reinterpret_cast<const uint16_t*>(rec + soff));
            v[q] = *reinterpret_cast<const uint4*>(rec + (int64_t)d + (colc >> 1));
          }
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {  // discard what the padding read
            const int i = i0 + q * 4 * kDnWaves;
            const bool in = i < nt && s_slot[i] >= 0;
            cv[q] = in ? cv[q] : 0.0f;
            v[q] = in ? v[q] : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
          for (int q = 0; q < kDnBatch; ++q) {
            const uint32_t ws[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
#pragma unroll
              for (int nb = 0; nb < 8; ++nb) {
                const int nib = (int)((ws[e] >> (4 * nb)) & 0xfu);
                const float qv = (float)(nib >= 8 ? nib - 16 : nib);
                acc4[8 * e + nb] = fmaf(cv[q], qv, acc4[8 * e + nb]);
              }
            }
          }
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) acc8[e] += __shfl_xor(acc8[e], 32);
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    acc4[e] += __shfl_xor(acc4[e], 16);
    acc4[e] += __shfl_xor(acc4[e], 32);
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
      for (int q = 1; q < kDnWaves; ++q) v += P[q][c];
      if (n_groups == 1)
        y[col] += v;  // accumulate into the residual stream
      else
        y_part[(int64_t)grp * d + col] = v;
    }
  }
}

// y[j] += sum over groups of the partial rows, in group order. All of a
// column's partials are loaded before the ordered sum. A separate launch
// rather than a last-arriver inside the down kernel: a device-scope release
// there writes back the XCD's whole L2, including the slot lines an
// overlapping fill has just written, which cost more than this launch.
__global__ __launch_bounds__(256) void ffn_reduce_kernel(const float* __restrict__ y_part,
                                                         int n_groups, int d,
                                                         float* __restrict__ y) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= d) return;
  float v[kMaxGroups];
#pragma unroll
  for (int g = 0; g < kMaxGroups; ++g) v[g] = g < n_groups ? y_part[(int64_t)g * d + j] : 0.0f;
  float acc = v[0];
#pragma unroll
  for (int g = 1; g < kMaxGroups; ++g)
    if (g < n_groups) acc += v[g];
  y[j] += acc;  // accumulate into the residual stream
}

hipError_t launch_ffn(m2c_layer* L, const uint16_t* x, int batch, const uint8_t* plan, float* y,
                      hipStream_t stream) {
  if (batch > 1) return launch_ffn_batch(L, x, batch, plan, y, stream);
  if (!(L->desc.flags & M2C_FLAG_DETERMINISTIC_FFN))
    return ffn_fused_supported(L) ? launch_ffn_fused(L, x, plan, y, stream)
                                                : launch_ffn_split(L, x, plan, y, stream);
  const int d = L->desc.d_model;
  const m2c_plan_layout& lay = L->layout;
  const int32_t* counts = reinterpret_cast<const int32_t*>(plan + lay.counts);
  const int32_t* work_slot = reinterpret_cast<const int32_t*>(plan + lay.work_slot);
  const int64_t sb = L->info.slot_bytes;
  const int n_slots = L->desc.cache_slots + L->S;
  int blocks = L->num_cus;
  const int waves = kUpThreads / 64;
  const int need = (4 * L->cap + waves - 1) / waves;
  if (blocks > need) blocks = need > 0 ? need : 1;
  const size_t lds = (size_t)d * 4;
  if (d <= 2048)
    hipLaunchKernelGGL(ffn_up_kernel<1>, dim3(blocks), dim3(kUpThreads), lds, stream, x, d,
                       counts, work_slot, L->slots, sb, L->cap, n_slots, L->ab);
  else if (d <= 4096)
    hipLaunchKernelGGL(ffn_up_kernel<2>, dim3(blocks), dim3(kUpThreads), lds, stream, x, d,
                       counts, work_slot, L->slots, sb, L->cap, n_slots, L->ab);
  else if (d <= 8192)
    hipLaunchKernelGGL(ffn_up_kernel<4>, dim3(blocks), dim3(kUpThreads), lds, stream, x, d,
                       counts, work_slot, L->slots, sb, L->cap, n_slots, L->ab);
  else
    hipLaunchKernelGGL(ffn_up_kernel<8>, dim3(blocks), dim3(kUpThreads), lds, stream, x, d,
                       counts, work_slot, L->slots, sb, L->cap, n_slots, L->ab);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int ng = L->ffn_groups;
  hipLaunchKernelGGL(ffn_down_kernel, dim3((d + kDnCols - 1) / kDnCols, ng), dim3(kDnThreads), 0,
                     stream, d, counts, work_slot, L->slots, sb, L->cap, n_slots, L->ab, ng,
                     L->y_part, y);
  e = hipGetLastError();
  if (e != hipSuccess || ng == 1) return e;
  hipLaunchKernelGGL(ffn_reduce_kernel, dim3((d + 255) / 256), dim3(256), 0, stream, L->y_part, ng,
                     d, y);
  return hipGetLastError();
}

}  // namespace m2c
