// Sparse mixed-precision SwiGLU FFN for one token in two launches (Sec. 1 and
// Sec. 5.2: only the active neurons are computed, each at its precision).
//
//   y += sum_i silu(<g_i, x>) * <u_i, x> * d_i
//
// The sum couples every neuron (h_i needs the whole of g_i and u_i) with
// every output column (d_i spans all of them). One kernel per neuron range
// has to reduce a full d-wide partial row per workgroup across the chip, and
// at a few hundred workgroups those atomics cost as much as streaming the
// weights. So the work is cut twice:
//
//   ffn_h_kernel   h_i for every neuron of the plan's work list. A workgroup
//                  of 8 waves takes 8 consecutive "units" of one tier -- a
//                  unit is d bytes of a neuron's gate and up rows, so 2 FP16,
//                  4 INT8 or 8 INT4 neurons -- issues all of its loads at
//                  once, reduces each unit with v_dot2_f32_f16 against x in
//                  LDS (INT8 / INT4 codes unpacked to exact fp16 pairs), and
//                  forms h_i from its units in LDS, in unit order.
//   ffn_dn_kernel  y by (column slice) x (neuron group): each lane owns 32
//                  output columns of the slice for every tier, so every byte
//                  of a down vector is loaded once, 16 bytes at a time, and
//                  the lanes that share columns are combined by shuffles and
//                  LDS; one fp32 atomic add per column and workgroup brings
//                  the groups together.
//
// Workgroups are one-shot (no loops over work), so the hardware dispatcher
// keeps every CU streaming. The grid is sized for the largest plan the layer
// can produce; workgroups past the plan's counts return at once.
#include "ffn_device.h"

namespace m2c {

constexpr int kHThreads = 512;
constexpr int kHUnits = kHThreads / 64;  // one unit per wave

// Neurons and units per workgroup of the h kernel, by tier.
__device__ __forceinline__ void h_block(int b, int n3, int n2, int n1, int& tier, int& item0,
                                        int& nitems) {
  const int w3 = (n3 + 1) >> 1, w2 = (n2 + 3) >> 2, w1 = (n1 + 7) >> 3;
  if (b < w3) {
    tier = 3;
    item0 = 2 * b;
    nitems = min(2, n3 - item0);
  } else if (b < w3 + w2) {
    tier = 2;
    item0 = 4 * (b - w3);
    nitems = min(4, n2 - item0);
    item0 += n3;
  } else if (b < w3 + w2 + w1) {
    tier = 1;
    item0 = 8 * (b - w3 - w2);
    nitems = min(8, n1 - item0);
    item0 += n3 + n2;
  } else {
    tier = 0;
    item0 = 0;
    nitems = 0;
  }
}

// K: 16-byte chunks per lane per unit, K >= ceil(2 * (d / 32) / 64) = ceil(d / 1024).
template <int K>
__global__ __launch_bounds__(kHThreads) void ffn_h_kernel(
    const uint16_t* __restrict__ x, int d, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ work_slot, const uint8_t* __restrict__ slots, int64_t slot_bytes,
    int cap, int n_slots, float* __restrict__ h_out) {
  extern __shared__ uint4 xs[];  // x: natural order (FP16, INT8) or INT4 pair order
  __shared__ float2 s_ab[kHUnits];
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  int tier, item0, nitems;
  h_block(blockIdx.x, n3, n2, n1, tier, item0, nitems);
  if (nitems <= 0) return;  // workgroup-uniform
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int upi = tier == 3 ? 4 : tier == 2 ? 2 : 1;  // units per neuron
  const int G = d >> 7;
  const int ncu = d >> 5;  // 16-byte chunks per row in a unit
  const int k = w / upi, part = w % upi;
  const bool has_unit = k < nitems;
  const int slot = work_slot[item0 + (has_unit ? k : 0)];
  const bool uok = has_unit && slot >= 0 && slot < n_slots;
  // slot n_slots is all zeros: units that do not exist read it
  const uint8_t* rec = slots + (int64_t)(uok ? slot : n_slots) * slot_bytes;
  const uint8_t* zero = slots + (int64_t)n_slots * slot_bytes;
  const int64_t row = tier == 3 ? 2 * (int64_t)d : tier == 2 ? d : (d >> 1);  // up row offset
  const int64_t sbase = tier == 1 ? 3 * (int64_t)(d >> 1) : 3 * (int64_t)d;  // gate scales
  const int c0 = part * ncu;  // first chunk of this unit in its row
  // x chunks this thread stages, loaded first so that waiting for them does
  // not wait for the unit data as well (loads complete in issue order)
  constexpr int XPT = (K + 3) / 4;  // d / 8 / kHThreads <= XPT
  const int nc8 = d >> 3;
  const uint4* xg = reinterpret_cast<const uint4*>(x);
  uint4 xv[XPT];
#pragma unroll
  for (int j = 0; j < XPT; ++j) xv[j] = xg[min((int)threadIdx.x + kHThreads * j, nc8 - 1)];
  // keep the x loads ahead of the unit loads: the LDS write of x then waits
  // for x alone, and the dot products start while unit data still arrives
  __builtin_amdgcn_sched_barrier(0);
  // Every load of the unit: chunk q < ncu of the gate row-part, q >= ncu of
  // the up row-part. Lanes past the unit read the zero slot, so no load sits
  // under a branch and no loaded value needs a select.
  uint4 v[K];
  uint16_t sc[K];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    int q = lane + 64 * j;
    const bool in = q < 2 * ncu;
    q = in ? q : 2 * ncu - 1;
    const bool up = q >= ncu;
    const int c = c0 + (up ? q - ncu : q);
    const uint8_t* base = in ? rec : zero;
    v[j] = *reinterpret_cast<const uint4*>(base + (up ? row : 0) + 16 * (int64_t)c);
    const int g = tier == 2 ? (c >> 3) : (c >> 2);  // INT8: 16 codes per chunk, INT4: 32
    sc[j] = *reinterpret_cast<const uint16_t*>(base + sbase + 2 * (int64_t)((up ? G : 0) + g));
  }
  if (tier == 1) {
#pragma unroll
    for (int j = 0; j < XPT; ++j) {
      const int c = threadIdx.x + kHThreads * j;
      const uint4 t = xv[j];
      uint4 p;  // (x0,x4) (x1,x5) (x2,x6) (x3,x7): pairs that match the nibble unpack
      p.x = (t.x & 0xffffu) | (t.z << 16);
      p.y = (t.x >> 16) | (t.z & 0xffff0000u);
      p.z = (t.y & 0xffffu) | (t.w << 16);
      p.w = (t.y >> 16) | (t.w & 0xffff0000u);
      if (c < nc8) xs[c] = p;
    }
  } else {
#pragma unroll
    for (int j = 0; j < XPT; ++j) {
      const int c = threadIdx.x + kHThreads * j;
      if (c < nc8) xs[c] = xv[j];
    }
  }
  __syncthreads();
  float a = 0.0f, b = 0.0f;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int q0 = lane + 64 * j;
    const int q = q0 < 2 * ncu ? q0 : 2 * ncu - 1;
    const bool up = q >= ncu;
    const int c = c0 + (up ? q - ncu : q);
    float p;
    if (tier == 3) {
      p = dot8_f16(v[j], xs[c], 0.0f);
    } else if (tier == 2) {
      p = h2f(sc[j]) * dot16_i8(v[j], xs[2 * c], xs[2 * c + 1], 0.0f);
    } else {
      float t = dot8_i4(v[j].x, xs[4 * c], 0.0f);
      t = dot8_i4(v[j].y, xs[4 * c + 1], t);
      t = dot8_i4(v[j].z, xs[4 * c + 2], t);
      t = dot8_i4(v[j].w, xs[4 * c + 3], t);
      p = h2f(sc[j]) * t;
    }
    // zero-slot lanes give p = 0 for INT8 / INT4 (scale 0) and FP16 (data 0)
    a += up ? 0.0f : p;
    b += up ? p : 0.0f;
  }
  a = wave_sum(a);
  b = wave_sum(b);
  if (lane == 0) s_ab[w] = make_float2(a, b);
  __syncthreads();
  if (threadIdx.x < nitems) {  // h of neuron t from its units, in unit order
    const int t = threadIdx.x;
    float sa = s_ab[t * upi].x, sb = s_ab[t * upi].y;
    for (int u = 1; u < upi; ++u) {
      sa += s_ab[t * upi + u].x;
      sb += s_ab[t * upi + u].y;
    }
    const int s = work_slot[item0 + t];
    h_out[item0 + t] = (s >= 0 && s < n_slots) ? silu_mul(sa, sb) : 0.0f;
  }
}

constexpr int kDThreads = 256;
constexpr int kDCols = 32;   // output columns per lane
constexpr int kDLoads = 8;   // 16-byte loads per lane of a workgroup, all in flight together

// Workgroup b of a column slice takes one tier and a run of that tier's
// neurons sized so that every lane issues kDLoads loads: rounds of NPR
// neurons, 2 rounds of FP16 (4 loads each), 4 of INT8, 8 of INT4.
template <int NPR>
__device__ __forceinline__ void dn_block(int b, int n3, int n2, int n1, int& tier, int& lo,
                                         int& hi) {
  const int i3 = 2 * NPR, i2 = 4 * NPR, i1 = 8 * NPR;  // neurons per workgroup
  const int w3 = (n3 + i3 - 1) / i3, w2 = (n2 + i2 - 1) / i2, w1 = (n1 + i1 - 1) / i1;
  if (b < w3) {
    tier = 3;
    lo = b * i3;
    hi = min(lo + i3, n3);
  } else if (b < w3 + w2) {
    tier = 2;
    lo = n3 + (b - w3) * i2;
    hi = min(lo + i2, n3 + n2);
  } else if (b < w3 + w2 + w1) {
    tier = 1;
    lo = n3 + n2 + (b - w3 - w2) * i1;
    hi = min(lo + i1, n3 + n2 + n1);
  } else {
    tier = 0;
    lo = hi = 0;
  }
}

// Down projection of tier TIER over items [lo, hi) for the lane's 32 columns
// starting at `col`. s_slot / s_h hold the items' slots and h (staged by the
// caller, item lo at index 0); every data and scale load is issued before
// any arithmetic. NPR neurons per round, LPN lanes per neuron.
template <int TIER, int LPN>
__device__ __forceinline__ void dn_tier(int lo, int hi, int col, int d, int G,
                                        const int* s_slot, const float* s_h,
                                        const uint8_t* __restrict__ slots, int64_t slot_bytes,
                                        int n_slots, float (&acc)[kDCols]) {
  constexpr int NPR = kDThreads / LPN;
  constexpr int NV = TIER == 3 ? 4 : TIER == 2 ? 2 : 1;  // 16-byte loads per lane and neuron
  constexpr int R = kDLoads / NV;                        // rounds
  const int r = threadIdx.x / LPN;                       // neuron within a round
  uint4 v[R][NV];
  float sc[R];
#pragma unroll
  for (int q = 0; q < R; ++q) {
    // padding reads slot n_slots (s_slot holds n_slots there), which is all
    // zeros: data 0 and scale 0, so it adds nothing and needs no select
    const int ii = min(q * NPR + r, hi - lo - 1);
    const int sl = q * NPR + r < hi - lo ? s_slot[ii] : n_slots;
    const uint8_t* rec = slots + (int64_t)sl * slot_bytes;
    if (TIER == 3) {
#pragma unroll
      for (int e = 0; e < NV; ++e)
        v[q][e] = *reinterpret_cast<const uint4*>(rec + 4 * (int64_t)d + 2 * (int64_t)col + 16 * e);
      sc[q] = s_h[ii];
    } else if (TIER == 2) {
#pragma unroll
      for (int e = 0; e < NV; ++e)
        v[q][e] = *reinterpret_cast<const uint4*>(rec + 2 * (int64_t)d + col + 16 * e);
      sc[q] = s_h[ii] * h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)d + 4 * G +
                                                              2 * (col >> 7)));
    } else {
      v[q][0] = *reinterpret_cast<const uint4*>(rec + (int64_t)d + (col >> 1));
      sc[q] = s_h[ii] * h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)(d >> 1) +
                                                              4 * G + 2 * (col >> 7)));
    }
  }
#pragma unroll
  for (int q = 0; q < R; ++q) {
    const float c = sc[q];
    if (TIER == 3) {
#pragma unroll
      for (int e = 0; e < NV; ++e) {
        const uint32_t ws[4] = {v[q][e].x, v[q][e].y, v[q][e].z, v[q][e].w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc[8 * e + 2 * u] = fmaf(c, h2f((uint16_t)(ws[u] & 0xffffu)), acc[8 * e + 2 * u]);
          acc[8 * e + 2 * u + 1] = fmaf(c, h2f((uint16_t)(ws[u] >> 16)), acc[8 * e + 2 * u + 1]);
        }
      }
    } else if (TIER == 2) {
#pragma unroll
      for (int e = 0; e < NV; ++e) {
        const uint32_t ws[4] = {v[q][e].x, v[q][e].y, v[q][e].z, v[q][e].w};
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int bb = 0; bb < 4; ++bb)
            acc[16 * e + 4 * u + bb] =
                fmaf(c, (float)(int8_t)((ws[u] >> (8 * bb)) & 0xffu), acc[16 * e + 4 * u + bb]);
      }
    } else {
      const uint32_t ws[4] = {v[q][0].x, v[q][0].y, v[q][0].z, v[q][0].w};
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
          const int nib = (int)((ws[u] >> (4 * nb)) & 0xfu);
          acc[8 * u + nb] = fmaf(c, (float)(nib >= 8 ? nib - 16 : nib), acc[8 * u + nb]);
        }
    }
  }
}

// SW: slice width in columns (128 or 256); LPN = SW / 32 lanes per neuron.
// blockIdx.x = slice + n_slices * (tier-run index).
template <int SW>
__global__ __launch_bounds__(kDThreads) void ffn_dn_kernel(
    int d, const int32_t* __restrict__ counts, const int32_t* __restrict__ work_slot,
    const float* __restrict__ h, const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap,
    int n_slots, float* __restrict__ y) {
  constexpr int LPN = SW / kDCols;
  constexpr int NPR = kDThreads / LPN;
  __shared__ float s_row[kDThreads / 64][SW];
  __shared__ int s_slot[8 * NPR];
  __shared__ float s_h[8 * NPR];
  const int n_slices = d / SW;
  const int slice = blockIdx.x % n_slices;
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  int tier, lo, hi;
  dn_block<NPR>(blockIdx.x / n_slices, n3, n2, n1, tier, lo, hi);
  if (lo >= hi) return;  // workgroup-uniform
  const int G = d >> 7;
  const int m = threadIdx.x % LPN;
  const int col = slice * SW + kDCols * m;
  // slots and h of the workgroup's items (at most 8 * NPR = kDThreads * 8 / LPN
  // items; kDThreads per pass), one coalesced load per thread
  for (int t = threadIdx.x; t < hi - lo; t += kDThreads) {
    const int sl = work_slot[lo + t];
    s_slot[t] = sl >= 0 && sl < n_slots ? sl : n_slots;
    s_h[t] = h[lo + t];
  }
  __syncthreads();
  float acc[kDCols];
#pragma unroll
  for (int e = 0; e < kDCols; ++e) acc[e] = 0.0f;
  if (tier == 3)
    dn_tier<3, LPN>(lo, hi, col, d, G, s_slot, s_h, slots, slot_bytes, n_slots, acc);
  else if (tier == 2)
    dn_tier<2, LPN>(lo, hi, col, d, G, s_slot, s_h, slots, slot_bytes, n_slots, acc);
  else
    dn_tier<1, LPN>(lo, hi, col, d, G, s_slot, s_h, slots, slot_bytes, n_slots, acc);
  // Lanes m, m + LPN, ... of a wave hold the same columns: fold them, then
  // the waves through LDS, in a fixed order.
#pragma unroll
  for (int off = LPN; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < kDCols; ++e) acc[e] += __shfl_xor(acc[e], off);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane < LPN) {
#pragma unroll
    for (int e = 0; e < kDCols; ++e) s_row[w][kDCols * lane + e] = acc[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < SW; c += kDThreads) {
    float t = s_row[0][c];
#pragma unroll
    for (int q = 1; q < kDThreads / 64; ++q) t += s_row[q][c];
    atomicAdd(y + slice * SW + c, t);
  }
}

template <int K>
static void launch_h(int blocks, size_t lds, hipStream_t stream, const uint16_t* x, int d,
                     const int32_t* counts, const int32_t* work_slot, const uint8_t* slots,
                     int64_t sb, int cap, int n_slots, float* h) {
  hipLaunchKernelGGL(ffn_h_kernel<K>, dim3(blocks), dim3(kHThreads), lds, stream, x, d, counts,
                     work_slot, slots, sb, cap, n_slots, h);
}

hipError_t launch_ffn_split(m2c_layer* L, const uint16_t* x, const uint8_t* plan, float* y,
                            hipStream_t stream) {
  const int d = L->desc.d_model;
  const m2c_plan_layout& lay = L->layout;
  const int32_t* counts = reinterpret_cast<const int32_t*>(plan + lay.counts);
  const int32_t* work_slot = reinterpret_cast<const int32_t*>(plan + lay.work_slot);
  const int64_t sb = L->info.slot_bytes;
  const int n_slots = L->desc.cache_slots + L->S;
  const int cap = L->cap;
  if (cap <= 0) return hipSuccess;
  float* h = reinterpret_cast<float*>(L->ab);
  // h kernel: enough workgroups for any split of cap neurons into tiers
  // (ceil(n3/2) + ceil(n2/4) + ceil(n1/8) <= cap/2 + 3); the ones past the
  // plan return at once.
  const int hblocks = (cap + 1) / 2 + 3;
  const size_t lds = (size_t)d * 2;
  const int kneed = (d + 1023) / 1024;
  if (kneed <= 1)
    launch_h<1>(hblocks, lds, stream, x, d, counts, work_slot, L->slots, sb, cap, n_slots, h);
  else if (kneed <= 2)
    launch_h<2>(hblocks, lds, stream, x, d, counts, work_slot, L->slots, sb, cap, n_slots, h);
  else if (kneed <= 4)
    launch_h<4>(hblocks, lds, stream, x, d, counts, work_slot, L->slots, sb, cap, n_slots, h);
  else if (kneed <= 5)
    launch_h<5>(hblocks, lds, stream, x, d, counts, work_slot, L->slots, sb, cap, n_slots, h);
  else if (kneed <= 8)
    launch_h<8>(hblocks, lds, stream, x, d, counts, work_slot, L->slots, sb, cap, n_slots, h);
  else
    launch_h<16>(hblocks, lds, stream, x, d, counts, work_slot, L->slots, sb, cap, n_slots, h);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // down kernel: per slice, runs of 2 * NPR neurons cover any plan in
  // cap / (2 NPR) + 3 workgroups
  const int sw = d % 256 == 0 ? 256 : 128;
  const int n_slices = d / sw;
  const int npr = kDThreads / (sw / kDCols);
  const int per_slice = cap / (2 * npr) + 3;
  if (sw == 256)
    hipLaunchKernelGGL(ffn_dn_kernel<256>, dim3(n_slices * per_slice), dim3(kDThreads), 0, stream,
                       d, counts, work_slot, h, L->slots, sb, cap, n_slots, y);
  else
    hipLaunchKernelGGL(ffn_dn_kernel<128>, dim3(n_slices * per_slice), dim3(kDThreads), 0, stream,
                       d, counts, work_slot, h, L->slots, sb, cap, n_slots, y);
  return hipGetLastError();
}

}  // namespace m2c
