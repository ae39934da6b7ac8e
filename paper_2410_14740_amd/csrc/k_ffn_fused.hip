// Fused sparse mixed-precision SwiGLU FFN: one launch per call (Sec. 1 and
// Sec. 5.2: only the active neurons are computed, each at its precision).
//
//   y += sum_i silu(<g_i, x>) * <u_i, x> * d_i
//
// A launch costs a few microseconds of dispatch, ramp and drain, which is a
// large share of a 10 us decode GEMV, so everything happens in one kernel:
//   * Workgroup b takes a contiguous, cost-balanced range of the plan's work
//     list (tier-major, so the range is FP16 items, then INT8, then INT4).
//   * It walks the range in blocks of up to 8 up-units (a unit = d bytes of a
//     neuron's gate and up rows: an FP16 quarter, an INT8 half or a whole INT4
//     neuron), one unit per wave. For a block it issues the gate/up loads of
//     the units and the down loads of the block's neurons at once -- the down
//     loads do not depend on h -- then reduces the units with v_dot2_f32_f16
//     against x in LDS, forms h_i = silu(a_i) * b_i in LDS, and applies h_i to
//     the down data already in registers.
//   * Wave w owns output columns [w d/8, (w+1) d/8) (in 8-column chunks), so
//     the down accumulation stays in registers; at the end the workgroup
//     stages its partial row in LDS and adds it into y with fp32 atomics,
//     consecutive lanes on consecutive columns.
// The atomic adds make the summation order across workgroups vary from run to
// run (results agree to fp32 rounding); the three-kernel path in k_ffn.hip is
// the deterministic alternative.
#include "ffn_device.h"

namespace m2c {

constexpr int kFuThreads = 512;
constexpr int kFuWaves = kFuThreads / 64;
constexpr int kFuUnits = kFuWaves;  // up-units per block, one per wave

// First item whose cumulative record cost reaches `c` (items are tier-major
// with per-item costs c3, c2, c1).
__device__ __forceinline__ int item_at_cost(long long c, int n3, int n2, int n1, long long c3,
                                            long long c2, long long c1) {
  const long long t3 = n3 * c3, t2 = t3 + n2 * c2;
  long long i;
  if (c <= t3)
    i = (c + c3 - 1) / c3;
  else if (c <= t2)
    i = n3 + (c - t3 + c2 - 1) / c2;
  else
    i = n3 + n2 + (c - t2 + c1 - 1) / c1;
  const int n = n3 + n2 + n1;
  return (int)(i < n ? i : n);
}

// Down data of one neuron for one 8-column chunk, by tier.
template <int TIER> struct DownT;
template <> struct DownT<3> { typedef uint4 T; };     // 8 fp16
template <> struct DownT<2> { typedef uint2 T; };     // 8 int8
template <> struct DownT<1> { typedef uint32_t T; };  // 8 int4

// One block of neurons of one tier: up-units, h, down accumulation.
// SZ: size class, d <= 4096 * SZ (chunks per lane: 2*SZ per unit row, SZ
// output chunks). d <= 8192 (SZ <= 2); larger d use the three-kernel path.
template <int TIER, int SZ>
__device__ __forceinline__ void fused_block(int p, int nb, int d, int G, const uint4* xn,
                                            const uint4* xp, const int32_t* __restrict__ work_slot,
                                            const uint8_t* __restrict__ slots, int64_t slot_bytes,
                                            int n_slots, int lane, int w, float2* s_ab, float* s_h,
                                            float (&acc)[SZ][8]) {
  constexpr int UPI = TIER == 3 ? 4 : TIER == 2 ? 2 : 1;  // units per neuron
  constexpr int NBMAX = kFuUnits / UPI;                   // neurons per block
  constexpr int CPL = 2 * SZ;                             // unit chunks per lane and row
  typedef typename DownT<TIER>::T DT;
  const int ncu = d >> 5;  // 16-byte chunks per row of a unit
  const int cpw = d >> 6;  // 8-column output chunks per wave

  // ---- issue: this wave's up-unit (if any) and every neuron's down data
  const bool has_unit = w < nb * UPI;
  const int item = p + (has_unit ? w / UPI : 0);
  const int part = w % UPI;
  int slot = work_slot[item];
  const bool uok = has_unit && slot >= 0 && slot < n_slots;
  const uint8_t* urec = slots + (int64_t)(uok ? slot : 0) * slot_bytes;
  const int64_t row = TIER == 3 ? 2 * (int64_t)d : TIER == 2 ? d : (d >> 1);
  const int c0 = part * ncu;
  // Loads carry no branches (a load under a per-lane branch becomes its own
  // block and the waitcnt pass drains earlier loads before it): out-of-range
  // lanes read valid memory of slot 0 and their results are discarded.
  uint4 gq[CPL], uq[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int c = min(lane + 64 * i, ncu - 1);
    gq[i] = reinterpret_cast<const uint4*>(urec)[c0 + c];
    uq[i] = reinterpret_cast<const uint4*>(urec + row)[c0 + c];
  }
  DT dv[NBMAX][SZ];
  float dscale[NBMAX][SZ];
#pragma unroll
  for (int k = 0; k < NBMAX; ++k) {
    const int s = work_slot[p + min(k, nb - 1)];
    const bool ok = k < nb && s >= 0 && s < n_slots;
    const uint8_t* rec = slots + (int64_t)(ok ? s : 0) * slot_bytes;
#pragma unroll
    for (int i = 0; i < SZ; ++i) {
      const bool in = ok && lane + 64 * i < cpw;
      const int qc = w * cpw + min(lane + 64 * i, cpw - 1);  // output chunk (8 columns)
      float sc;
      if (TIER == 3) {
        dv[k][i] = *reinterpret_cast<const DT*>(rec + 4 * (int64_t)d + 16 * (int64_t)qc);
        sc = 1.0f;
      } else if (TIER == 2) {
        dv[k][i] = *reinterpret_cast<const DT*>(rec + 2 * (int64_t)d + 8 * (int64_t)qc);
        sc = h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)d + 4 * G + 2 * (qc >> 4)));
      } else {
        dv[k][i] = *reinterpret_cast<const DT*>(rec + (int64_t)d + 4 * (int64_t)qc);
        sc = h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)(d >> 1) + 4 * G +
                                                    2 * (qc >> 4)));
      }
      dscale[k][i] = in ? sc : 0.0f;
    }
  }

  // ---- up-unit partial dot products
  float a = 0.0f, b = 0.0f;
  if (TIER == 3) {
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = min(lane + 64 * i, ncu - 1);
      const uint4 xv = xn[c0 + c];
      const float pa = dot8_f16(gq[i], xv, 0.0f), pb = dot8_f16(uq[i], xv, 0.0f);
      const bool v = uok && lane + 64 * i < ncu;
      a += v ? pa : 0.0f;
      b += v ? pb : 0.0f;
    }
  } else if (TIER == 2) {
    const uint16_t* gs = reinterpret_cast<const uint16_t*>(urec + 3 * (int64_t)d);
    const uint16_t* us = gs + G;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = c0 + min(lane + 64 * i, ncu - 1);
      const float pa = h2f(gs[c >> 3]) * dot16_i8(gq[i], xn[2 * c], xn[2 * c + 1], 0.0f);
      const float pb = h2f(us[c >> 3]) * dot16_i8(uq[i], xn[2 * c], xn[2 * c + 1], 0.0f);
      const bool v = uok && lane + 64 * i < ncu;
      a += v ? pa : 0.0f;
      b += v ? pb : 0.0f;
    }
  } else {
    const uint16_t* gs = reinterpret_cast<const uint16_t*>(urec + 3 * (int64_t)(d >> 1));
    const uint16_t* us = gs + G;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
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
      const bool v = uok && lane + 64 * i < ncu;
      a += v ? h2f(gs[c >> 2]) * pa : 0.0f;
      b += v ? h2f(us[c >> 2]) * pb : 0.0f;
    }
  }
  a = wave_sum(a);
  b = wave_sum(b);
  if (lane == 0) s_ab[w] = make_float2(a, b);
  __syncthreads();
  if (threadIdx.x < nb) {  // h of neuron k from its units, in unit order
    const int k = threadIdx.x;
    float sa = s_ab[k * UPI].x, sb = s_ab[k * UPI].y;
#pragma unroll
    for (int q = 1; q < UPI; ++q) {
      sa += s_ab[k * UPI + q].x;
      sb += s_ab[k * UPI + q].y;
    }
    const int s = work_slot[p + k];
    s_h[k] = (s >= 0 && s < n_slots) ? silu_mul(sa, sb) : 0.0f;
  }
  __syncthreads();

  // ---- down accumulation from the registers
#pragma unroll
  for (int k = 0; k < NBMAX; ++k) {
    if (k < nb) {
      const float hk = s_h[k];
#pragma unroll
      for (int i = 0; i < SZ; ++i) {
        if (dscale[k][i] != 0.0f) {  // 0 for padding lanes and zero-scale groups
          const float c = hk * dscale[k][i];
          if (TIER == 3) {
            const uint4 v = *reinterpret_cast<const uint4*>(&dv[k][i]);
            const uint32_t ws[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              acc[i][2 * e] = fmaf(c, h2f((uint16_t)(ws[e] & 0xffffu)), acc[i][2 * e]);
              acc[i][2 * e + 1] = fmaf(c, h2f((uint16_t)(ws[e] >> 16)), acc[i][2 * e + 1]);
            }
          } else if (TIER == 2) {
            const uint2 v = *reinterpret_cast<const uint2*>(&dv[k][i]);
            const uint32_t ws[2] = {v.x, v.y};
#pragma unroll
            for (int e = 0; e < 2; ++e)
#pragma unroll
              for (int bb = 0; bb < 4; ++bb)
                acc[i][4 * e + bb] =
                    fmaf(c, (float)(int8_t)((ws[e] >> (8 * bb)) & 0xffu), acc[i][4 * e + bb]);
          } else {
            const uint32_t v = *reinterpret_cast<const uint32_t*>(&dv[k][i]);
#pragma unroll
            for (int nbb = 0; nbb < 8; ++nbb) {
              const int nib = (int)((v >> (4 * nbb)) & 0xfu);
              acc[i][nbb] = fmaf(c, (float)(nib >= 8 ? nib - 16 : nib), acc[i][nbb]);
            }
          }
        }
      }
    }
  }
  __syncthreads();  // s_ab / s_h are reused by the next block
}

template <int SZ>
__global__ __launch_bounds__(kFuThreads) void ffn_fused_kernel(
    const uint16_t* __restrict__ x, int d, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ work_slot, const uint8_t* __restrict__ slots, int64_t slot_bytes,
    int cap, int n_slots, float* __restrict__ y) {
  extern __shared__ uint4 xs[];
  __shared__ float2 s_ab[kFuUnits];
  __shared__ float s_h[kFuUnits];
  const int nc8 = d >> 3;
  uint4* xn = xs;        // x in natural order, 8 halves per entry
  uint4* xp = xs + nc8;  // x in INT4 pair order
  for (int c = threadIdx.x; c < nc8; c += blockDim.x) {
    const uint4 v = reinterpret_cast<const uint4*>(x)[c];
    xn[c] = v;
    uint4 q;
    q.x = (v.x & 0xffffu) | (v.z << 16);
    q.y = (v.x >> 16) | (v.z & 0xffff0000u);
    q.z = (v.y & 0xffffu) | (v.w << 16);
    q.w = (v.y >> 16) | (v.w & 0xffff0000u);
    xp[c] = q;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  const int G = d >> 7;
  const long long c3 = 6LL * d, c2 = 3LL * d + 6 * G, c1 = 3LL * d / 2 + 6 * G;
  const long long T = n3 * c3 + n2 * c2 + n1 * c1;
  const int lo = item_at_cost(T * blockIdx.x / gridDim.x, n3, n2, n1, c3, c2, c1);
  const int hi = item_at_cost(T * (blockIdx.x + 1) / gridDim.x, n3, n2, n1, c3, c2, c1);
  float acc[SZ][8];
#pragma unroll
  for (int i = 0; i < SZ; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[i][e] = 0.0f;
  for (int p = lo; p < hi;) {
    if (p < n3) {
      const int q = min(min(p + kFuUnits / 4, hi), n3);
      fused_block<3, SZ>(p, q - p, d, G, xn, xp, work_slot, slots, slot_bytes, n_slots, lane, w,
                         s_ab, s_h, acc);
      p = q;
    } else if (p < n3 + n2) {
      const int q = min(min(p + kFuUnits / 2, hi), n3 + n2);
      fused_block<2, SZ>(p, q - p, d, G, xn, xp, work_slot, slots, slot_bytes, n_slots, lane, w,
                         s_ab, s_h, acc);
      p = q;
    } else {
      const int q = min(p + kFuUnits, hi);
      fused_block<1, SZ>(p, q - p, d, G, xn, xp, work_slot, slots, slot_bytes, n_slots, lane, w,
                         s_ab, s_h, acc);
      p = q;
    }
  }
  if (lo == hi) return;
  // Partial row -> LDS (over x, which is no longer needed), then added into
  // y with consecutive lanes on consecutive columns, so each atomic
  // instruction covers 256 contiguous bytes.
  float* row = reinterpret_cast<float*>(xs);
  const int cpw = d >> 6;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < SZ; ++i) {
    if (lane + 64 * i < cpw) {
      float* rc = row + 8 * (w * cpw + lane + 64 * i);
#pragma unroll
      for (int e = 0; e < 8; ++e) rc[e] = acc[i][e];
    }
  }
  __syncthreads();
  for (int j = threadIdx.x; j < d; j += kFuThreads) atomicAdd(y + j, row[j]);
}

hipError_t launch_ffn_fused(m2c_layer* L, const uint16_t* x, const uint8_t* plan, float* y,
                            hipStream_t stream) {
  const int d = L->desc.d_model;
  const m2c_plan_layout& lay = L->layout;
  const int32_t* counts = reinterpret_cast<const int32_t*>(plan + lay.counts);
  const int32_t* work_slot = reinterpret_cast<const int32_t*>(plan + lay.work_slot);
  const int64_t sb = L->info.slot_bytes;
  const int n_slots = L->desc.cache_slots + L->S;
  // as many workgroups as fit at once (two per CU at d <= 4096, one above:
  // register bound), but no more than there are blocks of work
  int blocks = (d <= 4096 ? 2 : 1) * L->num_cus;
  const int max_blocks = (4 * L->cap + kFuUnits - 1) / kFuUnits;
  if (blocks > max_blocks) blocks = max_blocks > 0 ? max_blocks : 1;
  const size_t lds = (size_t)d * 4;
  if (d <= 4096)
    hipLaunchKernelGGL(ffn_fused_kernel<1>, dim3(blocks), dim3(kFuThreads), lds, stream, x, d,
                       counts, work_slot, L->slots, sb, L->cap, n_slots, y);
  else
    hipLaunchKernelGGL(ffn_fused_kernel<2>, dim3(blocks), dim3(kFuThreads), lds, stream, x, d,
                       counts, work_slot, L->slots, sb, L->cap, n_slots, y);
  return hipGetLastError();
}

}  // namespace m2c
