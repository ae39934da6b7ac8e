// Cache fill: copies every missing neuron record, at its tier, from the
// pinned host-DRAM store into its HBM slot (Sec. 1 "Selective Loading into
// GPU"; Sec. 5.3 loads only the neurons that differ between tokens).
//
// The fill list lives in device memory (written by the plan kernel), so the
// copy is a device gather kernel that reads host memory over the host link:
// no device-to-host round trip is needed to learn what to copy, and the
// whole step stays on the GPU's queues. One workgroup copies one record at a
// time with 16-byte loads, four in flight per thread.
//
// A fill to INT8 / INT4 of a neuron whose slot holds its FP16 record (a
// neuron that fell out of the FP16 tier) is made on the GPU instead: the
// workgroup stages the FP16 record's rows in LDS and quantizes them over the
// record with the create-time quantizer, which yields the store's record byte
// for byte and takes nothing from the host link. The kernel keeps, per slot,
// which record (neuron and tier) it last wrote there, and derives only from
// bytes that are the same neuron's FP16 record: a fill run twice on one plan
// copies the second time instead of quantizing the INT8 / INT4 bytes again.
#include "quant_device.h"

namespace m2c {

#ifndef M2C_FILL_BLOCKS
#define M2C_FILL_BLOCKS 32
#endif
constexpr int kFillThreads = 256;
constexpr int kFillBlocks = M2C_FILL_BLOCKS;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct FillSrc {
  const uint8_t* host[4];
  int64_t stride[4];
};

__global__ __launch_bounds__(kFillThreads) void fill_kernel(const int32_t* __restrict__ counts,
                                                            const int32_t* __restrict__ fill_ids,
                                                            const uint8_t* __restrict__ fill_tier,
                                                            const int32_t* __restrict__ fill_slot,
                                                            const uint8_t* __restrict__ fill_from,
                                                            int32_t* __restrict__ slot_rec,
                                                            FillSrc src, uint8_t* __restrict__ slots,
                                                            SlotMap map, int cap, int d_ff, int d,
                                                            int n_slots) {
  extern __shared__ u32x4 stage[];  // 2 d + 6 d / 128 bytes: one FP16 row and the scales
  int n = counts[M2C_CNT_FILL];
  n = n < 0 ? 0 : n > cap ? cap : n;
  for (int e = blockIdx.x; e < n; e += gridDim.x) {
    const int t = fill_tier[e];
    const int id = fill_ids[e], slot = fill_slot[e];
    // plans written by m2c_cache_plan always pass; anything else is skipped
    // (workgroup-uniform: every thread reads the same entry), as is a slot
    // outside the pool of the fill's tier
    if (t < 1 || t > 3 || id < 0 || id >= d_ff || slot < 0 || slot >= n_slots) continue;
    if ((uint32_t)(slot - map.first[t]) >= (uint32_t)map.count[t]) continue;
    const bool derive = fill_from[e] == 3 && t < 3 && slot_rec[slot] == 4 * id + 3;
    __syncthreads();  // every thread has read slot_rec[slot] before it changes
    if (threadIdx.x == 0) slot_rec[slot] = 4 * id + t;
    // where the slot's record starts (in the pool of the fill's tier)
    uint8_t* rec = slots + map.base[t] + (int64_t)(slot - map.first[t]) * map.stride[t];
    if (derive) {
      // Derive in place (uniform over the workgroup), one d-element row at a
      // time: row v's codes land below byte 2 d (v + 1), which the staged
      // rows 0..v cover; the scales, which overlap the up row's FP16 bytes
      // for INT8, are written last.
      uint16_t* sc_stage = reinterpret_cast<uint16_t*>(stage + ((2 * d) >> 4));
      const uint32_t* w = reinterpret_cast<const uint32_t*>(stage);
      const int G = d >> 7, lane = threadIdx.x & 63;
      for (int v = 0; v < 3; ++v) {
        const u32x4* row = reinterpret_cast<const u32x4*>(rec + (int64_t)v * 2 * d);
        for (int c = threadIdx.x; c < (2 * d) >> 4; c += kFillThreads) stage[c] = row[c];
        __syncthreads();
        for (int g = threadIdx.x >> 6; g < G; g += kFillThreads / 64) {  // one wave per group
          const uint32_t pair = w[g * 64 + lane];
          const float amax = group_amax(pair);
          uint16_t sc;
          if (t == 2)
            *reinterpret_cast<uint16_t*>(rec + (int64_t)v * d + g * 128 + 2 * lane) =
                int8_codes(pair, amax, sc);
          else
            rec[(int64_t)v * (d / 2) + g * 64 + lane] = int4_codes(pair, amax, sc);
          if (lane == 0) sc_stage[v * G + g] = sc;
        }
        __syncthreads();  // the staging area takes the next row
      }
      const int64_t sbase = t == 2 ? 3 * (int64_t)d : 3 * (int64_t)(d / 2);
      for (int q = threadIdx.x; q < 3 * G; q += kFillThreads)
        *reinterpret_cast<uint16_t*>(rec + sbase + 2 * q) = sc_stage[q];
      __syncthreads();  // and the scales the next record's
      continue;
    }
    const int64_t bytes = src.stride[t];  // multiple of 16, <= slot_bytes
    const u32x4* s = reinterpret_cast<const u32x4*>(src.host[t] + (int64_t)id * bytes);
    u32x4* dst = reinterpret_cast<u32x4*>(rec);
    const int nvec = (int)(bytes >> 4);
    int v = threadIdx.x;
    for (; v + 3 * kFillThreads < nvec; v += 4 * kFillThreads) {
      // host records are read once: non-temporal loads keep them out of the caches
      const u32x4 r0 = __builtin_nontemporal_load(s + v);
      const u32x4 r1 = __builtin_nontemporal_load(s + v + kFillThreads);
      const u32x4 r2 = __builtin_nontemporal_load(s + v + 2 * kFillThreads);
      const u32x4 r3 = __builtin_nontemporal_load(s + v + 3 * kFillThreads);
      dst[v] = r0;
      dst[v + kFillThreads] = r1;
      dst[v + 2 * kFillThreads] = r2;
      dst[v + 3 * kFillThreads] = r3;
    }
    for (; v < nvec; v += kFillThreads) dst[v] = __builtin_nontemporal_load(s + v);
  }
}

hipError_t launch_fill(const m2c_layer* L, const uint8_t* plan, const uint8_t* const host[4],
                       hipStream_t stream) {
  const m2c_plan_layout& lay = L->layout;
  FillSrc src;
  for (int t = 0; t < 4; ++t) {
    src.host[t] = host[t];
    src.stride[t] = t ? L->info.record_stride[t] : 0;
  }
  // The host link, not the CUs, bounds a fill: 32 workgroups keep 512 KB of
  // reads in flight, enough for the link's rate. More in flight does not
  // speed the fill, and the kernels that overlap it (predictor, select, plan,
  // FFN) wait longer for memory: their requests queue behind the host reads.
  // A stack of 70B layers decodes 9% faster with 32 workgroups than with 64,
  // 15% faster than with 128 (16 and 8 starve the link).
  int blocks = kFillBlocks;
  if (blocks > L->cap) blocks = L->cap > 0 ? L->cap : 1;
  const int d = L->desc.d_model;
  const size_t lds = (size_t)2 * d + 6 * (d / 128);
  hipLaunchKernelGGL(fill_kernel, dim3(blocks), dim3(kFillThreads), lds, stream,
                     reinterpret_cast<const int32_t*>(plan + lay.counts),
                     reinterpret_cast<const int32_t*>(plan + lay.fill_ids), plan + lay.fill_tier,
                     reinterpret_cast<const int32_t*>(plan + lay.fill_slot), plan + lay.fill_from,
                     L->st.slot_rec, src, L->slots, L->map, L->cap, L->desc.d_ff, d,
                     L->desc.cache_slots + L->S);
  return hipGetLastError();
}

// Test support: 0xFF over every slot the fill of a plan writes, except the
// slots a fill may derive from (fill_from == 3, INT8 / INT4), whose FP16
// bytes the fill reads.
__global__ __launch_bounds__(kFillThreads) void poison_kernel(const int32_t* __restrict__ counts,
                                                              const uint8_t* __restrict__ fill_tier,
                                                              const int32_t* __restrict__ fill_slot,
                                                              const uint8_t* __restrict__ fill_from,
                                                              uint8_t* __restrict__ slots,
                                                              SlotMap map, int cap, int n_slots) {
  int n = counts[M2C_CNT_FILL];
  n = n < 0 ? 0 : n > cap ? cap : n;
  const u32x4 ones = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
  for (int e = blockIdx.x; e < n; e += gridDim.x) {
    const int t = fill_tier[e], slot = fill_slot[e];
    if (t < 1 || t > 3 || slot < 0 || slot >= n_slots || (fill_from[e] == 3 && t < 3)) continue;
    if ((uint32_t)(slot - map.first[t]) >= (uint32_t)map.count[t]) continue;
    u32x4* dst = reinterpret_cast<u32x4*>(slots + map.base[t] +
                                          (int64_t)(slot - map.first[t]) * map.stride[t]);
    for (int v = threadIdx.x; v < (int)(map.stride[t] >> 4); v += kFillThreads) dst[v] = ones;
  }
}

hipError_t launch_poison_fill_slots(const m2c_layer* L, const uint8_t* plan, hipStream_t stream) {
  const m2c_plan_layout& lay = L->layout;
  hipLaunchKernelGGL(poison_kernel, dim3(kFillBlocks), dim3(kFillThreads), 0, stream,
                     reinterpret_cast<const int32_t*>(plan + lay.counts), plan + lay.fill_tier,
                     reinterpret_cast<const int32_t*>(plan + lay.fill_slot), plan + lay.fill_from,
                     L->slots, L->map, L->cap, L->desc.cache_slots + L->S);
  return hipGetLastError();
}

}  // namespace m2c
