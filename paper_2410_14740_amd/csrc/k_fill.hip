// Cache fill: copies every missing neuron record, at its tier, from the
// pinned host-DRAM store into its HBM slot (Sec. 1 "Selective Loading into
// GPU"; Sec. 5.3 loads only the neurons that differ between tokens).
//
// The fill list lives in device memory (written by the plan kernel), so the
// copy is a device gather kernel that reads host memory over the host link:
// no device-to-host round trip is needed to learn what to copy, and the
// whole step stays on the GPU's queues. One workgroup copies one record at a
// time with 16-byte loads, four in flight per thread.
#include "m2c_internal.h"

namespace m2c {

#ifndef M2C_FILL_BLOCKS
#define M2C_FILL_BLOCKS 64
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
                                                            FillSrc src, uint8_t* __restrict__ slots,
                                                            int64_t slot_bytes, int cap, int d_ff,
                                                            int n_slots) {
  int n = counts[M2C_CNT_FILL];
  n = n < 0 ? 0 : n > cap ? cap : n;
  for (int e = blockIdx.x; e < n; e += gridDim.x) {
    const int t = fill_tier[e];
    const int id = fill_ids[e], slot = fill_slot[e];
    // plans written by m2c_cache_plan always pass; anything else is skipped
    if (t < 1 || t > 3 || id < 0 || id >= d_ff || slot < 0 || slot >= n_slots) continue;
    const int64_t bytes = src.stride[t];  // multiple of 16, <= slot_bytes
    const u32x4* s = reinterpret_cast<const u32x4*>(src.host[t] + (int64_t)id * bytes);
    u32x4* dst = reinterpret_cast<u32x4*>(slots + (int64_t)slot * slot_bytes);
    const int nvec = (int)(bytes >> 4);
    int v = threadIdx.x;
    for (; v + 3 * kFillThreads < nvec; v += 4 * kFillThreads) {
      // host records are read once: non-temporal loads keep them out of the caches
      const u32x4 a = __builtin_nontemporal_load(s + v);
      const u32x4 b = __builtin_nontemporal_load(s + v + kFillThreads);
      const u32x4 c = __builtin_nontemporal_load(s + v + 2 * kFillThreads);
      const u32x4 d = __builtin_nontemporal_load(s + v + 3 * kFillThreads);
      dst[v] = a;
      dst[v + kFillThreads] = b;
      dst[v + 2 * kFillThreads] = c;
      dst[v + 3 * kFillThreads] = d;
    }
    for (; v < nvec; v += kFillThreads) dst[v] = __builtin_nontemporal_load(s + v);
  }
}

hipError_t launch_fill(const m2c_layer* L, const uint8_t* plan, hipStream_t stream) {
  const m2c_plan_layout& lay = L->layout;
  FillSrc src;
  for (int t = 0; t < 4; ++t) {
    src.host[t] = L->store->host[t];
    src.stride[t] = L->store->stride[t];
  }
  // The host link, not the CUs, bounds a fill: 64 workgroups keep about
  // 1 MB of reads in flight, enough to cover its latency, while leaving the
  // CUs and the memory system's request queues to the kernels that overlap.
  int blocks = kFillBlocks;
  if (blocks > L->cap) blocks = L->cap > 0 ? L->cap : 1;
  hipLaunchKernelGGL(fill_kernel, dim3(blocks), dim3(kFillThreads), 0, stream,
                     reinterpret_cast<const int32_t*>(plan + lay.counts),
                     reinterpret_cast<const int32_t*>(plan + lay.fill_ids), plan + lay.fill_tier,
                     reinterpret_cast<const int32_t*>(plan + lay.fill_slot), src, L->slots,
                     (int64_t)L->info.slot_bytes, L->cap, L->desc.d_ff,
                     L->desc.cache_slots + L->S);
  return hipGetLastError();
}

}  // namespace m2c
