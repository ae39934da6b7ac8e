// Task geometry of the one-launch batch-1 FFN (k_ffn_fused.hip): the task
// sizes, the launch order of the six task regions, the task of a workgroup
// id, and the task table the cache plan writes for it. Shared by the FFN
// kernel and the plan kernels that write the table.
#pragma once

#include "ffn_device.h"

namespace m2c {

#ifndef M2C_FFN_THREADS
#define M2C_FFN_THREADS 256
#endif
constexpr int kFT = M2C_FFN_THREADS;     // threads per workgroup
constexpr int kFWaves = kFT / 64;
constexpr int kFL = 8;                   // 16-byte data loads per lane and task
constexpr int kFSW = 512;                // down tasks: output columns per slice
constexpr int kFLPN = kFSW / 32;         // lanes per neuron row of a slice
constexpr int kFNPR = kFT / kFLPN;       // neurons per round of a down task
constexpr int kFMaxItems = kFL * kFNPR;  // most work items of one task (INT4 down)
// Rounds of kFNPR neurons per down task by tier (INT4, INT8, FP16): one
// load per lane and round for INT4, two for INT8, four for FP16.
constexpr int kDnRounds1 = kFL, kDnRounds2 = kFL / 2, kDnRounds3 = kFL / 4;
constexpr int kFSpin = 1 << 16;          // polls of one h word before giving up
constexpr float kTwo24 = 16777216.0f;
static_assert(kFMaxItems <= kFT, "one slot id / h word per thread");
// The task table in a plan: task count and zero slot (16 bytes), one 32-byte
// header per workgroup, then kTaskIds slot ids per workgroup from a 256-byte
// boundary.
constexpr int kTaskIds = kFL * kFNPR;
inline int64_t task_ids_offset(int grid) { return (16 + 32 * (int64_t)grid + 255) / 256 * 256; }
static_assert(kFLPN == 16, "the fold pairs lanes 16 and 32 apart");
static_assert(kFSW % kFT == 0, "the cross-wave fold gives each thread whole columns of the slice");

struct FMap {
  int n3, n2, n1;  // work items by tier
  int w1, w2, w3;  // h tasks by tier (INT4, INT8, FP16)
  int n_slices;
  int e[6];        // ends of the six task regions in launch order
};

struct FTask {
  int kind;  // 0 none, 1 h, 2 down
  int tier;
  int lo, hi;
  int slice;
};

// K: 16-byte loads per lane and unit (a unit is d bytes of a neuron's gate and
// up rows); a wave takes kFL / K units of an h task.
// Launch order of the six task regions: (kind, tier) per region.
constexpr int kOrderKind[6] = {1, 1, 1, 2, 2, 2};
constexpr int kOrderTier[6] = {1, 2, 3, 1, 2, 3};

template <int K>
__device__ __forceinline__ FMap make_map_n(int n3, int n2, int n1, int d) {
  constexpr int U = kFWaves * (kFL / K);  // units per h task
  FMap m;
  m.n3 = n3;
  m.n2 = n2;
  m.n1 = n1;
  m.w1 = (m.n1 + U - 1) / U;
  m.w2 = (m.n2 + U / 2 - 1) / (U / 2);
  m.w3 = (m.n3 + U / 4 - 1) / (U / 4);
  m.n_slices = (d + kFSW - 1) / kFSW;
  const int u1 = (m.n1 + kDnRounds1 * kFNPR - 1) / (kDnRounds1 * kFNPR);
  const int u2 = (m.n2 + kDnRounds2 * kFNPR - 1) / (kDnRounds2 * kFNPR);
  const int u3 = (m.n3 + kDnRounds3 * kFNPR - 1) / (kDnRounds3 * kFNPR);
  int end = 0;
#pragma unroll
  for (int r = 0; r < 6; ++r) {
    const int tr = kOrderTier[r];
    end += kOrderKind[r] == 1 ? (tr == 1 ? m.w1 : tr == 2 ? m.w2 : m.w3)
                              : (tr == 1 ? u1 : tr == 2 ? u2 : u3) * m.n_slices;
    m.e[r] = end;
  }
  return m;
}
template <int K>
__device__ __forceinline__ FMap make_map(const int32_t* counts, int cap, int d) {
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  return make_map_n<K>(n3, n2, n1, d);
}

// Task t in launch order. Work items are tier-major in the plan: FP16, INT8,
// INT4.
template <int K>
__device__ __forceinline__ FTask decode(const FMap& m, int t) {
  constexpr int U = kFWaves * (kFL / K);
  FTask k;
  k.kind = 0;
  k.tier = 1;
  k.lo = k.hi = 0;
  k.slice = 0;
  // region by comparisons (no indexed array: it would live in scratch memory)
  int kind = 0, tier = 1, start = 0;
#pragma unroll
  for (int r = 5; r >= 0; --r) {
    const int lo_r = r ? m.e[r - 1] : 0;
    if (t >= lo_r && t < m.e[r]) {
      kind = kOrderKind[r];
      tier = kOrderTier[r];
      start = lo_r;
    }
  }
  if (kind == 0) return k;
  const int q = t - start;
  k.tier = tier;
  // by value (a select between fields would index a stack copy of the map)
  const int i1 = tier == 1, i2 = tier == 2, i3 = tier == 3;
  const int base = i1 * (m.n3 + m.n2) + i2 * m.n3;
  const int n = i1 * m.n1 + i2 * m.n2 + i3 * m.n3;
  if (kind == 1) {
    k.kind = 1;
    const int per = tier == 1 ? U : tier == 2 ? U / 2 : U / 4;
    k.lo = base + per * q;
    k.hi = base + min(per * (q + 1), n);
  } else {
    k.kind = 2;
    const int per = (tier == 1 ? kDnRounds1 : tier == 2 ? kDnRounds2 : kDnRounds3) * kFNPR;
    // Runs in blocks of 8, slice-major within a block: workgroup b runs on
    // XCD b % 8, so all slices of a run (which read the same scale lines of
    // the run's records) land on one XCD and its L2.
    const int nr = (n + per - 1) / per;
    const int blk = q / (8 * m.n_slices);
    const int within = q - blk * 8 * m.n_slices;
    const int nb = min(8, nr - 8 * blk);
    k.slice = within / nb;
    const int run = 8 * blk + (within - k.slice * nb);
    k.lo = base + per * run;
    k.hi = base + min(per * (run + 1), n);
  }
  return k;
}


// The task table, one wave per task: the 32-byte header {kind | tier << 8,
// first work item, items, slice, then the tier pool's byte offset, first slot
// id, slot count, record stride} and the slot ids in the order the FFN's
// waves read them (a down task's items in work order; an h task's units at
// entry (uw / 4) kFNPR + 4 w + uw % 4 for unit w UW + uw). The table starts
// with the task count and the zero slot's byte offset. wave / n_waves: this
// wave among those that write the table; slot(e): the slot of work item e.
template <int K, typename SlotOf>
__device__ __forceinline__ void write_task_table(const FMap& m, int grid, const SlotMap& map,
                                                 int32_t* __restrict__ tasks,
                                                 int32_t* __restrict__ task_ids, int wave,
                                                 int n_waves, SlotOf slot) {
  constexpr int UW = kFL / K;
  const int n_tasks = m.e[5] < grid ? m.e[5] : grid;
  if (wave == 0 && (threadIdx.x & 63) == 0) {
    tasks[0] = n_tasks;
    tasks[1] = (int32_t)map.zero;
  }
  const int lane = threadIdx.x & 63;
  for (int t = wave; t < n_tasks; t += n_waves) {
    const FTask k = decode<K>(m, t);
    const int n = k.hi - k.lo;
    if (lane == 0) {
      const int tr = k.tier;
      int4* h = reinterpret_cast<int4*>(tasks + 4) + 2 * t;
      h[0] = make_int4(k.kind | (tr << 8), k.lo, n, k.slice);
      h[1] = make_int4((int)map.base[tr], map.first[tr], map.count[tr], (int)map.stride[tr]);
    }
    int32_t* out = task_ids + (int64_t)t * kTaskIds;
    if (k.kind == 2) {
      for (int e = lane; e < n; e += 64) out[e] = slot(k.lo + e);
    } else if (k.kind == 1) {
      const int upi = k.tier == 3 ? 4 : k.tier == 2 ? 2 : 1;
      const int item = lane / upi;  // unit lane of the task
      if (lane < kFWaves * UW && item < n) {
        const int w = lane / UW, uw = lane % UW;
        out[(uw >> 2) * kFNPR + 4 * w + (uw & 3)] = slot(k.lo + item);
      }
    }
  }
}

}  // namespace m2c
