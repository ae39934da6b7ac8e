// Cache plan: resolves one step's active neurons against the layer's
// isolated HBM cache unit (Sec. 5.3) with LRU replacement of neurons
// (Sec. 1, Sec. 6.4). One workgroup does the whole step:
//
//   A  required set R = neurons with tier > 0 in some row (max tier, row
//      mask), compacted in ascending id by a block scan; resident ones are
//      HIT (same tier) or REFILL (other tier, refilled in place) and are
//      stamped last_use = step, which also marks them "touched".
//   C  victims: the LRU order of the slots is kept explicitly as a
//      permutation sorted by (last_use, slot). The untouched slots, in that
//      order, are the victims; the j-th NEW neuron (ascending id) takes the
//      j-th of them, NEW neurons beyond that go to staging slots (bypass).
//   D  new order = untouched non-victims in their old order, then every
//      touched slot in slot order (they all now share last_use = step, the
//      largest value), which keeps the permutation sorted.
//   E  fill list (every non-HIT, ascending id) and the FFN work list
//      (tier-major FP16, INT8, INT4; ascending id inside a tier).
// Ranks in id / position order come from block scans over contiguous
// per-thread ranges.
#include "m2c_internal.h"

namespace m2c {

constexpr int kPlanThreads = 1024;

struct PlanPtrs {
  int32_t* counts;
  int32_t* req_ids;
  uint8_t* req_tier;
  uint8_t* req_hit;
  int32_t* req_slot;
  uint32_t* req_mask;
  int32_t* fill_ids;
  uint8_t* fill_tier;
  int32_t* fill_slot;
  int32_t* evicted_ids;
  int32_t* work_slot;
  uint32_t* work_mask;
};

__device__ __forceinline__ void thread_range(int n, int& lo, int& hi) {
  const int per = (n + kPlanThreads - 1) / kPlanThreads;
  lo = threadIdx.x * per;
  if (lo > n) lo = n;
  hi = lo + per;
  if (hi > n) hi = n;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(const uint8_t* __restrict__ tier_map,
                                                            int B, int d_ff, int C, int cap,
                                                            int step, DeviceState st, PlanPtrs P) {
  __shared__ unsigned long long scan64[kPlanThreads / 64 + 1];
  __shared__ uint32_t scan32[kPlanThreads / 64 + 1];
  __shared__ int sh_hit, sh_refill, sh_empty;
  const int tid = threadIdx.x;
  if (tid == 0) {
    sh_hit = 0;
    sh_refill = 0;
    sh_empty = 0;
  }
  // ---------------- A: required set, hits, refills
  int i0, i1;
  thread_range(d_ff, i0, i1);
  uint32_t nreq = 0, nnew = 0;
  unsigned long long tiers = 0;  // 21-bit counts: FP16 | INT8 << 21 | INT4 << 42
  for (int i = i0; i < i1; ++i) {
    int t = 0;
    for (int b = 0; b < B; ++b) {
      const int tb = tier_map[(int64_t)b * d_ff + i];
      t = tb > t ? tb : t;
    }
    t = t > 3 ? 3 : t;  // codes above FP16 read as FP16
    if (t) {
      ++nreq;
      tiers += 1ull << (21 * (3 - t));
      if (st.slot_of[i] < 0) ++nnew;
    }
  }
  unsigned long long tot;
  const unsigned long long preA = block_exclusive_scan<unsigned long long>(
      (unsigned long long)nreq | ((unsigned long long)nnew << 32), scan64, &tot);
  const int NREQ = (int)(tot & 0xffffffffu), NNEW = (int)(tot >> 32);
  unsigned long long totT;
  const unsigned long long preT = block_exclusive_scan<unsigned long long>(tiers, scan64, &totT);
  const int N3 = (int)(totT & 0x1fffff), N2 = (int)((totT >> 21) & 0x1fffff),
            N1 = (int)((totT >> 42) & 0x1fffff);
  if (NREQ > cap) {
    // More active neurons than the layer was sized for (a tier map that did
    // not come from m2c_predict_rank with k <= k_max): write an empty plan
    // with the overflow flagged and leave the cache untouched.
    if (tid == 0) {
      for (int q = 0; q < M2C_NCOUNTS; ++q) P.counts[q] = 0;
      P.counts[M2C_NCOUNTS - 1] = NREQ;
      atomicOr(st.status, M2C_STATUS_PLAN_OVERFLOW);
    }
    return;
  }
  {
    int pos = (int)(preA & 0xffffffffu), pnew = (int)(preA >> 32);
    int r3 = (int)(preT & 0x1fffff), r2 = N3 + (int)((preT >> 21) & 0x1fffff),
        r1 = N3 + N2 + (int)((preT >> 42) & 0x1fffff);
    int hits = 0, refills = 0;
    for (int i = i0; i < i1; ++i) {
      int t = 0;
      uint32_t m = 0;
      for (int b = 0; b < B; ++b) {
        const int tb = tier_map[(int64_t)b * d_ff + i];
        if (tb) m |= 1u << b;
        t = tb > t ? tb : t;
      }
      t = t > 3 ? 3 : t;
      if (!t) continue;
      P.req_ids[pos] = i;
      P.req_tier[pos] = (uint8_t)t;
      P.req_mask[pos] = m;
      st.work_pos[pos] = t == 3 ? r3++ : t == 2 ? r2++ : r1++;
      const int s = st.slot_of[i];
      if (s >= 0) {
        const bool same = st.slot_tier[s] == t;
        P.req_hit[pos] = same ? 1 : 2;
        P.req_slot[pos] = s;
        st.slot_last[s] = step;
        if (!same) st.slot_tier[s] = (uint8_t)t;
        hits += same;
        refills += !same;
      } else {
        st.new_pos[pnew++] = pos;
      }
      ++pos;
    }
    if (hits) atomicAdd(&sh_hit, hits);
    if (refills) atomicAdd(&sh_refill, refills);
  }
  __syncthreads();
  // ---------------- C: victims in LRU order
  const int cur = *st.lru_cur;
  const int32_t* lru_in = st.lru + (int64_t)cur * C;
  int32_t* lru_out = st.lru + (int64_t)(1 - cur) * C;
  int p0, p1;
  thread_range(C, p0, p1);
  uint32_t nunt = 0;
  for (int p = p0; p < p1; ++p) nunt += st.slot_last[lru_in[p]] != step;
  uint32_t tot32;
  uint32_t u = block_exclusive_scan<uint32_t>(nunt, scan32, &tot32);
  const int NUNT = (int)tot32;
  const int NV = NNEW < NUNT ? NNEW : NUNT;
  {
    int empties = 0;
    for (int p = p0; p < p1; ++p) {
      const int s = lru_in[p];
      if (st.slot_last[s] == step) continue;
      if ((int)u < NV) {
        const int old = st.slot_key[s];
        st.vict_slot[u] = s;
        st.vict_old[u] = old;
        empties += old < 0;
        st.slot_last[s] = step;
      } else {
        lru_out[u - NV] = s;
      }
      ++u;
    }
    if (empties) atomicAdd(&sh_empty, empties);
  }
  __syncthreads();
  const int NEMPTY = sh_empty;
  // ---------------- C2: NEW neurons take their victims or a staging slot
  for (int j = tid; j < NNEW; j += kPlanThreads) {
    const int pos = st.new_pos[j];
    const int i = P.req_ids[pos];
    if (j < NV) {
      const int s = st.vict_slot[j];
      const int old = st.vict_old[j];
      if (old >= 0) {
        st.slot_of[old] = -1;
        P.evicted_ids[j - NEMPTY] = old;
      }
      st.slot_of[i] = s;
      st.slot_key[s] = i;
      st.slot_tier[s] = P.req_tier[pos];
      P.req_slot[pos] = s;
      P.req_hit[pos] = 0;
    } else {
      P.req_slot[pos] = C + (j - NV);
      P.req_hit[pos] = 3;
    }
  }
  __syncthreads();
  // ---------------- D: touched slots go to the end of the order, by slot id
  {
    uint32_t ntch = 0;
    for (int s = p0; s < p1; ++s) ntch += st.slot_last[s] == step;
    uint32_t r = block_exclusive_scan<uint32_t>(ntch, scan32, &tot32);
    int pos = NUNT - NV + (int)r;
    for (int s = p0; s < p1; ++s)
      if (st.slot_last[s] == step) lru_out[pos++] = s;
  }
  // ---------------- E: fill list and FFN work list
  int q0, q1;
  thread_range(NREQ, q0, q1);
  uint32_t nf = 0;
  unsigned long long ftiers = 0;
  for (int q = q0; q < q1; ++q) {
    if (P.req_hit[q] != 1) {
      ++nf;
      ftiers += 1ull << (21 * (3 - P.req_tier[q]));
    }
  }
  uint32_t f = block_exclusive_scan<uint32_t>(nf, scan32, &tot32);
  const int NF = (int)tot32;
  unsigned long long ftot;
  block_exclusive_scan<unsigned long long>(ftiers, scan64, &ftot);
  for (int q = q0; q < q1; ++q) {
    const int ws = P.req_slot[q];
    const int w = st.work_pos[q];
    P.work_slot[w] = ws;
    P.work_mask[w] = P.req_mask[q];
    if (P.req_hit[q] != 1) {
      P.fill_ids[f] = P.req_ids[q];
      P.fill_tier[f] = P.req_tier[q];
      P.fill_slot[f] = ws;
      ++f;
    }
  }
  if (tid == 0) {
    const int F3 = (int)(ftot & 0x1fffff), F2 = (int)((ftot >> 21) & 0x1fffff),
              F1 = (int)((ftot >> 42) & 0x1fffff);
    int32_t c[M2C_NCOUNTS] = {0};
    c[M2C_CNT_REQ] = NREQ;
    c[M2C_CNT_HIT] = sh_hit;
    c[M2C_CNT_REFILL] = sh_refill;
    c[M2C_CNT_NEW] = NV;
    c[M2C_CNT_BYPASS] = NNEW - NV;
    c[M2C_CNT_EVICT] = NV - NEMPTY;
    c[M2C_CNT_FILL] = NF;
    c[M2C_CNT_REQ_FP16] = N3;
    c[M2C_CNT_REQ_INT8] = N2;
    c[M2C_CNT_REQ_INT4] = N1;
    c[M2C_CNT_FILL_FP16] = F3;
    c[M2C_CNT_FILL_INT8] = F2;
    c[M2C_CNT_FILL_INT4] = F1;
    for (int q = 0; q < M2C_NCOUNTS; ++q) P.counts[q] = c[q];
    *st.lru_cur = 1 - cur;
    // cumulative statistics: plans, req, hit, refill, new, bypass, evict,
    // fills by tier [7..9] = INT4, INT8, FP16
    atomicAdd(&st.stats[0], 1ull);
    atomicAdd(&st.stats[1], (unsigned long long)NREQ);
    atomicAdd(&st.stats[2], (unsigned long long)sh_hit);
    atomicAdd(&st.stats[3], (unsigned long long)sh_refill);
    atomicAdd(&st.stats[4], (unsigned long long)NV);
    atomicAdd(&st.stats[5], (unsigned long long)(NNEW - NV));
    atomicAdd(&st.stats[6], (unsigned long long)(NV - NEMPTY));
    atomicAdd(&st.stats[7], (unsigned long long)F1);
    atomicAdd(&st.stats[8], (unsigned long long)F2);
    atomicAdd(&st.stats[9], (unsigned long long)F3);
  }
}

__global__ void reset_kernel(DeviceState st, int d_ff, int C) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  const int n = gridDim.x * blockDim.x;
  for (int i = idx; i < d_ff; i += n) st.slot_of[i] = -1;
  for (int s = idx; s < C; s += n) {
    st.slot_key[s] = -1;
    st.slot_tier[s] = 0;
    st.slot_last[s] = -1;
    st.lru[s] = s;
    st.lru[C + s] = s;
  }
  if (idx == 0) *st.lru_cur = 0;
  if (idx < 16) st.stats[idx] = 0;
}

hipError_t launch_plan(m2c_layer* L, const uint8_t* tier_map, int batch, int step, uint8_t* plan,
                       hipStream_t stream) {
  const m2c_plan_layout& lay = L->layout;
  PlanPtrs P;
  P.counts = reinterpret_cast<int32_t*>(plan + lay.counts);
  P.req_ids = reinterpret_cast<int32_t*>(plan + lay.req_ids);
  P.req_tier = plan + lay.req_tier;
  P.req_hit = plan + lay.req_hit;
  P.req_slot = reinterpret_cast<int32_t*>(plan + lay.req_slot);
  P.req_mask = reinterpret_cast<uint32_t*>(plan + lay.req_mask);
  P.fill_ids = reinterpret_cast<int32_t*>(plan + lay.fill_ids);
  P.fill_tier = plan + lay.fill_tier;
  P.fill_slot = reinterpret_cast<int32_t*>(plan + lay.fill_slot);
  P.evicted_ids = reinterpret_cast<int32_t*>(plan + lay.evicted_ids);
  P.work_slot = reinterpret_cast<int32_t*>(plan + lay.work_slot);
  P.work_mask = reinterpret_cast<uint32_t*>(plan + lay.work_mask);
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, tier_map, batch,
                     L->desc.d_ff, L->desc.cache_slots, L->cap, step, L->st, P);
  return hipGetLastError();
}

hipError_t launch_reset(m2c_layer* L, hipStream_t stream) {
  const int n = L->desc.d_ff > L->desc.cache_slots ? L->desc.d_ff : L->desc.cache_slots;
  int blocks = (n + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(reset_kernel, dim3(blocks), dim3(256), 0, stream, L->st, L->desc.d_ff,
                     L->desc.cache_slots);
  return hipGetLastError();
}

}  // namespace m2c
