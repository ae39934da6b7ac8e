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
//
// Three launches build this plan: plan_kernel (any d_ff, the steps above
// over per-thread ranges), plan_fast_kernel (d_ff <= 32768, the same steps
// as coalesced sweeps with LDS-resident per-neuron state) and, for the
// per-tier arena, pool_compact_kernel (which pool serves each neuron; each
// pool's required ids, per chunk) -> plan_pools_kernel (one workgroup per
// pool, the fast plan over that pool's list) -> plan_merge_kernel (the
// three pools' plans merged by id into the caller's plan).
#include "m2c_internal.h"
#include "ffn_tasks.h"

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
  uint8_t* fill_from;
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
                                                            int step, int dom, DeviceState st,
                                                            PlanPtrs P) {
  __shared__ unsigned long long scan64[kPlanThreads / 64 + 1];
  __shared__ uint32_t scan32[kPlanThreads / 64 + 1];
  __shared__ int sh_hit, sh_refill, sh_empty, sh_der[2];
  const int tid = threadIdx.x;
  if (tid == 0) {
    sh_hit = 0;
    sh_der[0] = sh_der[1] = 0;
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
      const int s = st.slot_of[i];
      if (dom && s >= 0 && st.slot_tier[s] > t) t = st.slot_tier[s];  // hit at the resident tier
      ++nreq;
      tiers += 1ull << (21 * (3 - t));
      if (s < 0) ++nnew;
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
      const int s = st.slot_of[i];
      // the first sweep took the same step tier (slot_tier of a neuron's slot
      // changes only below, by the thread that owns the neuron)
      if (dom && s >= 0 && st.slot_tier[s] > t) t = st.slot_tier[s];
      P.req_ids[pos] = i;
      P.req_tier[pos] = (uint8_t)t;
      P.req_mask[pos] = m;
      st.work_pos[pos] = t == 3 ? r3++ : t == 2 ? r2++ : r1++;
      if (s >= 0) {
        const bool same = st.slot_tier[s] == t;
        P.req_hit[pos] = same ? 1 : 2;
        P.req_slot[pos] = s;
        st.slot_last[s] = step;
        st.prev_tier[pos] = st.slot_tier[s];
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
      const int from = P.req_hit[q] == 2 ? st.prev_tier[q] : 0;
      P.fill_ids[f] = P.req_ids[q];
      P.fill_tier[f] = P.req_tier[q];
      P.fill_slot[f] = ws;
      P.fill_from[f] = (uint8_t)from;
      if (from == 3 && P.req_tier[q] < 3) atomicAdd(&sh_der[P.req_tier[q] - 1], 1);
      ++f;
    }
  }
  __syncthreads();
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
    c[M2C_CNT_FILL_DERIVED] = sh_der[0] + sh_der[1];
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
    // required neurons by tier [10..12] = INT4, INT8, FP16
    atomicAdd(&st.stats[10], (unsigned long long)N1);
    atomicAdd(&st.stats[11], (unsigned long long)N2);
    atomicAdd(&st.stats[12], (unsigned long long)N3);
    atomicAdd(&st.stats[13], (unsigned long long)sh_der[1]);  // INT8
    atomicAdd(&st.stats[14], (unsigned long long)sh_der[0]);  // INT4
  }
}

// ---------------------------------------------------------------------------
// The same plan for d_ff <= 32768, built from coalesced sweeps: neuron i is
// handled by thread i % 1024 in chunk i / 1024, so every sweep issues its
// loads together, and each ordered list (R, NEW, fills, the three tiers of
// the work list, untouched and touched slots) is a compaction whose
// positions come from wave ballots plus one block scan over the per-(chunk,
// wave) counts. A first read-only sweep classifies every neuron (hit codes
// in LDS, touched slots in an LDS bitmap) and counts; nothing is written
// before the required set is known to fit in the plan.
constexpr int kPJ = 32;       // chunks of 1024 neurons (d_ff <= 32768)
constexpr int kPGroup = 12;   // chunks whose loads are in flight together
constexpr int kPWaves = kPlanThreads / 64;

__device__ __forceinline__ unsigned long long pk3(uint32_t a, uint32_t b, uint32_t c) {
  return (unsigned long long)a | ((unsigned long long)b << 21) | ((unsigned long long)c << 42);
}
__device__ __forceinline__ int fd3(unsigned long long v, int f) {
  return (int)((v >> (21 * f)) & 0x1fffffu);
}
__device__ __forceinline__ int popc(unsigned long long v) { return __popcll(v); }

// Exclusive prefixes of s_a[0..n) and s_b[0..n) (n <= kPlanThreads, one entry
// of each per thread), in place, sharing the barriers; the totals go to *ta,
// *tb. tmp: 2 (kPWaves + 1) entries. Contains barriers.
__device__ void scan_entries2(unsigned long long* s_a, unsigned long long* s_b, int n,
                              unsigned long long* tmp, unsigned long long* ta,
                              unsigned long long* tb) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned long long va = tid < n ? s_a[tid] : 0ull, vb = tid < n ? s_b[tid] : 0ull;
  unsigned long long ia = va, ib = vb;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned long long oa = __shfl_up(ia, off), ob = __shfl_up(ib, off);
    if (lane >= off) {
      ia += oa;
      ib += ob;
    }
  }
  if (lane == 63) {
    tmp[wave] = ia;
    tmp[kPWaves + 1 + wave] = ib;
  }
  __syncthreads();
  // every wave scans the wave totals itself (lane q: wave q's totals)
  unsigned long long wa = lane < kPWaves ? tmp[lane] : 0ull;
  unsigned long long wb = lane < kPWaves ? tmp[kPWaves + 1 + lane] : 0ull;
#pragma unroll
  for (int off = 1; off < kPWaves; off <<= 1) {
    const unsigned long long oa = __shfl_up(wa, off), ob = __shfl_up(wb, off);
    if (lane >= off) {
      wa += oa;
      wb += ob;
    }
  }
  const unsigned long long ba = wave > 0 ? __shfl(wa, wave - 1) : 0ull;
  const unsigned long long bb = wave > 0 ? __shfl(wb, wave - 1) : 0ull;
  if (tid < n) {
    s_a[tid] = ba + ia - va;
    s_b[tid] = bb + ib - vb;
  }
  *ta = __shfl(wa, kPWaves - 1);
  *tb = __shfl(wb, kPWaves - 1);
  __syncthreads();
}

// Exclusive prefix of s_v[0..n) (n <= kPlanThreads, one entry per thread), in
// place; returns the total. Contains barriers.
template <typename T>
__device__ T scan_entries(T* s_v, int n, T* tmp) {
  const int tid = threadIdx.x;
  const T v = tid < n ? s_v[tid] : T(0);
  T tot;
  const T ex = block_exclusive_scan<T>(v, tmp, &tot);
  if (tid < n) s_v[tid] = ex;
  __syncthreads();
  return tot;
}

// Step tier (max over rows, codes above FP16 read as FP16) and row mask of
// neuron i. ONE_ROW: B is 1 (a separate instantiation, so that no branch
// join forces a wait for the load).
template <bool ONE_ROW>
__device__ __forceinline__ void neuron_tiers(const uint8_t* __restrict__ tm, int d_ff, int i,
                                             int B, int& t, uint32_t& m) {
  t = 0;
  m = 0;
  if (ONE_ROW) {
    const int v = tm[i];
    t = v;
    m = v ? 1u : 0u;
  } else {
    for (int b0 = 0; b0 < B; b0 += 8) {
      uint8_t v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = tm[(int64_t)min(b0 + q, B - 1) * d_ff + i];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (b0 + q < B) {
          t = v[q] > t ? v[q] : t;
          m |= v[q] ? 1u << (b0 + q) : 0u;
        }
      }
    }
  }
  t = t > 3 ? 3 : t;
}

// pool_tier 0: the whole cache unit. pool_tier t (per-tier arena): only the
// neurons whose step tier is t, against that pool's state. Every pool's
// workgroup checks the whole required set against cap, so all of them leave
// their pool unchanged together when it does not fit; the FP16 pool's
// workgroup reports it (status word, and *abort for the merge).
//
// Memory round trips are what a one-workgroup plan waits on, so each neuron's
// slot and resident tier are kept in LDS from the first sweep to the second
// (with one batch row the second sweep reads no global memory), and the LRU
// order read for the victim count is kept for the victim pass. A pool's
// slots hold records of its own tier only, so a resident neuron of a pool is
// a hit without reading the slot's tier.
// The plan's LDS (one per kernel, shared by the body's instantiations).
struct PlanLds {
  // tier | code << 2 (1 hit, 2 refill, 0 new) | resident tier << 4
  uint8_t info[kPJ * kPlanThreads];
  // per thread-owned index i = tid + kPlanThreads j: the slot of resident
  // neuron i (sweeps A1, A2), then position i of the LRU order (C)
  uint16_t sl[kPJ * kPlanThreads];
  uint32_t touch[kPJ * kPlanThreads / 32];  // slots touched this step
  unsigned long long ca[kPJ * kPWaves];     // R, NEW, fills per (chunk, wave)
  unsigned long long cb[kPJ * kPWaves];     // FP16, INT8, INT4 per (chunk, wave)
  uint32_t cu[kPJ * kPWaves];               // slot compactions per (chunk, wave)
  unsigned long long scan64[2 * (kPWaves + 1)];
  uint32_t scan32[kPWaves + 1];
  int pre[kPJ + 1];  // pool plans: offsets of the pool's per-chunk lists
  int hit, refill, empty, all, f[4], der[2];
};

// POOL: a per-tier pool's plan (pool_tier > 0, no dominance inside a pool),
// over the pool's required neurons as pool_compact_kernel listed them: plist
// (chunk j's ids from j * kPlanThreads, ascending) and pcount ([3][NJ], every
// pool's, for the capacity check); tier_map and B are not read.
template <bool ONE_ROW, bool POOL>
__device__ __forceinline__ void plan_fast_body(
    const uint8_t* __restrict__ tier_map, int B, int d_ff, int C, int cap, int step, int dom,
    const DeviceState& st, const PlanPtrs& P, int pool_tier, int32_t* __restrict__ abort_word,
    PlanLds& sm, const int32_t* __restrict__ plist = nullptr,
    const int32_t* __restrict__ pcount = nullptr) {
  uint8_t* s_info = sm.info;
  uint16_t* s_sl = sm.sl;
  uint32_t* s_touch = sm.touch;
  unsigned long long *s_ca = sm.ca, *s_cb = sm.cb, *scan64 = sm.scan64;
  uint32_t *s_cu = sm.cu, *scan32 = sm.scan32;
  int &sh_hit = sm.hit, &sh_refill = sm.refill, &sh_empty = sm.empty, &sh_all = sm.all;
  int *sh_f = sm.f, *sh_der = sm.der;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned long long lt = (1ull << lane) - 1ull;
  const int NJ = (d_ff + kPlanThreads - 1) / kPlanThreads;
  const int NC = (C + kPlanThreads - 1) / kPlanThreads;
  if (tid == 0) {
    sh_all = 0;
    sh_hit = sh_refill = sh_empty = 0;
    sh_der[0] = sh_der[1] = 0;
    sh_f[0] = sh_f[1] = sh_f[2] = sh_f[3] = 0;
  }
  for (int w = tid; w < (C + 31) / 32; w += kPlanThreads) s_touch[w] = 0;
  __syncthreads();
  int NREQ, NNEW, NF, N3, N2, N1;
  if constexpr (POOL) {
    // ---------------- A (pool): the pool's required list is the
    // concatenation of its chunk lists; entry e is required neuron e
    const int q = 3 - pool_tier;
    int* s_pre = sm.pre;
    if (wave == 0) {  // chunk offsets (NJ <= 32) and the total over every pool
      int own = lane < NJ ? pcount[q * NJ + lane] : 0;
      int all = lane < NJ ? pcount[lane] + pcount[NJ + lane] + pcount[2 * NJ + lane] : 0;
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) {
        const int o = __shfl_up(own, off), a = __shfl_up(all, off);
        if (lane >= off) {
          own += o;
          all += a;
        }
      }
      if (lane < NJ) s_pre[lane + 1] = own;
      if (lane == 0) s_pre[0] = 0;
      if (lane == 31) sh_all = all;
    }
    __syncthreads();
    const int R = s_pre[NJ], NALL = sh_all;
    if (NALL > cap) {  // workgroup-uniform: an empty plan, the cache untouched
      if (tid == 0) {
        for (int c = 0; c < M2C_NCOUNTS; ++c) P.counts[c] = 0;
        P.counts[M2C_NCOUNTS - 1] = NALL;
        if (pool_tier == 3) {
          atomicOr(st.status, M2C_STATUS_PLAN_OVERFLOW);
          *abort_word = 1;
        }
      }
      return;
    }
    if (pool_tier == 3 && tid == 0) *abort_word = 0;
    // entry e of the list: chunk j with s_pre[j] <= e < s_pre[j + 1]
    auto entry = [&](int e) {
      int lo = 0, hi = NJ;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_pre[mid] <= e) lo = mid;
        else hi = mid;
      }
      return plist[lo * kPlanThreads + (e - s_pre[lo])];
    };
    const int NE = (R + kPlanThreads - 1) / kPlanThreads;  // rounds of entries (<= kPJ)
    constexpr int kPR = 4;  // rounds whose loads are in flight together
    // pass 1: the NEW neurons (not resident) per (round, wave); resident
    // neurons touch their slots
    for (int r0 = 0; r0 < NE; r0 += kPR) {
      int id[kPR], sl[kPR];
#pragma unroll
      for (int u = 0; u < kPR; ++u) id[u] = entry(min(tid + kPlanThreads * (r0 + u), max(R - 1, 0)));
#pragma unroll
      for (int u = 0; u < kPR; ++u) sl[u] = st.slot_of[id[u]];
#pragma unroll
      for (int u = 0; u < kPR; ++u) {
        const int r = r0 + u;
        const bool in = r < NE && tid + kPlanThreads * r < R;
        if (in && sl[u] >= 0) atomicOr(&s_touch[sl[u] >> 5], 1u << (sl[u] & 31));
        const unsigned long long b = __ballot(in && sl[u] < 0);
        if (lane == 0 && r < NE) s_cu[r * kPWaves + wave] = (uint32_t)popc(b);
      }
    }
    __syncthreads();
    const int nnew = (int)scan_entries<uint32_t>(s_cu, NE * kPWaves, scan32);
    // pass 2: required, NEW and fill lists (the fills are the NEW neurons)
    for (int r0 = 0; r0 < NE; r0 += kPR) {
      int id[kPR], sl[kPR];
#pragma unroll
      for (int u = 0; u < kPR; ++u) id[u] = entry(min(tid + kPlanThreads * (r0 + u), max(R - 1, 0)));
#pragma unroll
      for (int u = 0; u < kPR; ++u) sl[u] = st.slot_of[id[u]];
#pragma unroll
      for (int u = 0; u < kPR; ++u) {
        const int r = r0 + u, e = tid + kPlanThreads * r;
        const bool in = r < NE && e < R, nw = in && sl[u] < 0;
        const unsigned long long b = __ballot(nw);
        if (!in) continue;
        P.req_ids[e] = id[u];
        P.req_tier[e] = (uint8_t)pool_tier;
        P.req_mask[e] = 1u;
        st.work_pos[e] = e;
        if (!nw) {
          P.req_slot[e] = sl[u];
          P.req_hit[e] = 1;
          st.slot_last[sl[u]] = step;
          st.fill_pos[e] = -1;
        } else {
          const int inew = (int)s_cu[r * kPWaves + wave] + popc(b & lt);
          st.new_pos[inew] = e;
          st.fill_pos[e] = inew;
          P.fill_ids[inew] = id[u];
          P.fill_tier[inew] = (uint8_t)pool_tier;
          P.fill_from[inew] = 0;
        }
      }
    }
    NREQ = R;
    NNEW = NF = nnew;
    N3 = pool_tier == 3 ? R : 0;
    N2 = pool_tier == 2 ? R : 0;
    N1 = pool_tier == 1 ? R : 0;
    if (tid == 0) sh_hit = R - nnew;
  } else {
  // ---------------- A1: classify and count (reads only)
  // every load of a group is issued before the first value is used; the
  // wave's counts stay in registers until the end of the sweep
  int c_all = 0, c_hit = 0, c_ref = 0;
  for (int j0 = 0; j0 < NJ; j0 += kPGroup) {
    int t[kPGroup], sl[kPGroup];
    uint32_t m[kPGroup];
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      const int i = min(tid + kPlanThreads * (j0 + g), d_ff - 1);
      neuron_tiers<ONE_ROW>(tier_map, d_ff, i, B, t[g], m[g]);
      sl[g] = st.slot_of[i];
    }
    int old[kPGroup];
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      if (pool_tier) {  // the whole required set, for the capacity check
        c_all += popc(__ballot(j0 + g < NJ && tid + kPlanThreads * (j0 + g) < d_ff && t[g] > 0));
        if (t[g] != pool_tier) t[g] = 0;  // another pool's neuron
      }
      old[g] = sl[g] < 0 ? 0 : pool_tier ? pool_tier : st.slot_tier[sl[g]];
    }
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      const int j = j0 + g, i = tid + kPlanThreads * j;
      const bool valid = j < NJ && i < d_ff;
      const bool req = valid && t[g] > 0;
      const bool res = req && sl[g] >= 0;
      const bool hit = res && (old[g] == t[g] || (dom && old[g] > t[g]));
      if (hit) t[g] = old[g];  // the step tier of a hit is the resident tier
      if (valid) s_info[i] = req ? (uint8_t)(t[g] | ((hit ? 1 : res ? 2 : 0) << 2) | (old[g] << 4)) : 0;
      if (res) s_sl[i] = (uint16_t)sl[g];
      if (res) atomicOr(&s_touch[sl[g] >> 5], 1u << (sl[g] & 31));
      if constexpr (POOL) {
        // one tier, resident = hit: fills are the NEW neurons, every count
        // follows from two ballots
        const int n0 = popc(__ballot(req)), n1 = popc(__ballot(req && !res));
        if (lane == 0 && j < NJ) {
          s_ca[j * kPWaves + wave] = pk3(n0, n1, n1);
          s_cb[j * kPWaves + wave] = pk3(pool_tier == 3 ? n0 : 0, pool_tier == 2 ? n0 : 0,
                                         pool_tier == 1 ? n0 : 0);
        }
        c_hit += n0 - n1;
      } else {
        const unsigned long long b0 = __ballot(req), b1 = __ballot(req && !res),
                                 b2 = __ballot(req && !hit), b3 = __ballot(req && t[g] == 3),
                                 b4 = __ballot(req && t[g] == 2), b5 = __ballot(req && t[g] == 1),
                                 bh = __ballot(hit), br = __ballot(res && !hit);
        if (lane == 0 && j < NJ) {
          s_ca[j * kPWaves + wave] = pk3(popc(b0), popc(b1), popc(b2));
          s_cb[j * kPWaves + wave] = pk3(popc(b3), popc(b4), popc(b5));
        }
        c_hit += popc(bh);
        c_ref += popc(br);
      }
    }
  }
  if (lane == 0) {
    if (c_all) atomicAdd(&sh_all, c_all);
    if (c_hit) atomicAdd(&sh_hit, c_hit);
    if (c_ref) atomicAdd(&sh_refill, c_ref);
  }
  __syncthreads();
  unsigned long long totA, totB;
  scan_entries2(s_ca, s_cb, NJ * kPWaves, scan64, &totA, &totB);
  NREQ = fd3(totA, 0);
  NNEW = fd3(totA, 1);
  NF = fd3(totA, 2);
  N3 = fd3(totB, 0);
  N2 = fd3(totB, 1);
  N1 = fd3(totB, 2);
  const int NALL = pool_tier ? sh_all : NREQ;  // sh_all is final after the scans' barriers
  if (NALL > cap) {  // workgroup-uniform: an empty plan, the cache untouched
    if (tid == 0) {
      for (int q = 0; q < M2C_NCOUNTS; ++q) P.counts[q] = 0;
      P.counts[M2C_NCOUNTS - 1] = NALL;
      if (pool_tier == 0 || pool_tier == 3) atomicOr(st.status, M2C_STATUS_PLAN_OVERFLOW);
      if (pool_tier == 3) *abort_word = 1;
    }
    return;
  }
  if (pool_tier == 3 && tid == 0) *abort_word = 0;
  // ---------------- A2: required list, NEW list, fill ids, work positions
  for (int j0 = 0; j0 < NJ; j0 += kPGroup) {
    uint32_t m[kPGroup];
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      m[g] = 1u;  // one batch row: every required neuron's row mask
      if (!ONE_ROW) {
        int tt;
        neuron_tiers<ONE_ROW>(tier_map, d_ff, min(tid + kPlanThreads * (j0 + g), d_ff - 1), B, tt, m[g]);
      }
    }
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      const int j = j0 + g, i = tid + kPlanThreads * j;
      const bool valid = j < NJ && i < d_ff;
      const int info = valid ? s_info[i] : 0;
      const int t = info & 3, code = (info >> 2) & 3;
      const bool req = t > 0, res = code != 0, hit = code == 1;
      int pos, wp, inew, ifill;
      if constexpr (POOL) {  // one tier: the work order is the required order
        const unsigned long long b0 = __ballot(req), b1 = __ballot(req && !res);
        if (!req) continue;
        const unsigned long long pa = s_ca[j * kPWaves + wave];
        pos = wp = fd3(pa, 0) + popc(b0 & lt);
        inew = fd3(pa, 1) + popc(b1 & lt);
        ifill = fd3(pa, 2) + popc(b1 & lt);
      } else {
        const unsigned long long b0 = __ballot(req), b1 = __ballot(req && !res),
                                 b2 = __ballot(req && !hit), b3 = __ballot(req && t == 3),
                                 b4 = __ballot(req && t == 2), b5 = __ballot(req && t == 1);
        if (!req) continue;
        const unsigned long long pa = s_ca[j * kPWaves + wave], pb = s_cb[j * kPWaves + wave];
        pos = fd3(pa, 0) + popc(b0 & lt);
        wp = t == 3 ? fd3(pb, 0) + popc(b3 & lt)
             : t == 2 ? N3 + fd3(pb, 1) + popc(b4 & lt)
                      : N3 + N2 + fd3(pb, 2) + popc(b5 & lt);
        inew = fd3(pa, 1) + popc(b1 & lt);
        ifill = fd3(pa, 2) + popc(b2 & lt);
      }
      P.req_ids[pos] = i;
      P.req_tier[pos] = (uint8_t)t;
      P.req_mask[pos] = m[g];
      st.work_pos[pos] = wp;
      int from = 0;
      if (res) {
        const int sl = s_sl[i];
        P.req_slot[pos] = sl;
        P.req_hit[pos] = hit ? 1 : 2;
        st.slot_last[sl] = step;
        from = info >> 4;
        if (!hit) st.slot_tier[sl] = (uint8_t)t;
      } else {
        st.new_pos[inew] = pos;
      }
      if (!hit) {
        const int fr = ifill;
        st.fill_pos[pos] = fr;
        P.fill_ids[fr] = i;
        P.fill_tier[fr] = (uint8_t)t;
        P.fill_from[fr] = (uint8_t)from;
        if (from == 3 && t < 3) atomicAdd(&sh_der[t - 1], 1);
      } else {
        st.fill_pos[pos] = -1;
      }
    }
  }
  }  // A1, A2 (the touched-slot marks were made before the scans' barriers)
  // ---------------- C: victims = untouched slots in LRU order
  const int cur = *st.lru_cur;
  const int32_t* lru_in = st.lru + (int64_t)cur * C;
  int32_t* lru_out = st.lru + (int64_t)(1 - cur) * C;
  for (int j0 = 0; j0 < NC; j0 += kPGroup) {
    int sv[kPGroup];
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) sv[g] = lru_in[min(tid + kPlanThreads * (j0 + g), C - 1)];
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      const int j = j0 + g;
      const bool valid = j < NC && tid + kPlanThreads * j < C;
      if (valid) s_sl[tid + kPlanThreads * j] = (uint16_t)sv[g];
      const bool unt = valid && !((s_touch[sv[g] >> 5] >> (sv[g] & 31)) & 1u);
      const unsigned long long bu = __ballot(unt);
      if (lane == 0 && j < NC) s_cu[j * kPWaves + wave] = (uint32_t)popc(bu);
    }
  }
  __syncthreads();
  const int NUNT = (int)scan_entries<uint32_t>(s_cu, NC * kPWaves, scan32);
  const int NV = NNEW < NUNT ? NNEW : NUNT;
  {
    int empties = 0;
    for (int j0 = 0; j0 < NC; j0 += kPGroup) {
      int sv[kPGroup];
#pragma unroll
      for (int g = 0; g < kPGroup; ++g)
        sv[g] = s_sl[min(tid + kPlanThreads * (j0 + g), kPJ * kPlanThreads - 1)];
#pragma unroll
      for (int g = 0; g < kPGroup; ++g) {
        const int j = j0 + g;
        const bool valid = j < NC && tid + kPlanThreads * j < C;
        // only this thread looks at slot sv[g]'s bit, so marking victims below
        // does not disturb the test
        const bool unt = valid && !((s_touch[sv[g] >> 5] >> (sv[g] & 31)) & 1u);
        const unsigned long long bu = __ballot(unt);
        if (!unt) continue;
        const int u = (int)s_cu[j * kPWaves + wave] + popc(bu & lt);
        if (u < NV) {
          const int s = sv[g];
          const int old = st.slot_key[s];
          st.vict_slot[u] = s;
          st.vict_old[u] = old;
          empties += old < 0;
          st.slot_last[s] = step;
          atomicOr(&s_touch[s >> 5], 1u << (s & 31));
        } else {
          lru_out[u - NV] = sv[g];
        }
      }
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
  for (int j0 = 0; j0 < NC; j0 += kPGroup) {
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      const int j = j0 + g, s = tid + kPlanThreads * j;
      const bool tch = j < NC && s < C && ((s_touch[s >> 5] >> (s & 31)) & 1u);
      const unsigned long long bt = __ballot(tch);
      if (lane == 0 && j < NC) s_cu[j * kPWaves + wave] = (uint32_t)popc(bt);
    }
  }
  __syncthreads();
  scan_entries<uint32_t>(s_cu, NC * kPWaves, scan32);
  for (int j0 = 0; j0 < NC; j0 += kPGroup) {
#pragma unroll
    for (int g = 0; g < kPGroup; ++g) {
      const int j = j0 + g, s = tid + kPlanThreads * j;
      const bool tch = j < NC && s < C && ((s_touch[s >> 5] >> (s & 31)) & 1u);
      const unsigned long long bt = __ballot(tch);
      if (tch) lru_out[NUNT - NV + (int)s_cu[j * kPWaves + wave] + popc(bt & lt)] = s;
    }
  }
  // ---------------- E: work list and fill slots
  for (int q = tid; q < NREQ; q += kPlanThreads) {
    const int ws = P.req_slot[q];
    const int wp = st.work_pos[q];
    P.work_slot[wp] = ws;
    P.work_mask[wp] = P.req_mask[q];
    const int fp = st.fill_pos[q];
    if (fp >= 0) {
      P.fill_slot[fp] = ws;
      atomicAdd(&sh_f[P.req_tier[q]], 1);
    }
  }
  __syncthreads();
  if (tid == 0) {
    const int F3 = sh_f[3], F2 = sh_f[2], F1 = sh_f[1];
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
    c[M2C_CNT_FILL_DERIVED] = sh_der[0] + sh_der[1];
    c[M2C_CNT_FILL_INT4] = F1;
    for (int q = 0; q < M2C_NCOUNTS; ++q) P.counts[q] = c[q];
    *st.lru_cur = 1 - cur;
    if (pool_tier == 0 || pool_tier == 3) atomicAdd(&st.stats[0], 1ull);  // one plan per step
    atomicAdd(&st.stats[1], (unsigned long long)NREQ);
    atomicAdd(&st.stats[2], (unsigned long long)sh_hit);
    atomicAdd(&st.stats[3], (unsigned long long)sh_refill);
    atomicAdd(&st.stats[4], (unsigned long long)NV);
    atomicAdd(&st.stats[5], (unsigned long long)(NNEW - NV));
    atomicAdd(&st.stats[6], (unsigned long long)(NV - NEMPTY));
    atomicAdd(&st.stats[7], (unsigned long long)F1);
    atomicAdd(&st.stats[8], (unsigned long long)F2);
    atomicAdd(&st.stats[9], (unsigned long long)F3);
    atomicAdd(&st.stats[10], (unsigned long long)N1);
    atomicAdd(&st.stats[11], (unsigned long long)N2);
    atomicAdd(&st.stats[12], (unsigned long long)N3);
    atomicAdd(&st.stats[13], (unsigned long long)sh_der[1]);  // INT8
    atomicAdd(&st.stats[14], (unsigned long long)sh_der[0]);  // INT4
  }
}

__global__ __launch_bounds__(kPlanThreads) void plan_fast_kernel(
    const uint8_t* __restrict__ tier_map, int B, int d_ff, int C, int cap, int step, int dom,
    DeviceState st, PlanPtrs P, int32_t* __restrict__ abort_word) {
  __shared__ PlanLds sm;
  if (B == 1)
    plan_fast_body<true, false>(tier_map, B, d_ff, C, cap, step, dom, st, P, 0, abort_word, sm);
  else
    plan_fast_body<false, false>(tier_map, B, d_ff, C, cap, step, dom, st, P, 0, abort_word, sm);
}

// Per-tier arena: workgroup q plans pool 3 - q (FP16, INT8, INT4) into its
// own plan buffer; the pools are independent, so they run side by side.
struct PoolJobs {
  DeviceState st[3];
  PlanPtrs P[3];
  int C[3];
};

__global__ __launch_bounds__(kPlanThreads) void plan_pools_kernel(
    const int32_t* __restrict__ lists, const int32_t* __restrict__ counts, int d_ff, int cap,
    int step, PoolJobs jobs, int32_t* __restrict__ abort_word) {
  const int q = blockIdx.x;
  __shared__ PlanLds sm;
  plan_fast_body<true, true>(nullptr, 1, d_ff, jobs.C[q], cap, step, 0, jobs.st[q], jobs.P[q],
                             3 - q, abort_word, sm, lists + (int64_t)q * d_ff, counts);
}

// Per-tier arena: the pool that serves each neuron this step, and each
// pool's required neurons as lists per chunk of kPlanThreads neurons (one
// workgroup per chunk; ascending id inside a chunk, so the chunk lists in
// order are the pool's required list). A neuron's step tier is its highest
// over the batch rows. With dominance hits (dom), a neuron required at tier t
// that is not resident in pool t but is resident in a pool of higher
// precision goes to the lowest such pool, as a hit at that pool's tier; any
// other neuron keeps its tier. Residency is read before any pool plans the
// step. slot_of: the pools' tables [3][d_ff], FP16 first; lists [3][d_ff]
// (chunk j's from j * kPlanThreads), counts [3][gridDim.x].
__global__ __launch_bounds__(kPlanThreads) void pool_compact_kernel(
    const uint8_t* __restrict__ tier_map, int B, int d_ff, int dom,
    const int32_t* __restrict__ slot_of, int32_t* __restrict__ lists,
    int32_t* __restrict__ counts) {
  __shared__ uint32_t s_wc[3][kPWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = blockIdx.x * kPlanThreads + tid;
  const int nc = min(n, d_ff - 1);
  // every load at once (one memory round trip; this kernel runs beside the
  // fills, whose host reads make each round trip long)
  bool r3 = false, r2 = false, r1 = false;
  if (dom) {
    r3 = slot_of[nc] >= 0;
    r2 = slot_of[(int64_t)d_ff + nc] >= 0;
    r1 = slot_of[2 * (int64_t)d_ff + nc] >= 0;
  }
  int t = 0;
  for (int b = 0; b < B; ++b) t = max(t, (int)tier_map[(int64_t)b * d_ff + nc]);
  t = min(t, 3);
  if (dom) {
    const bool own = t == 3 ? r3 : t == 2 ? r2 : t == 1 ? r1 : true;
    if (!own) t = (t < 2 && r2) ? 2 : r3 ? 3 : t;
  }
  if (n >= d_ff) t = 0;
  unsigned long long mine = 0ull;
#pragma unroll
  for (int p = 3; p >= 1; --p) {
    const unsigned long long b = __ballot(t == p);
    if (t == p) mine = b;
    if (lane == 0) s_wc[3 - p][wave] = (uint32_t)popc(b);
  }
  __syncthreads();
  if (t > 0) {
    const int q = 3 - t;
    int pre = 0;
    for (int w = 0; w < wave; ++w) pre += (int)s_wc[q][w];
    lists[(int64_t)q * d_ff + (int64_t)blockIdx.x * kPlanThreads + pre +
          popc(mine & ((1ull << lane) - 1ull))] = n;
  }
  if (tid < 3) {
    int c = 0;
    for (int w = 0; w < kPWaves; ++w) c += (int)s_wc[tid][w];
    counts[tid * (int)gridDim.x + blockIdx.x] = c;
  }
}

// Empties one cache unit (or one pool of the per-tier arena: its own
// tables); clears n_rec entries of the fill's record table and, with
// clear_stats, the counters.
__global__ void reset_kernel(DeviceState st, int d_ff, int C, int n_rec, int clear_stats) {
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
  for (int s = idx; s < n_rec; s += n) st.slot_rec[s] = -1;
  if (idx == 0) *st.lru_cur = 0;
  if (clear_stats && idx < 16) st.stats[idx] = 0;
}

// Per-tier arena: the three pools' plans (each over its own tier, in
// ascending id) merged into the caller's plan. R and the fills are merged by
// id (a neuron has one step tier, so the lists are disjoint: an entry's
// position is its index in its own list plus the entries of the other lists
// with smaller ids); the work list is the pools' lists in tier order; the
// evictions are the pools' evictions in tier order. Slot ids become global.
struct PoolPlan {
  const int32_t* counts;
  const int32_t* req_ids;
  const uint8_t* req_hit;
  const int32_t* req_slot;
  const uint32_t* req_mask;
  const int32_t* fill_ids;
  const int32_t* fill_slot;
  const int32_t* evicted_ids;
};
struct PoolPlans {
  PoolPlan p[3];  // FP16, INT8, INT4
};

__device__ __forceinline__ int lower_bound(const int32_t* a, int n, int v) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// The merged lists are in ascending id order: an entry's position is its
// position in its pool's list plus its rank (a binary search) in each other
// pool's list. The pools' id lists are staged in LDS first (one memory round
// trip for all of them), so the searches cost no further round trips; lists
// longer than the staging area are searched in global memory.
constexpr int kMergeThreads = 256;
constexpr int kMergeIds = 4096;  // ids staged per list kind (required, fills)

// One of three kernel-argument values by a runtime index, as selects of
// values already in registers (indexing the argument struct would read it
// from memory).
template <typename T>
__device__ __forceinline__ T pick(int q, T a, T b, T c) {
  return q == 0 ? a : q == 1 ? b : c;
}

__device__ __forceinline__ void stage_ids(int32_t* __restrict__ dst, const int32_t* s0,
                                          const int32_t* s1, const int32_t* s2, const int n[3]) {
  const int tot = n[0] + n[1] + n[2];
  int32_t v[kMergeIds / kMergeThreads];
#pragma unroll
  for (int c = 0; c < kMergeIds / kMergeThreads; ++c) {
    const int e = c * kMergeThreads + (int)threadIdx.x;
    const int q = e < n[0] ? 0 : e < n[0] + n[1] ? 1 : 2;
    const int p = e - (q > 0 ? n[0] : 0) - (q > 1 ? n[1] : 0);
    v[c] = e < tot ? pick(q, s0, s1, s2)[p] : 0;
  }
#pragma unroll
  for (int c = 0; c < kMergeIds / kMergeThreads; ++c) {
    const int e = c * kMergeThreads + (int)threadIdx.x;
    if (e < tot) dst[e] = v[c];
  }
}

// The batch-1 FFN's task table, written beside the merge (workgroups from
// merge_blocks on), from the pools' plans: work item e of the merged plan is
// entry e of the pools' required lists in tier order.
struct TaskTable {
  int32_t* tasks;
  int32_t* task_ids;
  int d, grid, cap;
};

template <int K>
__device__ __forceinline__ void pool_task_table(const PoolPlans& pp, const SlotMap& map,
                                                const TaskTable& tt, bool ab, int block,
                                                int blocks) {
  int n3 = ab ? 0 : pp.p[0].counts[M2C_CNT_REQ];
  int n2 = ab ? 0 : pp.p[1].counts[M2C_CNT_REQ];
  int n1 = ab ? 0 : pp.p[2].counts[M2C_CNT_REQ];
  n3 = n3 < 0 ? 0 : n3 > tt.cap ? tt.cap : n3;
  n2 = n2 < 0 ? 0 : n2 > tt.cap - n3 ? tt.cap - n3 : n2;
  n1 = n1 < 0 ? 0 : n1 > tt.cap - n3 - n2 ? tt.cap - n3 - n2 : n1;
  const FMap m = make_map_n<K>(n3, n2, n1, tt.d);
  const int f3 = map.first[3], f2 = map.first[2], f1 = map.first[1];
  write_task_table<K>(m, tt.grid, map, tt.tasks, tt.task_ids,
                      (int)(block * blockDim.x + threadIdx.x) >> 6,
                      (int)(blocks * blockDim.x) >> 6, [&](int e) {
                        return e < n3        ? pp.p[0].req_slot[e] + f3
                               : e < n3 + n2 ? pp.p[1].req_slot[e - n3] + f2
                                             : pp.p[2].req_slot[e - n3 - n2] + f1;
                      });
}

// Workgroups [0, merge_blocks): the merge; the rest (if any): the task table.
template <int K>
__global__ __launch_bounds__(kMergeThreads) void plan_merge_kernel(PoolPlans pp, PlanPtrs out,
                                                                    SlotMap map,
                                                                    const int32_t* __restrict__ abort_word,
                                                                    int merge_blocks, TaskTable tt) {
  __shared__ int32_t s_req[kMergeIds], s_fill[kMergeIds];
  const bool ab = *abort_word != 0;
  if ((int)blockIdx.x >= merge_blocks) {
    pool_task_table<K>(pp, map, tt, ab, (int)blockIdx.x - merge_blocks,
                       (int)gridDim.x - merge_blocks);
    return;
  }
  int nr[3], nf[3], ne[3];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    nr[q] = ab ? 0 : pp.p[q].counts[M2C_CNT_REQ];
    nf[q] = ab ? 0 : pp.p[q].counts[M2C_CNT_FILL];
    ne[q] = ab ? 0 : pp.p[q].counts[M2C_CNT_EVICT];
  }
  const int tid = blockIdx.x * blockDim.x + threadIdx.x, nth = merge_blocks * blockDim.x;
  if (tid < M2C_NCOUNTS) {
    int v = 0;
    if (ab)
      v = tid == M2C_NCOUNTS - 1 ? pp.p[0].counts[M2C_NCOUNTS - 1] : 0;
    else if (tid <= M2C_CNT_FILL_INT4)
      v = pp.p[0].counts[tid] + pp.p[1].counts[tid] + pp.p[2].counts[tid];
    out.counts[tid] = v;
  }
  const int R = nr[0] + nr[1] + nr[2], NF = nf[0] + nf[1] + nf[2];
  const bool lr = R <= kMergeIds, lf = NF <= kMergeIds;  // uniform over the grid
  {
    if (lr) stage_ids(s_req, pp.p[0].req_ids, pp.p[1].req_ids, pp.p[2].req_ids, nr);
    if (lf) stage_ids(s_fill, pp.p[0].fill_ids, pp.p[1].fill_ids, pp.p[2].fill_ids, nf);
    __syncthreads();
  }
  for (int e = tid; e < R; e += nth) {
    const int q = e < nr[0] ? 0 : e < nr[0] + nr[1] ? 1 : 2;
    const int p = e - (q > 0 ? nr[0] : 0) - (q > 1 ? nr[1] : 0);
    const int t = 3 - q;
    const int id = lr ? s_req[e] : pick(q, pp.p[0].req_ids, pp.p[1].req_ids, pp.p[2].req_ids)[p];
    int pos = p;
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      if (u == q) continue;
      const int off = (u > 0 ? nr[0] : 0) + (u > 1 ? nr[1] : 0);
      pos += lr ? lower_bound(s_req + off, nr[u], id) : lower_bound(pp.p[u].req_ids, nr[u], id);
    }
    const int gs = pick(q, pp.p[0].req_slot, pp.p[1].req_slot, pp.p[2].req_slot)[p] +
                   pick(q, map.first[3], map.first[2], map.first[1]);
    const uint32_t mk = pick(q, pp.p[0].req_mask, pp.p[1].req_mask, pp.p[2].req_mask)[p];
    const uint8_t hit = pick(q, pp.p[0].req_hit, pp.p[1].req_hit, pp.p[2].req_hit)[p];
    out.req_ids[pos] = id;
    out.req_tier[pos] = (uint8_t)t;
    out.req_hit[pos] = hit;
    out.req_slot[pos] = gs;
    out.req_mask[pos] = mk;
    out.work_slot[e] = gs;  // pool order = tier-major, ascending id inside a tier
    out.work_mask[e] = mk;
  }
  for (int e = tid; e < NF; e += nth) {
    const int q = e < nf[0] ? 0 : e < nf[0] + nf[1] ? 1 : 2;
    const int p = e - (q > 0 ? nf[0] : 0) - (q > 1 ? nf[1] : 0);
    const int t = 3 - q;
    const int id = lf ? s_fill[e] : pick(q, pp.p[0].fill_ids, pp.p[1].fill_ids, pp.p[2].fill_ids)[p];
    int pos = p;
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      if (u == q) continue;
      const int off = (u > 0 ? nf[0] : 0) + (u > 1 ? nf[1] : 0);
      pos += lf ? lower_bound(s_fill + off, nf[u], id) : lower_bound(pp.p[u].fill_ids, nf[u], id);
    }
    out.fill_ids[pos] = id;
    out.fill_tier[pos] = (uint8_t)t;
    out.fill_slot[pos] = pick(q, pp.p[0].fill_slot, pp.p[1].fill_slot, pp.p[2].fill_slot)[p] +
                         pick(q, map.first[3], map.first[2], map.first[1]);
    out.fill_from[pos] = 0;
  }
  const int NE = ne[0] + ne[1] + ne[2];
  for (int e = tid; e < NE; e += nth) {
    const int q = e < ne[0] ? 0 : e < ne[0] + ne[1] ? 1 : 2;
    const int p = e - (q > 0 ? ne[0] : 0) - (q > 1 ? ne[1] : 0);
    out.evicted_ids[e] = pick(q, pp.p[0].evicted_ids, pp.p[1].evicted_ids, pp.p[2].evicted_ids)[p];
  }
}

DeviceState pool_state(const m2c_layer* L, int t) {
  DeviceState v = L->st;
  if (!L->pools) return v;
  const int q = 3 - t, rf = L->pool_rf[t];
  v.slot_of = L->st.slot_of + (int64_t)q * L->desc.d_ff;
  v.slot_key = L->st.slot_key + rf;
  v.slot_tier = L->st.slot_tier + rf;
  v.slot_last = L->st.slot_last + rf;
  v.lru = L->st.lru + 2 * (int64_t)rf;
  v.lru_cur = L->st.lru_cur + q;
  const int64_t cap = L->cap;
  v.new_pos = L->st.new_pos + q * cap;
  v.work_pos = L->st.work_pos + q * cap;
  v.vict_slot = L->st.vict_slot + q * cap;
  v.vict_old = L->st.vict_old + q * cap;
  v.fill_pos = L->st.fill_pos + q * cap;
  v.prev_tier = L->st.prev_tier + q * cap;
  return v;
}

static PlanPtrs plan_ptrs(const m2c_layer* L, uint8_t* plan) {
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
  P.fill_from = plan + lay.fill_from;
  P.evicted_ids = reinterpret_cast<int32_t*>(plan + lay.evicted_ids);
  P.work_slot = reinterpret_cast<int32_t*>(plan + lay.work_slot);
  P.work_mask = reinterpret_cast<uint32_t*>(plan + lay.work_mask);
  return P;
}

hipError_t launch_plan(m2c_layer* L, const uint8_t* tier_map, int batch, int step, uint8_t* plan,
                       hipStream_t stream) {
  const PlanPtrs P = plan_ptrs(L, plan);
  const int dom = (L->desc.flags & M2C_FLAG_DOMINANT_HITS) ? 1 : 0;
  if (!L->pools) {
    if (L->desc.d_ff <= kPJ * kPlanThreads)
      hipLaunchKernelGGL(plan_fast_kernel, dim3(1), dim3(kPlanThreads), 0, stream, tier_map, batch,
                         L->desc.d_ff, L->desc.cache_slots, L->cap, step, dom, L->st, P,
                         L->plan_abort);
    else
      hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, tier_map, batch,
                         L->desc.d_ff, L->desc.cache_slots, L->cap, step, dom, L->st, P);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? launch_ffn_tasks(L, plan, stream) : e;
  }
  // per-tier arena (d_ff <= 32768, checked at create): the three pools'
  // plans side by side in one launch, into the layer's pool plans, then the
  // merge into the caller's plan
  PoolPlans pp;
  PoolJobs jobs;
  for (int q = 0; q < 3; ++q) {
    const int t = 3 - q;
    const PlanPtrs Pq = plan_ptrs(L, L->pool_plan + (int64_t)q * L->plan_core_bytes);
    jobs.st[q] = pool_state(L, t);
    jobs.P[q] = Pq;
    jobs.C[q] = L->pool_C[t];
    pp.p[q] = {Pq.counts, Pq.req_ids, Pq.req_hit, Pq.req_slot, Pq.req_mask, Pq.fill_ids,
               Pq.fill_slot, Pq.evicted_ids};
  }
  const int NJ = (L->desc.d_ff + kPlanThreads - 1) / kPlanThreads;  // <= kPJ (checked at create)
  hipLaunchKernelGGL(pool_compact_kernel, dim3(NJ), dim3(kPlanThreads), 0, stream, tier_map, batch,
                     L->desc.d_ff, dom, L->st.slot_of, L->pool_lists, L->pool_counts);
  hipError_t e0 = hipGetLastError();
  if (e0 != hipSuccess) return e0;
  hipLaunchKernelGGL(plan_pools_kernel, dim3(3), dim3(kPlanThreads), 0, stream, L->pool_lists,
                     L->pool_counts, L->desc.d_ff, L->cap, step, jobs, L->plan_abort);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int blocks = (L->cap + kMergeThreads - 1) / kMergeThreads;
  blocks = blocks < 1 ? 1 : blocks > 64 ? 64 : blocks;
  // the FFN's task table in the same launch, from the pools' plans (one wave
  // per task, as in the single unit's table kernel)
  TaskTable tt{};
  int tblocks = 0;
  if (ffn_tasks_used(L) && L->ffn_grid > 0) {
    int32_t* tasks = reinterpret_cast<int32_t*>(plan + L->layout.ffn_tasks);
    tt = {tasks, tasks + task_ids_offset(L->ffn_grid) / 4, L->desc.d_model, L->ffn_grid,
          L->cap};
    tblocks = (L->ffn_grid + 3) / 4;
    tblocks = tblocks < 1 ? 1 : tblocks > 256 ? 256 : tblocks;
  }
  const dim3 g(blocks + tblocks), b(kMergeThreads);
  switch (ffn_loads_per_unit(L->desc.d_model)) {
    case 1: hipLaunchKernelGGL(plan_merge_kernel<1>, g, b, 0, stream, pp, P, L->map, L->plan_abort, blocks, tt); break;
    case 2: hipLaunchKernelGGL(plan_merge_kernel<2>, g, b, 0, stream, pp, P, L->map, L->plan_abort, blocks, tt); break;
    case 4: hipLaunchKernelGGL(plan_merge_kernel<4>, g, b, 0, stream, pp, P, L->map, L->plan_abort, blocks, tt); break;
    default: hipLaunchKernelGGL(plan_merge_kernel<8>, g, b, 0, stream, pp, P, L->map, L->plan_abort, blocks, tt); break;
  }
  return hipGetLastError();
}

hipError_t launch_reset(m2c_layer* L, hipStream_t stream) {
  const int n_rec = L->desc.cache_slots + L->S;
  int n = L->desc.d_ff > n_rec ? L->desc.d_ff : n_rec;
  int blocks = (n + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 1024) blocks = 1024;
  if (!L->pools) {
    hipLaunchKernelGGL(reset_kernel, dim3(blocks), dim3(256), 0, stream, L->st, L->desc.d_ff,
                       L->desc.cache_slots, n_rec, 1);
    return hipGetLastError();
  }
  for (int t = 3; t >= 1; --t) {
    hipLaunchKernelGGL(reset_kernel, dim3(blocks), dim3(256), 0, stream, pool_state(L, t),
                       L->desc.d_ff, L->pool_C[t], t == 3 ? n_rec : 0, t == 3 ? 1 : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace m2c
