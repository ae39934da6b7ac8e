// Host side of the m2c C ABI: argument checking, the layer object, the
// pinned host neuron store, create-time quantization and the entry points.
#include <errno.h>
#include <fcntl.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>
#include <unistd.h>

#include <new>

#include "m2c_internal.h"

using m2c::Store;

namespace {

thread_local char g_err[512] = "";

m2c_status fail(m2c_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

m2c_status hip_fail(hipError_t e, const char* what) {
  if (e == hipErrorOutOfMemory)
    return fail(M2C_ERR_OUT_OF_MEMORY, "%s: %s", what, hipGetErrorString(e));
  return fail(M2C_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIPOK(call, what)                   \
  do {                                      \
    hipError_t e_ = (call);                 \
    if (e_ != hipSuccess) {                 \
      (void)hipGetLastError();              \
      return hip_fail(e_, what);            \
    }                                       \
  } while (0)

// Makes `dev` current for the scope and restores the caller's device.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

int64_t rec_bytes(int d, int tier) {
  const int64_t G = d / 128;
  if (tier == 3) return 6LL * d;
  if (tier == 2) return 3LL * d + 6 * G;
  if (tier == 1) return 3LL * d / 2 + 6 * G;
  return -1;
}

m2c_status check_desc(const m2c_layer_desc* D, int* S_out, int* cap_out) {
  if (!D) return fail(M2C_ERR_INVALID_ARG, "desc is NULL");
  if (D->d_model < 128 || D->d_model > 16384 || D->d_model % 128)
    return fail(M2C_ERR_INVALID_ARG, "d_model %d: need a multiple of 128 in [128, 16384]",
                D->d_model);
  if (D->d_ff < 1 || D->d_ff > 262144)
    return fail(M2C_ERR_INVALID_ARG, "d_ff %d: need [1, 262144]", D->d_ff);
  if (D->pred_rank < 8 || D->pred_rank > 1024 || D->pred_rank % 8)
    return fail(M2C_ERR_INVALID_ARG, "pred_rank %d: need a multiple of 8 in [8, 1024]",
                D->pred_rank);
  if (D->group != 128) return fail(M2C_ERR_INVALID_ARG, "group %d: only 128 is supported", D->group);
  if (D->k_max < 0 || D->k_max > D->d_ff)
    return fail(M2C_ERR_INVALID_ARG, "k_max %d: need [0, d_ff]", D->k_max);
  if (D->max_batch < 1 || D->max_batch > 32)
    return fail(M2C_ERR_INVALID_ARG, "max_batch %d: need [1, 32]", D->max_batch);
  if (D->cache_slots < 0 || D->cache_slots > D->d_ff)
    return fail(M2C_ERR_INVALID_ARG, "cache_slots %d: need [0, d_ff]", D->cache_slots);
  const int64_t cap64 = (int64_t)D->max_batch * D->k_max;
  const int cap = (int)(cap64 < D->d_ff ? cap64 : D->d_ff);
  const int need = cap - D->cache_slots > 0 ? cap - D->cache_slots : 0;
  int S = D->staging_slots;
  if (S == -1) S = need;
  if (S < need)
    return fail(M2C_ERR_INVALID_ARG, "staging_slots %d: at least %d are needed (or -1)",
                D->staging_slots, need);
  if (D->flags & ~(M2C_FLAG_DETERMINISTIC_FFN | M2C_FLAG_DOMINANT_HITS | M2C_FLAG_TIER_POOLS))
    return fail(M2C_ERR_INVALID_ARG, "flags 0x%x: unknown bits", D->flags);
  if (D->flags & M2C_FLAG_TIER_POOLS) {
    if (D->flags & M2C_FLAG_DETERMINISTIC_FFN)
      return fail(M2C_ERR_INVALID_ARG, "tier pools do not take the deterministic FFN");
    if (D->max_batch != 1 || D->d_model > 8192 || D->d_ff > 32768 || D->staging_slots != -1)
      return fail(M2C_ERR_INVALID_ARG, "tier pools need max_batch 1, d_model <= 8192, d_ff <= "
                  "32768 and staging_slots -1");
    int64_t sum = 0;
    for (int t = 1; t <= 3; ++t) {
      if (D->tier_slots[t] < 0 || D->tier_slots[t] > D->d_ff)
        return fail(M2C_ERR_INVALID_ARG, "tier_slots[%d] %d: need [0, d_ff]", t, D->tier_slots[t]);
      sum += D->tier_slots[t];
    }
    if (sum != D->cache_slots)
      return fail(M2C_ERR_INVALID_ARG, "tier_slots sum to %lld, cache_slots is %d", (long long)sum,
                  D->cache_slots);
    S = 0;
    for (int t = 1; t <= 3; ++t) S += cap - D->tier_slots[t] > 0 ? cap - D->tier_slots[t] : 0;
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || D->device < 0 || D->device >= ndev)
    return fail(M2C_ERR_INVALID_ARG, "device %d: %d HIP devices visible", D->device, ndev);
  *S_out = S;
  *cap_out = cap;
  return M2C_OK;
}

void fill_info_layout(m2c_layer* L) {
  const m2c_layer_desc& D = L->desc;
  m2c_layer_info& I = L->info;
  memset(&I, 0, sizeof(I));
  for (int t = 1; t <= 3; ++t) {
    I.record_bytes[t] = (int32_t)rec_bytes(D.d_model, t);
    I.record_stride[t] = (int32_t)round_up(rec_bytes(D.d_model, t), 16);
  }
  I.slot_bytes = 6 * D.d_model;
  I.cache_slots = D.cache_slots;
  I.staging_slots = L->S;
  // the slot arena: one pool per tier (FP16 first) or one pool of FP16-sized
  // slots shared by the tiers, then the zero slot
  L->pools = (D.flags & M2C_FLAG_TIER_POOLS) != 0;
  int64_t arena = 0;
  if (L->pools) {
    int first = 0, rf = 0;
    for (int t = 3; t >= 1; --t) {
      L->pool_C[t] = D.tier_slots[t];
      L->pool_S[t] = L->cap - L->pool_C[t] > 0 ? L->cap - L->pool_C[t] : 0;
      L->pool_rf[t] = rf;
      I.pool_first[t] = first;
      I.pool_slots[t] = L->pool_C[t] + L->pool_S[t];
      I.pool_resident[t] = L->pool_C[t];
      I.pool_stride[t] = I.record_stride[t];
      L->map.base[t] = (uint32_t)arena;
      L->map.first[t] = first;
      L->map.count[t] = I.pool_slots[t];
      L->map.stride[t] = (uint32_t)I.record_stride[t];
      arena += (int64_t)I.pool_slots[t] * I.pool_stride[t];
      first += I.pool_slots[t];
      rf += L->pool_C[t];
    }
  } else {
    for (int t = 1; t <= 3; ++t) {
      I.pool_first[t] = 0;
      I.pool_slots[t] = D.cache_slots + L->S;
      I.pool_resident[t] = D.cache_slots;
      I.pool_stride[t] = I.slot_bytes;
      L->map.base[t] = 0;
      L->map.first[t] = 0;
      L->map.count[t] = D.cache_slots + L->S;
      L->map.stride[t] = (uint32_t)I.slot_bytes;
    }
    arena = (int64_t)(D.cache_slots + L->S) * I.slot_bytes;
  }
  L->map.base[0] = 0;
  L->map.first[0] = 0;
  L->map.count[0] = 0;
  L->map.stride[0] = (uint32_t)I.slot_bytes;
  L->map.zero = (uint32_t)arena;  // below 4 GiB when the one-launch FFN runs (checked there)
  L->arena_bytes = arena + I.slot_bytes;
  I.slot_arena_bytes = L->arena_bytes;
  I.plan_capacity = L->cap;
  m2c_plan_layout& P = L->layout;
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    int64_t o = off;
    off = round_up(off + (bytes > 0 ? bytes : 1), 256);
    return o;
  };
  const int64_t c = L->cap;
  P.counts = take(4 * M2C_NCOUNTS);
  P.req_ids = take(4 * c);
  P.req_tier = take(c);
  P.req_hit = take(c);
  P.req_slot = take(4 * c);
  P.req_mask = take(4 * c);
  P.fill_ids = take(4 * c);
  P.fill_tier = take(c);
  P.fill_slot = take(4 * c);
  P.fill_from = take(c);
  P.evicted_ids = take(4 * c);
  P.work_slot = take(4 * (c + m2c::kWorkSlotPad));
  P.work_mask = take(4 * c);
  L->plan_core_bytes = off;
  P.ffn_tasks = take(m2c::ffn_tasks_used(L)
                         ? m2c::ffn_task_table_bytes(m2c::ffn_fused_grid(
                               (int)L->desc.d_model, (int)c, L->num_cus))
                         : 0);
  P.total_bytes = off;
  I.plan_bytes = off;
}

void release_store(Store* s) {
  if (!s) return;
  if (--s->refs > 0) return;
  for (int t = 1; t <= 3; ++t)
    if (s->host[t]) (void)hipHostFree(s->host[t]);
  delete s;
}

void free_layer(m2c_layer* L) {
  if (!L) return;
  {
    DeviceGuard g(L->desc.device);
    if (L->dev_base) {
      (void)hipDeviceSynchronize();
      (void)hipFree(L->dev_base);
    }
    release_store(L->store);
    if (L->dram) m2c::dram_ref(L->dram, -1);
  }
  delete L;
}

// Device memory of a layer: one allocation, carved in 256-byte pieces.
m2c_status alloc_device(m2c_layer* L, bool with_bias) {
  const m2c_layer_desc& D = L->desc;
  const int64_t d = D.d_model, dff = D.d_ff, r = D.pred_rank, C = D.cache_slots;
  const int64_t cap = L->cap, mb = D.max_batch;
  const int64_t np = L->pools ? 3 : 1;
  const int n_slices = (int)((d + 511) / 512);
  // (column slices) x (neuron groups) workgroups for the down projection:
  // about 512, at most 64 partial rows, groups of at least 16 neurons.
  int ng = 512 / n_slices;
  if (ng < 1) ng = 1;
  if (ng > 64) ng = 64;
  const int ng_cap = (int)(cap / 16 > 1 ? cap / 16 : 1);
  if (ng > ng_cap) ng = ng_cap;
  L->ffn_groups = ng;
  struct Piece { void** dst; int64_t bytes; };
  void* p_pred_a; void* p_pred_b; void* p_bias; void* p_z; void* p_scores; void* p_slots;
  void* p_h; void* p_ypart; void* p_slot_of; void* p_slot_key; void* p_slot_tier;
  void* p_slot_last; void* p_lru; void* p_lru_cur; void* p_new_pos; void* p_work_pos;
  void* p_vslot; void* p_vold; void* p_fill_pos; void* p_prev_tier; void* p_have; void* p_stats;
  void* p_status;
  void* p_gen; void* p_hw; void* p_pool_plan; void* p_abort; void* p_pool_lists;
  void* p_pool_counts;
  Piece pieces[] = {
      // C resident + S staging slots, then one slot that stays zero: padding
      // lanes of the FFN kernels read it instead of branching around loads
      {&p_slots, L->arena_bytes},
      {&p_pred_a, r * d * 2},
      {&p_pred_b, dff * r * 2},
      {&p_bias, with_bias ? dff * 4 : 0},
      {&p_z, mb * r * 4},
      {&p_scores, mb * dff * 4},
      {&p_h, 4 * cap * mb * 8},
      {&p_ypart, (int64_t)ng * mb * d * 4},
      {&p_slot_of, (L->pools ? 3 : 1) * dff * 4},
      {&p_slot_key, C * 4},
      {&p_slot_tier, C},
      {&p_slot_last, C * 4},
      {&p_lru, 2 * C * 4},
      {&p_lru_cur, 3 * 4},
      // plan scratch, one set per pool (the pools are planned side by side)
      {&p_new_pos, np * cap * 4},
      {&p_work_pos, np * cap * 4},
      {&p_vslot, np * cap * 4},
      {&p_vold, np * cap * 4},
      {&p_fill_pos, np * cap * 4},
      {&p_prev_tier, np * cap},
      {&p_have, (C + L->S) * 4},
      {&p_stats, 16 * 8},
      {&p_status, 4},
      {&p_gen, (int64_t)m2c::ffn_fused_grid((int)d, (int)cap, L->num_cus) * 8},
      {&p_hw, cap * 8},
      {&p_pool_plan, L->pools ? 3 * L->plan_core_bytes : 0},
      {&p_abort, 4},
      {&p_pool_lists, L->pools ? 3 * dff * 4 : 0},
      {&p_pool_counts, L->pools ? 3 * 32 * 4 : 0},
  };
  int64_t total = 0;
  int64_t offs[sizeof(pieces) / sizeof(pieces[0])];
  for (size_t q = 0; q < sizeof(pieces) / sizeof(pieces[0]); ++q) {
    offs[q] = total;
    total = round_up(total + (pieces[q].bytes > 0 ? pieces[q].bytes : 1), 256);
  }
  void* base = nullptr;
  HIPOK(hipMalloc(&base, total), "hipMalloc(layer device memory)");
  L->dev_base = (uint8_t*)base;
  L->dev_bytes = total;
  for (size_t q = 0; q < sizeof(pieces) / sizeof(pieces[0]); ++q)
    *pieces[q].dst = L->dev_base + offs[q];
  L->slots = (uint8_t*)p_slots;
  L->pred_a = (uint16_t*)p_pred_a;
  L->pred_b = (uint16_t*)p_pred_b;
  L->bias = with_bias ? (float*)p_bias : nullptr;
  L->z = (float*)p_z;
  L->scores = (float*)p_scores;
  L->ab = (float2*)p_h;
  L->y_part = (float*)p_ypart;
  L->st.slot_of = (int32_t*)p_slot_of;
  L->st.slot_key = (int32_t*)p_slot_key;
  L->st.slot_tier = (uint8_t*)p_slot_tier;
  L->st.slot_last = (int32_t*)p_slot_last;
  L->st.lru = (int32_t*)p_lru;
  L->st.lru_cur = (int32_t*)p_lru_cur;
  L->st.new_pos = (int32_t*)p_new_pos;
  L->st.work_pos = (int32_t*)p_work_pos;
  L->st.vict_slot = (int32_t*)p_vslot;
  L->st.vict_old = (int32_t*)p_vold;
  L->st.fill_pos = (int32_t*)p_fill_pos;
  L->st.prev_tier = (uint8_t*)p_prev_tier;
  L->st.slot_rec = (int32_t*)p_have;
  L->st.stats = (unsigned long long*)p_stats;
  L->st.status = (int32_t*)p_status;
  L->st.ffn_gen = (unsigned long long*)p_gen;
  L->st.ffn_hw = (unsigned long long*)p_hw;
  L->pool_plan = (uint8_t*)p_pool_plan;
  L->plan_abort = (int32_t*)p_abort;
  L->pool_lists = (int32_t*)p_pool_lists;
  L->pool_counts = (int32_t*)p_pool_counts;
  L->info.device_bytes = total;
  HIPOK(hipMemset(L->slots + L->map.zero, 0, L->info.slot_bytes), "clear the zero slot");
  HIPOK(hipMemset(L->plan_abort, 0, 4), "clear the plan abort word");
  HIPOK(hipMemset(L->st.status, 0, 4), "clear the status word");
  L->ffn_grid = m2c::ffn_fused_grid((int)d, (int)cap, L->num_cus);
  HIPOK(hipMemset(L->st.ffn_gen, 0, (size_t)(L->ffn_grid > 0 ? L->ffn_grid : 1) * 8),
        "clear the FFN workgroup counters");
  HIPOK(hipMemset(L->st.ffn_hw, 0, (size_t)(cap > 0 ? cap : 1) * 8), "clear the FFN h words");
  return M2C_OK;
}

m2c_status upload_predictor(m2c_layer* L, const uint16_t* pred_a, const uint16_t* pred_b,
                            const float* bias) {
  const m2c_layer_desc& D = L->desc;
  HIPOK(hipMemcpy(L->pred_a, pred_a, (size_t)D.pred_rank * D.d_model * 2, hipMemcpyHostToDevice),
        "upload pred_a");
  HIPOK(hipMemcpy(L->pred_b, pred_b, (size_t)D.d_ff * D.pred_rank * 2, hipMemcpyHostToDevice),
        "upload pred_b");
  if (bias)
    HIPOK(hipMemcpy(L->bias, bias, (size_t)D.d_ff * 4, hipMemcpyHostToDevice), "upload bias");
  HIPOK(m2c::launch_reset(L, 0), "reset kernel");
  HIPOK(hipDeviceSynchronize(), "layer init");
  return M2C_OK;
}

// Builds the three records of every neuron on the device and copies them
// into the pinned store.
m2c_status build_store(m2c_layer* L, const uint16_t* w_gate, const uint16_t* w_up,
                       const uint16_t* w_down) {
  const int d = L->desc.d_model, dff = L->desc.d_ff;
  Store* S = L->store;
  for (int t = 1; t <= 3; ++t) {
    void* p = nullptr;
    HIPOK(hipHostMalloc(&p, (size_t)dff * S->stride[t], hipHostMallocDefault),
          "hipHostMalloc(neuron store)");
    S->host[t] = (uint8_t*)p;
    S->bytes += (int64_t)dff * S->stride[t];
  }
  const size_t wbytes = (size_t)dff * d * 2;
  const int chunk = dff < 4096 ? dff : 4096;
  const size_t rbytes = (size_t)chunk * (S->stride[1] + S->stride[2] + S->stride[3]);
  void *wg = nullptr, *wu = nullptr, *wd = nullptr, *wdT = nullptr, *rec = nullptr;
  m2c_status rc = M2C_OK;
  hipError_t e = hipMalloc(&wg, wbytes);
  if (e == hipSuccess) e = hipMalloc(&wu, wbytes);
  if (e == hipSuccess) e = hipMalloc(&wd, wbytes);
  if (e == hipSuccess) e = hipMalloc(&wdT, wbytes);
  if (e == hipSuccess) e = hipMalloc(&rec, rbytes);
  if (e == hipSuccess) e = hipMemcpy(wg, w_gate, wbytes, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(wu, w_up, wbytes, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(wd, w_down, wbytes, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = m2c::launch_transpose_u16((const uint16_t*)wd, (uint16_t*)wdT, d, dff, 0);
  uint8_t* r16 = (uint8_t*)rec;
  uint8_t* r8 = r16 + (size_t)chunk * S->stride[3];
  uint8_t* r4 = r8 + (size_t)chunk * S->stride[2];
  for (int i0 = 0; e == hipSuccess && i0 < dff; i0 += chunk) {
    const int n = dff - i0 < chunk ? dff - i0 : chunk;
    e = hipMemset(rec, 0, rbytes);
    if (e == hipSuccess)
      e = m2c::launch_quantize_records((const uint16_t*)wg, (const uint16_t*)wu,
                                       (const uint16_t*)wdT, d, i0, n, r16, S->stride[3], r8,
                                       S->stride[2], r4, S->stride[1], 0);
    if (e == hipSuccess)
      e = hipMemcpy(S->host[3] + (size_t)i0 * S->stride[3], r16, (size_t)n * S->stride[3],
                    hipMemcpyDeviceToHost);
    if (e == hipSuccess)
      e = hipMemcpy(S->host[2] + (size_t)i0 * S->stride[2], r8, (size_t)n * S->stride[2],
                    hipMemcpyDeviceToHost);
    if (e == hipSuccess)
      e = hipMemcpy(S->host[1] + (size_t)i0 * S->stride[1], r4, (size_t)n * S->stride[1],
                    hipMemcpyDeviceToHost);
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    (void)hipGetLastError();
    rc = hip_fail(e, "building the neuron store");
  }
  for (void* p : {wg, wu, wd, wdT, rec})
    if (p) (void)hipFree(p);
  return rc;
}

m2c_status new_layer(const m2c_layer_desc* desc, m2c_layer** out, m2c_layer** made) {
  if (!out) return fail(M2C_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int S = 0, cap = 0;
  m2c_status rc = check_desc(desc, &S, &cap);
  if (rc != M2C_OK) return rc;
  m2c_layer* L = new (std::nothrow) m2c_layer();
  if (!L) return fail(M2C_ERR_OUT_OF_MEMORY, "host allocation failed");
  L->desc = *desc;
  L->S = S;
  L->cap = cap;
  fill_info_layout(L);
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, desc->device) != hipSuccess) {
    delete L;
    return fail(M2C_ERR_HIP, "hipGetDeviceProperties failed");
  }
  L->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 1;
  *made = L;
  return M2C_OK;
}

}  // namespace

namespace m2c {

m2c_status api_fail(m2c_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

m2c_status check_predict_args(const m2c_layer* L, const uint16_t* x, int batch, int k, int n_fp16,
                              int n_int8, const uint8_t* tier_map) {
  if (!L || !x || !tier_map) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (batch < 1 || batch > L->desc.max_batch)
    return fail(M2C_ERR_CAPACITY, "batch %d outside [1, max_batch=%d]", batch, L->desc.max_batch);
  if (k < 0 || k > L->desc.k_max)
    return fail(M2C_ERR_CAPACITY, "k %d outside [0, k_max=%d]", k, L->desc.k_max);
  if (n_fp16 < 0 || n_int8 < 0 || (int64_t)n_fp16 + n_int8 > k)
    return fail(M2C_ERR_INVALID_ARG, "tier counts %d + %d exceed k %d", n_fp16, n_int8, k);
  return M2C_OK;
}

}  // namespace m2c

extern "C" {

int64_t m2c_record_bytes(int32_t d_model, int32_t tier) {
  if (d_model <= 0 || d_model % 128) return -1;
  return rec_bytes(d_model, tier);
}

const char* m2c_last_error(void) { return g_err; }

#ifndef M2C_SOURCE_ID
#define M2C_SOURCE_ID "unknown"
#endif
const char* m2c_build_id(void) { return M2C_SOURCE_ID; }

m2c_status m2c_layer_create(const m2c_layer_desc* desc, const uint16_t* w_gate,
                            const uint16_t* w_up, const uint16_t* w_down, const uint16_t* pred_a,
                            const uint16_t* pred_b, const float* score_bias, m2c_layer** out) {
  if (!w_gate || !w_up || !w_down || !pred_a || !pred_b)
    return fail(M2C_ERR_INVALID_ARG, "a weight or predictor pointer is NULL");
  m2c_layer* L = nullptr;
  m2c_status rc = new_layer(desc, out, &L);
  if (rc != M2C_OK) return rc;
  DeviceGuard g(desc->device);
  if (!g.ok) {
    delete L;
    return fail(M2C_ERR_HIP, "hipSetDevice(%d) failed", desc->device);
  }
  L->store = new (std::nothrow) Store();
  if (!L->store) {
    delete L;
    return fail(M2C_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  L->store->device = desc->device;
  L->store->d_model = desc->d_model;
  L->store->d_ff = desc->d_ff;
  for (int t = 1; t <= 3; ++t) L->store->stride[t] = L->info.record_stride[t];
  rc = build_store(L, w_gate, w_up, w_down);
  if (rc == M2C_OK) rc = alloc_device(L, score_bias != nullptr);
  if (rc == M2C_OK) rc = upload_predictor(L, pred_a, pred_b, score_bias);
  if (rc != M2C_OK) {
    char keep[sizeof(g_err)];
    memcpy(keep, g_err, sizeof(keep));
    free_layer(L);
    memcpy(g_err, keep, sizeof(keep));
    return rc;
  }
  L->info.host_store_bytes = L->store->bytes;
  *out = L;
  return M2C_OK;
}

m2c_status m2c_layer_create_shared(const m2c_layer_desc* desc, const m2c_layer* weights_of,
                                   const uint16_t* pred_a, const uint16_t* pred_b,
                                   const float* score_bias, m2c_layer** out) {
  if (!weights_of || !pred_a || !pred_b)
    return fail(M2C_ERR_INVALID_ARG, "weights_of or a predictor pointer is NULL");
  if (!weights_of->store)
    return fail(M2C_ERR_INVALID_ARG, "weights_of reads its records from a DRAM cache: create the "
                "layer with m2c_layer_create_from_dram instead");
  if (!desc || desc->d_model != weights_of->desc.d_model || desc->d_ff != weights_of->desc.d_ff ||
      desc->device != weights_of->desc.device)
    return fail(M2C_ERR_INVALID_ARG, "d_model, d_ff and device must match weights_of");
  m2c_layer* L = nullptr;
  m2c_status rc = new_layer(desc, out, &L);
  if (rc != M2C_OK) return rc;
  DeviceGuard g(desc->device);
  if (!g.ok) {
    delete L;
    return fail(M2C_ERR_HIP, "hipSetDevice(%d) failed", desc->device);
  }
  L->store = weights_of->store;
  L->store->refs++;
  rc = alloc_device(L, score_bias != nullptr);
  if (rc == M2C_OK) rc = upload_predictor(L, pred_a, pred_b, score_bias);
  if (rc != M2C_OK) {
    char keep[sizeof(g_err)];
    memcpy(keep, g_err, sizeof(keep));
    free_layer(L);
    memcpy(g_err, keep, sizeof(keep));
    return rc;
  }
  L->info.host_store_bytes = L->store->bytes;
  *out = L;
  return M2C_OK;
}

m2c_status m2c_layer_create_from_dram(const m2c_layer_desc* desc, m2c_dram* dram, int32_t index,
                                      const uint16_t* pred_a, const uint16_t* pred_b,
                                      const float* score_bias, m2c_layer** out) {
  if (!dram || !pred_a || !pred_b)
    return fail(M2C_ERR_INVALID_ARG, "dram or a predictor pointer is NULL");
  if (!m2c::dram_pinned(dram))
    return fail(M2C_ERR_INVALID_ARG, "the DRAM cache uses plain host memory; GPU fills need a "
                "pinned one (no M2C_DRAM_HOST_MEMORY)");
  if (index < 0 || index >= m2c::dram_layers(dram))
    return fail(M2C_ERR_INVALID_ARG, "index %d outside [0, %d)", index, m2c::dram_layers(dram));
  m2c_layer* L = nullptr;
  m2c_status rc = new_layer(desc, out, &L);
  if (rc != M2C_OK) return rc;
  int64_t want = 0;
  for (int t = 1; t <= 3; ++t) want += (int64_t)desc->d_ff * L->info.record_stride[t];
  if (want != m2c::dram_layer_bytes(dram) || desc->device != m2c::dram_device(dram)) {
    const long long have = (long long)m2c::dram_layer_bytes(dram);
    delete L;
    return fail(M2C_ERR_INVALID_ARG, "the DRAM cache holds %lld-byte layers on device %d; this "
                "layer needs %lld bytes on device %d", have, m2c::dram_device(dram),
                (long long)want, desc->device);
  }
  DeviceGuard g(desc->device);
  if (!g.ok) {
    delete L;
    return fail(M2C_ERR_HIP, "hipSetDevice(%d) failed", desc->device);
  }
  L->dram = dram;
  L->dram_index = index;
  m2c::dram_ref(dram, 1);
  rc = alloc_device(L, score_bias != nullptr);
  if (rc == M2C_OK) rc = upload_predictor(L, pred_a, pred_b, score_bias);
  if (rc != M2C_OK) {
    char keep[sizeof(g_err)];
    memcpy(keep, g_err, sizeof(keep));
    free_layer(L);
    memcpy(g_err, keep, sizeof(keep));
    return rc;
  }
  L->info.host_store_bytes = 0;
  *out = L;
  return M2C_OK;
}

m2c_status m2c_layer_write_store(const m2c_layer* L, const char* path, int64_t offset,
                                 int64_t* padded_bytes) {
  if (!L || !path) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (!L->store) return fail(M2C_ERR_INVALID_ARG, "the layer has no host store of its own");
  if (offset < 0 || offset % 4096)
    return fail(M2C_ERR_INVALID_ARG, "offset %lld: need a multiple of 4096", (long long)offset);
  const int fd = open(path, O_WRONLY | O_CREAT, 0644);
  if (fd < 0) return fail(M2C_ERR_INVALID_ARG, "open(%s): %s", path, strerror(errno));
  int64_t pos = offset;
  m2c_status rc = M2C_OK;
  for (int t = 3; t >= 1 && rc == M2C_OK; --t) {
    const uint8_t* p = L->store->host[t];
    int64_t left = (int64_t)L->desc.d_ff * L->store->stride[t];
    while (left > 0) {
      const ssize_t w = pwrite(fd, p, (size_t)(left < (1 << 30) ? left : (1 << 30)), pos);
      if (w < 0 && errno == EINTR) continue;
      if (w <= 0) {
        rc = fail(M2C_ERR_INVALID_ARG, "write(%s): %s", path, strerror(errno));
        break;
      }
      p += w;
      pos += w;
      left -= w;
    }
  }
  const int64_t pad = (4096 - (pos - offset) % 4096) % 4096;
  if (rc == M2C_OK && pad) {
    static const uint8_t zeros[4096] = {0};
    if (pwrite(fd, zeros, (size_t)pad, pos) != (ssize_t)pad)
      rc = fail(M2C_ERR_INVALID_ARG, "write(%s): %s", path, strerror(errno));
    pos += pad;
  }
  if (close(fd) != 0 && rc == M2C_OK)
    rc = fail(M2C_ERR_INVALID_ARG, "close(%s): %s", path, strerror(errno));
  if (rc == M2C_OK && padded_bytes) *padded_bytes = pos - offset;
  return rc;
}

m2c_status m2c_layer_destroy(m2c_layer* layer) {
  free_layer(layer);
  return M2C_OK;
}

m2c_status m2c_layer_get_info(const m2c_layer* layer, m2c_layer_info* out) {
  if (!layer || !out) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  *out = layer->info;
  return M2C_OK;
}

m2c_status m2c_plan_get_layout(const m2c_layer* layer, m2c_plan_layout* out) {
  if (!layer || !out) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  *out = layer->layout;
  return M2C_OK;
}

m2c_status m2c_predict_rank(m2c_layer* L, const uint16_t* x, int32_t batch, int32_t k,
                            int32_t n_fp16, int32_t n_int8, float* scores, uint8_t* tier_map,
                            void* stream) {
  m2c_status rc = m2c::check_predict_args(L, x, batch, k, n_fp16, n_int8, tier_map);
  if (rc != M2C_OK) return rc;
  DeviceGuard g(L->desc.device);
  hipStream_t s = (hipStream_t)stream;
  float* sc = scores ? scores : L->scores;
  HIPOK(m2c::launch_predict(L, x, batch, L->z, sc, s), "predictor launch");
  HIPOK(m2c::launch_select(sc, batch, L->desc.d_ff, k, n_fp16, n_int8, tier_map, s),
        "select launch");
  return M2C_OK;
}

m2c_status m2c_cache_plan(m2c_layer* L, const uint8_t* tier_map, int32_t batch, int64_t step,
                          void* plan, void* stream) {
  if (!L || !tier_map || !plan) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)plan) % 256) return fail(M2C_ERR_INVALID_ARG, "plan must be 256-byte aligned");
  if (batch < 1 || batch > L->desc.max_batch)
    return fail(M2C_ERR_CAPACITY, "batch %d outside [1, max_batch=%d]", batch, L->desc.max_batch);
  if (step < 0 || step >= 0x7fffffffLL) return fail(M2C_ERR_INVALID_ARG, "step %lld out of range",
                                                    (long long)step);
  if (step <= L->last_step)
    return fail(M2C_ERR_STATE, "step %lld is not after the previous step %lld", (long long)step,
                (long long)L->last_step);
  DeviceGuard g(L->desc.device);
  HIPOK(m2c::launch_plan(L, tier_map, batch, (int)step, (uint8_t*)plan, (hipStream_t)stream),
        "plan launch");
  L->last_step = step;
  return M2C_OK;
}

m2c_status m2c_cache_fill(m2c_layer* L, const void* plan, void* stream) {
  if (!L || !plan) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  DeviceGuard g(L->desc.device);
  if (!L->dram) {
    HIPOK(m2c::launch_fill(L, (const uint8_t*)plan, L->store->host, (hipStream_t)stream),
          "fill launch");
    return M2C_OK;
  }
  // records in a DRAM cache: hold the layer's buffer while the fill is
  // enqueued, release it behind an event after the fill
  const uint8_t* base = nullptr;
  int slot = -1;
  m2c_status rc = m2c::dram_acquire(L->dram, L->dram_index, &base, &slot);
  if (rc != M2C_OK) return rc;
  const uint8_t* host[4] = {nullptr, nullptr, nullptr, nullptr};
  int64_t off = 0;
  for (int t = 3; t >= 1; --t) {
    host[t] = base + off;
    off += (int64_t)L->desc.d_ff * L->info.record_stride[t];
  }
  hipError_t e = m2c::launch_fill(L, (const uint8_t*)plan, host, (hipStream_t)stream);
  hipEvent_t ev = nullptr;
  if (e == hipSuccess && slot >= 0) {
    ev = m2c::dram_event(L->dram);
    e = ev ? hipEventRecord(ev, (hipStream_t)stream) : hipErrorOutOfMemory;
  }
  if (e != hipSuccess) {
    // nothing can be known about the fill: wait for the device before the
    // buffer may be reused
    (void)hipGetLastError();
    (void)hipDeviceSynchronize();
    m2c::dram_release(L->dram, slot, nullptr);
    return hip_fail(e, "fill launch");
  }
  m2c::dram_release(L->dram, slot, ev);
  return M2C_OK;
}

m2c_status m2c_sparse_ffn(m2c_layer* L, const uint16_t* x, int32_t batch, const void* plan,
                          float* y, void* stream) {
  if (!L || !x || !plan || !y) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (batch < 1 || batch > L->desc.max_batch)
    return fail(M2C_ERR_CAPACITY, "batch %d outside [1, max_batch=%d]", batch, L->desc.max_batch);
  DeviceGuard g(L->desc.device);
  HIPOK(m2c::launch_ffn(L, x, batch, (const uint8_t*)plan, y, (hipStream_t)stream), "ffn launch");
  return M2C_OK;
}

m2c_status m2c_layer_reset_cache(m2c_layer* L, void* stream) {
  if (!L) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  DeviceGuard g(L->desc.device);
  HIPOK(m2c::launch_reset(L, (hipStream_t)stream), "reset launch");
  L->last_step = -1;
  return M2C_OK;
}

m2c_status m2c_layer_stats(const m2c_layer* L, m2c_stats* out) {
  if (!L || !out) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  DeviceGuard g(L->desc.device);
  long long st[16];
  int32_t status = 0;
  HIPOK(hipDeviceSynchronize(), "synchronize");
  HIPOK(hipMemcpy(st, L->st.stats, sizeof(st), hipMemcpyDeviceToHost), "read stats");
  HIPOK(hipMemcpy(&status, L->st.status, 4, hipMemcpyDeviceToHost), "read status");
  if (status) {
    HIPOK(hipMemset(L->st.status, 0, 4), "clear the status word");
    if (status & m2c::M2C_STATUS_FFN_WAIT)
      return fail(M2C_ERR_STATE, "a sparse FFN call gave up waiting for an h value and used 0 "
                  "(status 0x%x): its output is wrong", status);
    return fail(M2C_ERR_CAPACITY, "a cache plan since the last check had more active neurons than "
                "the layer was created for (k_max * max_batch); it was left empty (status 0x%x)",
                status);
  }
  memset(out, 0, sizeof(*out));
  out->plans = st[0];
  out->req = st[1];
  out->hit = st[2];
  out->refill = st[3];
  out->new_ = st[4];
  out->bypass = st[5];
  out->evict = st[6];
  out->fill[1] = st[7];
  out->fill[2] = st[8];
  out->fill[3] = st[9];
  out->req_tier[1] = st[10];
  out->req_tier[2] = st[11];
  out->req_tier[3] = st[12];
  out->derived[1] = st[13];
  out->derived[2] = st[14];
  for (int t = 1; t <= 3; ++t) {
    out->fill_bytes += out->fill[t] * L->info.record_bytes[t];
    out->host_bytes += (out->fill[t] - out->derived[t]) * L->info.record_bytes[t];
    out->req_bytes += out->req_tier[t] * L->info.record_bytes[t];
  }
  return M2C_OK;
}

m2c_status m2c_debug_read_record(const m2c_layer* L, int32_t tier, int32_t neuron, void* out,
                                 size_t bytes) {
  if (!L || !out) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (tier < 1 || tier > 3 || neuron < 0 || neuron >= L->desc.d_ff)
    return fail(M2C_ERR_INVALID_ARG, "tier %d / neuron %d out of range", tier, neuron);
  const int64_t stride = L->info.record_stride[tier];
  if ((int64_t)bytes > stride)
    return fail(M2C_ERR_INVALID_ARG, "%zu bytes exceed the record stride %lld", bytes,
                (long long)stride);
  if (L->store) {
    memcpy(out, L->store->host[tier] + (int64_t)neuron * stride, bytes);
    return M2C_OK;
  }
  const uint8_t* base = nullptr;
  int slot = -1;
  m2c_status rc = m2c::dram_acquire(L->dram, L->dram_index, &base, &slot);
  if (rc != M2C_OK) return rc;
  int64_t off = 0;
  for (int t = 3; t > tier; --t) off += (int64_t)L->desc.d_ff * L->info.record_stride[t];
  memcpy(out, base + off + (int64_t)neuron * stride, bytes);
  m2c::dram_release(L->dram, slot, nullptr);
  return M2C_OK;
}

m2c_status m2c_debug_read_slot(const m2c_layer* L, int32_t slot, void* out, size_t bytes) {
  if (!L || !out) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  int tier = 0;
  for (int t = 1; t <= 3; ++t)
    if (slot >= L->info.pool_first[t] && slot < L->info.pool_first[t] + L->info.pool_slots[t])
      tier = t;
  if (slot < 0 || tier == 0 || (int64_t)bytes > L->info.pool_stride[tier])
    return fail(M2C_ERR_INVALID_ARG, "slot %d / %zu bytes out of range", slot, bytes);
  DeviceGuard g(L->desc.device);
  HIPOK(hipDeviceSynchronize(), "synchronize");
  const int64_t off = L->map.base[tier] + (int64_t)(slot - L->map.first[tier]) * L->map.stride[tier];
  HIPOK(hipMemcpy(out, L->slots + off, bytes, hipMemcpyDeviceToHost), "read slot");
  return M2C_OK;
}

m2c_status m2c_debug_read_pool_tables(const m2c_layer* L, int32_t tier, int32_t* slot_of,
                                      int32_t* slot_key, int32_t* slot_last) {
  if (!L) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (!L->pools || tier < 1 || tier > 3)
    return fail(M2C_ERR_INVALID_ARG, "tier %d: the layer has %s", tier,
                L->pools ? "pools 1..3" : "no tier pools");
  DeviceGuard g(L->desc.device);
  const m2c::DeviceState v = m2c::pool_state(L, tier);
  const size_t C = (size_t)L->pool_C[tier];
  HIPOK(hipDeviceSynchronize(), "synchronize");
  if (slot_of)
    HIPOK(hipMemcpy(slot_of, v.slot_of, (size_t)L->desc.d_ff * 4, hipMemcpyDeviceToHost),
          "read slot_of");
  if (slot_key && C)
    HIPOK(hipMemcpy(slot_key, v.slot_key, C * 4, hipMemcpyDeviceToHost), "read slot_key");
  if (slot_last && C)
    HIPOK(hipMemcpy(slot_last, v.slot_last, C * 4, hipMemcpyDeviceToHost), "read slot_last");
  return M2C_OK;
}

m2c_status m2c_debug_poison_fill_slots(m2c_layer* L, const void* plan, void* stream) {
  if (!L || !plan) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  DeviceGuard g(L->desc.device);
  HIPOK(m2c::launch_poison_fill_slots(L, (const uint8_t*)plan, (hipStream_t)stream),
        "poison launch");
  return M2C_OK;
}

m2c_status m2c_debug_ffn_withhold_h(m2c_layer* L, int32_t polls) {
  if (!L) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  if (polls < 0) return fail(M2C_ERR_INVALID_ARG, "polls %d: need >= 0", polls);
  L->ffn_withhold = polls;
  return M2C_OK;
}

m2c_status m2c_debug_read_tables(const m2c_layer* L, int32_t* slot_of, int32_t* slot_key,
                                 uint8_t* slot_tier, int32_t* slot_last) {
  if (!L) return fail(M2C_ERR_INVALID_ARG, "NULL argument");
  DeviceGuard g(L->desc.device);
  const size_t C = (size_t)L->desc.cache_slots;
  HIPOK(hipDeviceSynchronize(), "synchronize");
  if (slot_of)
    HIPOK(hipMemcpy(slot_of, L->st.slot_of, (size_t)L->desc.d_ff * 4, hipMemcpyDeviceToHost),
          "read slot_of");
  if (slot_key && C)
    HIPOK(hipMemcpy(slot_key, L->st.slot_key, C * 4, hipMemcpyDeviceToHost), "read slot_key");
  if (slot_tier && C)
    HIPOK(hipMemcpy(slot_tier, L->st.slot_tier, C, hipMemcpyDeviceToHost), "read slot_tier");
  if (slot_last && C)
    HIPOK(hipMemcpy(slot_last, L->st.slot_last, C * 4, hipMemcpyDeviceToHost), "read slot_last");
  return M2C_OK;
}

}  // extern "C"
