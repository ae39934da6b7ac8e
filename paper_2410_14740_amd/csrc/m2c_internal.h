// Internal definitions of the m2c HIP library (gfx950). Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "m2c.h"

namespace m2c {

// Bits of the per-layer device status word, reported (and cleared) by
// m2c_layer_stats.
constexpr int M2C_STATUS_PLAN_OVERFLOW = 2;  // a tier map had more active neurons than cap
constexpr int M2C_STATUS_FFN_WAIT = 4;      // a sparse FFN gave up waiting for an h value
// Spare entries after the plan's work_slot array: the FFN kernels read slot
// ids in wave-uniform blocks (groups of four at batch 1, a whole run of up to
// 512 items in the batched down projection) that may run past the last item.
constexpr int kWorkSlotPad = 512;

// ---------------------------------------------------------------------------
// Host-side layer object

// Pinned host-DRAM neuron store: every neuron at all three tiers, record
// stores back to back per tier. Shared (refcounted) between layers created
// with m2c_layer_create_shared.
struct Store {
  int refs = 1;
  int device = 0;
  int d_model = 0, d_ff = 0;
  uint8_t* host[4] = {nullptr, nullptr, nullptr, nullptr};  // by tier, [1..3]
  int64_t stride[4] = {0, 0, 0, 0};
  int64_t bytes = 0;
};

// Offsets of the per-layer device scratch used by the plan kernel.
struct DeviceState {
  int32_t* slot_of = nullptr;    // [d_ff]
  int32_t* slot_key = nullptr;   // [C]
  uint8_t* slot_tier = nullptr;  // [C]
  int32_t* slot_last = nullptr;  // [C]
  int32_t* lru = nullptr;        // [2][C] ping-pong LRU order
  int32_t* lru_cur = nullptr;    // [1]
  int32_t* new_pos = nullptr;    // [cap] plan scratch: req position of the j-th NEW
  int32_t* work_pos = nullptr;   // [cap] plan scratch: work position of req p
  int32_t* vict_slot = nullptr;  // [cap] plan scratch
  int32_t* vict_old = nullptr;   // [cap] plan scratch
  int32_t* fill_pos = nullptr;   // [cap] plan scratch: fill position of req p (-1 for hits)
  uint8_t* prev_tier = nullptr;  // [cap] plan scratch: tier a REFILL's slot held before the step
  int32_t* slot_rec = nullptr;   // [C + S] record a slot's bytes hold, 4 * neuron + tier (-1: none), kept by the fill
  unsigned long long* stats = nullptr;  // [16] cumulative counters
  int32_t* status = nullptr;           // [1] M2C_STATUS_* bits set by kernels
  unsigned long long* ffn_gen = nullptr;  // [ffn_grid] per-workgroup call counters of the one-launch FFN
  unsigned long long* ffn_hw = nullptr;   // [cap] (call tag, h) words of the one-launch FFN
};

// Where the record in a slot starts: a slot of tier t's pool at global id s,
// first[t] <= s < first[t] + count[t], holds its record at byte
// base[t] + (s - first[t]) * stride[t] of the arena; `zero` is the all-zero
// padding slot (where every id outside the tier's pool points). Without tier
// pools every tier maps with base 0, first 0, count C + S, stride slot_bytes.
struct SlotMap {
  uint32_t base[4];
  int32_t first[4];
  int32_t count[4];
  uint32_t stride[4];
  uint32_t zero;
};

}  // namespace m2c

struct m2c_layer {
  m2c_layer_desc desc;
  int S = 0;    // staging slots
  int cap = 0;  // plan capacity
  int num_cus = 0;
  m2c::Store* store = nullptr;
  m2c_layer_info info;
  m2c_plan_layout layout;
  // device memory (one allocation, carved)
  uint8_t* dev_base = nullptr;
  int64_t dev_bytes = 0;
  uint16_t* pred_a = nullptr;  // [r][d]
  uint16_t* pred_b = nullptr;  // [d_ff][r]
  float* bias = nullptr;       // [d_ff] or null
  float* z = nullptr;          // [max_batch][r]
  float* scores = nullptr;     // [max_batch][d_ff]
  uint8_t* slots = nullptr;    // [C+S][slot_bytes]
  float2* ab = nullptr;        // [4 * cap] partial gate/up dot products per FFN unit
  float* y_part = nullptr;     // [ffn_groups][d] down-projection partial rows
  int ffn_groups = 1;
  int ffn_grid = 0;  // workgroups of the one-launch FFN
  m2c::DeviceState st;
  int64_t last_step = -1;
  int ffn_withhold = 0;  // test support: > 0 = h words withheld, polls before giving up
  m2c_dram* dram = nullptr;  // records come from this DRAM cache (store is null)
  int dram_index = -1;
  // per-tier record arena (M2C_FLAG_TIER_POOLS)
  bool pools = false;
  int pool_C[4] = {0, 0, 0, 0};   // resident slots per tier
  int pool_S[4] = {0, 0, 0, 0};   // staging slots per tier
  int pool_rf[4] = {0, 0, 0, 0};  // first resident table index of the pool
  m2c::SlotMap map;               // slot id -> byte offset, by tier
  int64_t arena_bytes = 0;        // pools + zero slot
  uint8_t* pool_plan = nullptr;   // [3][plan_core_bytes] the pools' own plans
  // per-tier arena: each pool's required neurons of a step, per chunk of
  // 1024 neurons in ascending id ([3][d_ff], FP16 first; chunk j from j * 1024),
  // and their counts ([3][32])
  int32_t* pool_lists = nullptr;
  int32_t* pool_counts = nullptr;
  int64_t plan_core_bytes = 0;    // a plan without the one-launch FFN's task table
  int32_t* plan_abort = nullptr;  // [1] set when a step's required set overflowed
};

namespace m2c {

// ---------------------------------------------------------------------------
// Host-side helpers of the entry points (m2c_api.hip)

// Sets the thread's error message (m2c_last_error) and returns `code`.
m2c_status api_fail(m2c_status code, const char* fmt, ...);
// The host-side argument checks of m2c_predict_rank.
m2c_status check_predict_args(const m2c_layer* L, const uint16_t* x, int batch, int k, int n_fp16,
                              int n_int8, const uint8_t* tier_map);

// SSD -> DRAM tier (dram_cache.hip)
m2c_status dram_acquire(m2c_dram* D, int layer, const uint8_t** data, int* slot);
void dram_release(m2c_dram* D, int slot, hipEvent_t reader);
hipEvent_t dram_event(m2c_dram* D);
int64_t dram_layer_bytes(const m2c_dram* D);
int dram_layers(const m2c_dram* D);
int dram_device(const m2c_dram* D);
bool dram_pinned(const m2c_dram* D);
void dram_ref(m2c_dram* D, int delta);

// ---------------------------------------------------------------------------
// Launchers (one per kernel file). All enqueue on `stream` and return the
// hipError_t of the launch.

hipError_t launch_transpose_u16(const uint16_t* in, uint16_t* out, int rows, int cols,
                                hipStream_t stream);
hipError_t launch_quantize_records(const uint16_t* wg, const uint16_t* wu, const uint16_t* wdT,
                                   int d, int i0, int n, uint8_t* r16, int64_t st16, uint8_t* r8,
                                   int64_t st8, uint8_t* r4, int64_t st4, hipStream_t stream);
hipError_t launch_predict(const m2c_layer* L, const uint16_t* x, int batch, float* z,
                          float* scores, hipStream_t stream);
hipError_t launch_select(const float* scores, int batch, int d_ff, int k, int n16, int n8,
                         uint8_t* tier_map, hipStream_t stream);
hipError_t launch_plan(m2c_layer* L, const uint8_t* tier_map, int batch, int step, uint8_t* plan,
                       hipStream_t stream);
hipError_t launch_reset(m2c_layer* L, hipStream_t stream);
hipError_t launch_fill(const m2c_layer* L, const uint8_t* plan, const uint8_t* const host[4],
                       hipStream_t stream);
hipError_t launch_poison_fill_slots(const m2c_layer* L, const uint8_t* plan, hipStream_t stream);
// The state and plan pointers of tier t's pool (M2C_FLAG_TIER_POOLS).
DeviceState pool_state(const m2c_layer* L, int t);
hipError_t launch_ffn(m2c_layer* L, const uint16_t* x, int batch, const uint8_t* plan, float* y,
                      hipStream_t stream);
hipError_t launch_ffn_batch(m2c_layer* L, const uint16_t* x, int batch, const uint8_t* plan,
                            float* y, hipStream_t stream);
hipError_t launch_ffn_split(m2c_layer* L, const uint16_t* x, const uint8_t* plan, float* y,
                            hipStream_t stream);
bool ffn_fused_supported(const m2c_layer* L);
int ffn_fused_grid(int d_model, int cap, int num_cus);  // workgroups (and gen counters) of the one-launch FFN
// The one-launch FFN's task table in a plan: whether the layer's plans carry
// one (batch-1 FFN calls use that kernel), its bytes for a grid, and the
// kernel that writes it from the plan's counts and work order.
bool ffn_tasks_used(const m2c_layer* L);
int ffn_loads_per_unit(int d);  // K of the one-launch FFN: 16-byte loads per lane and unit
int64_t ffn_task_table_bytes(int grid);
hipError_t launch_ffn_tasks(m2c_layer* L, uint8_t* plan, hipStream_t stream);
hipError_t launch_ffn_fused(m2c_layer* L, const uint16_t* x, const uint8_t* plan, float* y,
                            hipStream_t stream);

// ---------------------------------------------------------------------------
// Device helpers shared by the kernels

__device__ __forceinline__ float h2f(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

__device__ __forceinline__ uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Block-wide exclusive prefix sum over one value per thread (at most 1024
// threads). `tmp` holds at least blockDim.x / 64 entries of shared memory.
// Returns the exclusive prefix; *total gets the block sum. Each wave scans
// its lanes, then (after one barrier) the wave totals itself, lane q holding
// wave q's total, so no single thread walks the totals. Contains
// __syncthreads() (the second lets the caller reuse `tmp`).
template <typename T>
__device__ T block_exclusive_scan(T v, T* tmp, T* total) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = (blockDim.x + 63) >> 6;
  T incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    T o = __shfl_up(incl, off);
    if (lane >= off) incl += o;
  }
  if (lane == 63) tmp[wave] = incl;
  __syncthreads();
  T wt = lane < nwaves ? tmp[lane] : T(0);
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) {
    T o = __shfl_up(wt, off);
    if (lane >= off) wt += o;
  }
  const T before = wave > 0 ? __shfl(wt, wave - 1) : T(0);
  *total = __shfl(wt, nwaves - 1);
  __syncthreads();
  return before + incl - v;
}

}  // namespace m2c
