/*
 * m2c.h -- C ABI of the MI355X (gfx950) dynamic sparse mixed-precision FFN
 * with a neuron-level HBM slot cache (M2Cache, arXiv 2410.14740).
 *
 * One decode step of one FFN layer is four calls, in this order:
 *
 *   m2c_predict_rank  score every FFN neuron with the layer's low-rank
 *                     predictor, take the top-k, split them into FP16 / INT8 /
 *                     INT4 tiers by score rank            (Sec. 1 "Active Neuron
 *                     Identification" and "Active Score-based Quantization";
 *                     Sec. 5.2, Fig. 3)
 *   m2c_cache_plan    resolve the active neurons against the layer's HBM slot
 *                     cache: hit / refill / new / bypass, LRU victims, slot
 *                     table update                        (Sec. 5.3 "Overall
 *                     architecture" and "Cache Policy"; Sec. 1 LRU cache)
 *   m2c_cache_fill    copy every missing neuron record, at its tier, from the
 *                     pinned host-DRAM neuron store into its slot (Sec. 1
 *                     "Selective Loading into GPU"; Sec. 6.1 dedicated streams)
 *   m2c_sparse_ffn    gated FFN over only the active neurons, each read from
 *                     its slot and dequantized at its tier (Sec. 1, Sec. 5.2)
 *
 * Conventions shared by every call
 * --------------------------------
 * - All functions return an m2c_status. On an error detected on the host
 *   nothing is enqueued, the layer is unchanged and m2c_last_error() returns
 *   a message (thread-local). Nothing throws across the ABI.
 * - "dev" pointers are device memory of the layer's device; "host" pointers
 *   are ordinary host memory. The caller owns every pointer it passes.
 * - Streams are hipStream_t values passed as void*; NULL is the null stream.
 *   Asynchronous calls only enqueue work on the given stream and return.
 *   Ordering between streams (for example the fill stream and the FFN
 *   stream) is the caller's job, with events.
 * - fp16 values are passed as their IEEE binary16 bit patterns (uint16_t).
 *
 * Neuron and tiers (Sec. 1 footnote, Sec. 5.2)
 * --------------------------------------------
 * Neuron i of a SwiGLU FFN with W_gate, W_up [d_ff][d_model] and
 * W_down [d_model][d_ff] is row i of W_gate, row i of W_up and column i of
 * W_down. Tier codes: 0 inactive, 1 INT4, 2 INT8, 3 FP16 (higher score ->
 * higher precision, Sec. 5.2).
 *
 * Neuron records (the unit that is stored, copied and cached)
 * ----------------------------------------------------------
 * d = d_model, G = d / 128 (quantization group of 128 consecutive elements).
 *   FP16 record (tier 3), 6d bytes:
 *     gate[d] fp16 | up[d] fp16 | down[d] fp16
 *   INT8 record (tier 2), 3d + 6G bytes:
 *     gate[d] int8 | up[d] int8 | down[d] int8 |
 *     gate_scale[G] fp16 | up_scale[G] fp16 | down_scale[G] fp16
 *   INT4 record (tier 1), 1.5d + 6G bytes:
 *     gate[d/2] | up[d/2] | down[d/2] | gate_scale[G] | up_scale[G] | down_scale[G]
 *     byte m of a vector holds element 2m in bits 0-3 and element 2m+1 in
 *     bits 4-7, each a two's-complement nibble.
 * Quantization (symmetric, per group g of one vector, qmax = 127 or 7):
 *     amax = max |w| over the group (w are the fp16 weights),
 *     s    = fp16_rne( fp32(amax) / qmax )        (IEEE fp32 division),
 *     q    = clamp( rne( fp32(w) / fp32(s) ), -qmax, qmax ), q = 0 if s == 0,
 *     dequantized weight = q * s (exact in fp32).
 * Records of tier t are stored back to back with a stride of
 * record_stride[t] = record_bytes[t] rounded up to 16 bytes.
 *
 * Predictor scores (Sec. 5.2; low-rank predictor of Sec. 1)
 * ---------------------------------------------------------
 *   z = A x  (A [r][d] fp16),   s = B z + bias  (B [d_ff][r] fp16, bias fp32).
 * Every dot product is evaluated in fp32 in one fixed order, so that scores
 * (and therefore the selected ids) are reproducible bit for bit:
 *   n-element dot product, n % 8 == 0: split into chunks of 8 consecutive
 *   elements; L = min(64, largest power of two <= n/8) partial sums; chunk c
 *   belongs to partial c % L; each partial starts at +0.0f and takes
 *   acc = fmaf(a_j, b_j, acc) over its chunks in ascending order, elements in
 *   ascending order inside a chunk; then for off = L/2, L/4, ..., 1 every
 *   partial p becomes p[l] + p[l ^ off]; the result is p[0]. z stays fp32;
 *   the bias, when present, is one fp32 addition after the dot product.
 *
 * Selection and tiers (Sec. 5.2)
 * ------------------------------
 * Neurons are ranked by score descending, ties by id ascending; scores are
 * compared as order-preserving unsigned keys of their fp32 bit patterns
 * (so -0.0 ranks below +0.0). Rank rho < n_fp16 -> tier 3;
 * rho < n_fp16 + n_int8 -> tier 2; rho < k -> tier 1; else tier 0.
 *
 * Cache policy (Sec. 5.3; LRU of Sec. 1 and Sec. 6.4)
 * ---------------------------------------------------
 * One cache unit per layer: C resident slots plus S staging slots, each
 * slot_bytes = 6d bytes (an FP16 record). The required set R of a step is
 * every neuron with tier > 0 in some batch row, taken at the highest tier any
 * row asks for. The step is atomic: for i in R (ascending id)
 *   HIT     i is resident at the requested tier (with M2C_FLAG_DOMINANT_HITS:
 *           at the requested tier or above; the step then uses the resident
 *           tier);
 *   REFILL  i is resident at another tier (with M2C_FLAG_DOMINANT_HITS: a
 *           lower one): it is refilled in its own slot;
 *   NEW     i is not resident.
 * Victims are the slots holding no neuron of R, ordered by (last use
 * ascending, slot ascending); never-used slots count as last use -1. The j-th
 * NEW neuron in ascending id takes the j-th victim and evicts its previous
 * neuron. NEW neurons beyond the number of victims are BYPASS: they are
 * filled into staging slot C + j' (j' counts bypasses in ascending id) and
 * are not retained. Every slot of R gets last use = step. With C = k and a
 * single tier this reduces to the paper's Adjacent Token Update policy.
 */
#ifndef M2C_H
#define M2C_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  M2C_OK = 0,
  M2C_ERR_INVALID_ARG = 1,  /* bad pointer, size, count or descriptor        */
  M2C_ERR_OUT_OF_MEMORY = 2,/* device or pinned host allocation failed       */
  M2C_ERR_HIP = 3,          /* a HIP runtime call failed (message has detail)*/
  M2C_ERR_CAPACITY = 4,     /* a size beyond what the layer was created for  */
  M2C_ERR_STATE = 5         /* call out of order (e.g. step not increasing)  */
} m2c_status;

typedef struct m2c_layer m2c_layer; /* opaque; one per FFN layer */

enum { M2C_TIER_NONE = 0, M2C_TIER_INT4 = 1, M2C_TIER_INT8 = 2, M2C_TIER_FP16 = 3 };

/* Layer descriptor. All fields are required. */
typedef struct {
  int32_t d_model;       /* d: multiple of 128, 128..16384                      */
  int32_t d_ff;          /* neurons: 1..262144                                  */
  int32_t pred_rank;     /* r: multiple of 8, 8..1024                           */
  int32_t group;         /* quantization group; must be 128                     */
  int32_t k_max;         /* largest k any call will use: 0..d_ff                */
  int32_t max_batch;     /* largest batch any call will use: 1..32              */
  int32_t cache_slots;   /* C: resident slots, 0..d_ff                          */
  int32_t staging_slots; /* S: bypass slots; -1 = the minimum that can never
                            overflow, max(0, min(d_ff, max_batch*k_max) - C);
                            smaller explicit values are rejected               */
  int32_t device;        /* HIP device ordinal                                  */
  int32_t flags;         /* M2C_FLAG_* bits, 0 for the defaults                 */
  int32_t tier_slots[4]; /* with M2C_FLAG_TIER_POOLS: resident slots of the INT4
                            [1], INT8 [2] and FP16 [3] pools, summing to
                            cache_slots ([0] unused); otherwise ignored        */
} m2c_layer_desc;

/* m2c_layer_desc.flags */
enum {
  /* Sparse FFN by three kernels (up, down by column slices, ordered reduce)
     whose output is the same bit pattern on every run. The default is two
     kernels (h of every neuron, then the down projection by column slice and
     neuron group) whose neuron groups are added into y with fp32 atomics,
     so the summation order, and the last bits of y, vary from run to run. */
  M2C_FLAG_DETERMINISTIC_FFN = 1,
  /* Cache policy variant (Sec. 5.3 "Cache Policy"): a neuron resident at a
     tier at or above the requested one is a HIT and the step uses it at its
     resident tier (req_tier and the FFN then carry the resident tier); only
     a resident tier below the requested one is a REFILL. The default is the
     exact-tier policy: any other resident tier is a REFILL. With dominance
     hits the output depends on the cache history, not only on the step. */
  M2C_FLAG_DOMINANT_HITS = 2,
  /* Per-tier record arena: the cache unit is split into one pool per tier,
     pool t with tier_slots[t] resident slots of record_stride[t] bytes (an
     INT4 neuron no longer takes an FP16-sized slot, so the same HBM holds
     more neurons). Each pool is its own step-atomic LRU cache over the
     neurons whose step tier is t: HIT if resident in that pool, else NEW
     there (victims from that pool, BYPASS into that pool's staging slots,
     max(0, plan_capacity - tier_slots[t]) of them). A neuron may be resident
     in several pools; there are no REFILLs. Global slot ids are numbered in
     tier blocks, FP16 first (see m2c_layer_info.pool_first). With
     M2C_FLAG_DOMINANT_HITS a neuron required at tier t that is not resident
     in pool t but is resident (at the start of the step) in a pool of higher
     precision is served by the lowest such pool, a HIT at that pool's tier
     (req_tier and the FFN carry it). Needs max_batch == 1, d_model <= 8192,
     d_ff <= 32768, staging_slots == -1, and not M2C_FLAG_DETERMINISTIC_FFN. */
  M2C_FLAG_TIER_POOLS = 4
};

/* Sizes that follow from a descriptor. */
typedef struct {
  int32_t record_bytes[4];  /* by tier; [0] = 0                               */
  int32_t record_stride[4]; /* host store stride by tier; [0] = 0             */
  int32_t slot_bytes;       /* 6 * d_model                                    */
  int32_t cache_slots;      /* C                                              */
  int32_t staging_slots;    /* S (resolved)                                   */
  int32_t plan_capacity;    /* entries of every plan list: min(d_ff, max_batch*k_max) */
  int64_t plan_bytes;       /* size of one plan buffer                        */
  int64_t host_store_bytes; /* pinned host neuron store (all three tiers)     */
  int64_t device_bytes;     /* device memory the layer owns                   */
  /* Slots of the tier-t records, by tier [1..3]: global slot ids
     [pool_first[t], pool_first[t] + pool_slots[t]), resident ones first,
     each pool_stride[t] bytes. Without M2C_FLAG_TIER_POOLS every tier shares
     one pool: pool_first 0, pool_slots C + S, pool_stride slot_bytes. */
  int32_t pool_first[4];
  int32_t pool_slots[4];
  int32_t pool_resident[4]; /* resident slots of the pool (the rest stage)    */
  int32_t pool_stride[4];
  int64_t slot_arena_bytes; /* every pool plus the all-zero padding slot      */
} m2c_layer_info;

/* A plan is one caller-allocated device buffer of info.plan_bytes bytes,
 * 256-byte aligned. These are the byte offsets of its arrays; every list has
 * plan_capacity entries of which counts[...] are valid. */
enum {
  M2C_CNT_REQ = 0,     /* |R|                                                 */
  M2C_CNT_HIT = 1,
  M2C_CNT_REFILL = 2,
  M2C_CNT_NEW = 3,     /* NEW that got a resident victim slot                 */
  M2C_CNT_BYPASS = 4,  /* NEW that went to a staging slot                     */
  M2C_CNT_EVICT = 5,   /* victims that held a neuron                          */
  M2C_CNT_FILL = 6,    /* REFILL + NEW + BYPASS                               */
  M2C_CNT_REQ_FP16 = 7,/* |R| by tier                                         */
  M2C_CNT_REQ_INT8 = 8,
  M2C_CNT_REQ_INT4 = 9,
  M2C_CNT_FILL_FP16 = 10, /* fills by tier                                    */
  M2C_CNT_FILL_INT8 = 11,
  M2C_CNT_FILL_INT4 = 12,
  M2C_CNT_FILL_DERIVED = 13, /* INT8 / INT4 fills of a neuron whose slot held its
                             FP16 record: made on the GPU from that record,
                             no host read (fill_from == 3)                     */
  M2C_NCOUNTS = 16
};
typedef struct {
  int64_t counts;      /* int32 [M2C_NCOUNTS]                                 */
  int64_t req_ids;     /* int32 [cap] R in ascending neuron id                */
  int64_t req_tier;    /* uint8 [cap] tier taken for the step (max over rows) */
  int64_t req_hit;     /* uint8 [cap] 0 NEW, 1 HIT, 2 REFILL, 3 BYPASS        */
  int64_t req_slot;    /* int32 [cap] slot read by the FFN                    */
  int64_t req_mask;    /* uint32[cap] bit b set if batch row b selected it    */
  int64_t fill_ids;    /* int32 [cap] misses in ascending neuron id           */
  int64_t fill_tier;   /* uint8 [cap]                                         */
  int64_t fill_slot;   /* int32 [cap]                                         */
  int64_t fill_from;   /* uint8 [cap] REFILL: tier of the record the slot held
                          for the neuron before the step; NEW / BYPASS: 0     */
  int64_t evicted_ids; /* int32 [cap] evicted neurons in victim order         */
  int64_t work_slot;   /* int32 [cap] R regrouped tier-major (FP16, INT8,
                          INT4), ascending id inside a tier: FFN work order;
                          512 spare entries follow (read, never used)         */
  int64_t work_mask;   /* uint32[cap] row masks in work order                 */
  int64_t ffn_tasks;   /* the batch-1 FFN kernel's per-workgroup task table:
                          library-internal format, written by m2c_cache_plan
                          (empty for layers whose FFN does not use it)       */
  int64_t total_bytes;
} m2c_plan_layout;

/* Cumulative per-layer counters since creation or the last cache reset. */
typedef struct {
  int64_t plans;
  int64_t req, hit, refill, new_, bypass, evict;
  int64_t fill[4];        /* fills by tier                                    */
  int64_t fill_bytes;     /* sum of record_bytes over fills                   */
  int64_t derived[4];     /* fills by tier made from the resident FP16 record */
  int64_t host_bytes;     /* sum of record_bytes over fills read from the host
                             store: fill_bytes minus the derived fills'       */
  int64_t req_tier[4];    /* required neurons by step tier                    */
  int64_t req_bytes;      /* sum of record_bytes over required neurons: what
                             the sparse FFN reads from the slots              */
} m2c_stats;

/* Bytes of one neuron record of `tier` (1..3) for d_model d, or -1. */
int64_t m2c_record_bytes(int32_t d_model, int32_t tier);

/* Create a layer (Sec. 5.3 isolated cache unit + the layer's share of the
 * host-DRAM neuron store). Host inputs, copied; may be freed on return:
 *   w_gate, w_up  [d_ff][d_model] fp16; w_down [d_model][d_ff] fp16;
 *   pred_a [pred_rank][d_model] fp16;  pred_b [d_ff][pred_rank] fp16;
 *   score_bias [d_ff] fp32 or NULL (no addition).
 * Quantizes every neuron to the INT8 and INT4 records on the device and keeps
 * all three records in pinned host memory; the cache starts cold.
 * Synchronous. */
m2c_status m2c_layer_create(const m2c_layer_desc* desc, const uint16_t* w_gate,
                            const uint16_t* w_up, const uint16_t* w_down,
                            const uint16_t* pred_a, const uint16_t* pred_b,
                            const float* score_bias, m2c_layer** out);

/* Create a layer that reads its neuron records from the host store of
 * `weights_of` (same d_model, d_ff and device) instead of owning a copy; it
 * has its own predictor, slot cache and tables. The store lives until every
 * layer using it is destroyed. Synchronous. */
m2c_status m2c_layer_create_shared(const m2c_layer_desc* desc, const m2c_layer* weights_of,
                                   const uint16_t* pred_a, const uint16_t* pred_b,
                                   const float* score_bias, m2c_layer** out);

/* Wait for the device, then free everything the layer owns. NULL is a no-op. */
m2c_status m2c_layer_destroy(m2c_layer* layer);

m2c_status m2c_layer_get_info(const m2c_layer* layer, m2c_layer_info* out);
m2c_status m2c_plan_get_layout(const m2c_layer* layer, m2c_plan_layout* out);

/* Scores and tiers for `batch` tokens.
 *   x        dev fp16 [batch][d_model]
 *   scores   dev fp32 [batch][d_ff] output, or NULL (kept internally)
 *   tier_map dev uint8 [batch][d_ff] output, tier of every neuron
 * 0 <= n_fp16, 0 <= n_int8, n_fp16 + n_int8 <= k <= k_max, 1 <= batch <= max_batch. */
m2c_status m2c_predict_rank(m2c_layer* layer, const uint16_t* x, int32_t batch, int32_t k,
                            int32_t n_fp16, int32_t n_int8, float* scores, uint8_t* tier_map,
                            void* stream);

/* Bytes of the fixed device scratch array of m2c_predict_rank_noalloc. */
#define M2C_NOALLOC_SCRATCH_BYTES (4u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * scores and tier map as m2c_predict_rank, bit for bit, with the call's
 * scratch -- z [batch][pred_rank] fp32 and, when `scores` is NULL, the scores
 * [batch][d_ff] fp32 -- in one fixed device array of M2C_NOALLOC_SCRATCH_BYTES
 * that the library keeps on every GPU it runs on until the process ends,
 * instead of the layer's own buffers. Allocates nothing: no hipMalloc, no
 * hipFree, no allocating library call.
 * Limit: round_up(4 * batch * pred_rank, 256) + (scores ? 0 : 4 * batch *
 * d_ff) <= M2C_NOALLOC_SCRATCH_BYTES, else M2C_ERR_CAPACITY with nothing
 * enqueued. Every call on one GPU, from any layer, shares that GPU's array:
 * calls that can run at the same time on one GPU (streams not ordered with
 * each other, or other threads) race and give wrong results; calls ordered
 * on one stream are safe. The array is fully written before it is read, so
 * what an earlier call left in it never matters. */
m2c_status m2c_predict_rank_noalloc(m2c_layer* layer, const uint16_t* x, int32_t batch, int32_t k,
                                    int32_t n_fp16, int32_t n_int8, float* scores,
                                    uint8_t* tier_map, void* stream);

/* Resolve tier_map (dev uint8 [batch][d_ff]) against the slot cache for
 * decode step `step`, write the plan into `plan` (dev, plan_bytes) and update
 * the slot tables. `step` must be >= 0, < 2^31 and strictly greater than the
 * previous step given to this layer (M2C_ERR_STATE otherwise). The plan must
 * not be reused until every fill and FFN that reads it has completed. */
m2c_status m2c_cache_plan(m2c_layer* layer, const uint8_t* tier_map, int32_t batch, int64_t step,
                          void* plan, void* stream);

/* Copy every fill of `plan` from the pinned host store into its slot, on
 * `stream`, by a device gather kernel that reads host memory over the host
 * link. A fill to INT8 / INT4 whose slot holds the neuron's FP16 record
 * (fill_from == 3) is instead quantized in place from that record, which
 * gives the bytes of the store's record (both are the group-128 quantization
 * of the same fp16 values); the layer tracks which slots hold FP16 bytes, so
 * running the fill of a plan again copies instead and gives the same slots.
 * Must run after the plan on the same stream or behind an event, and before
 * the FFN that reads the plan. No host synchronization. */
m2c_status m2c_cache_fill(m2c_layer* layer, const void* plan, void* stream);

/* y += sum over i in R of silu(<g_i, x>) * <u_i, x> * d_i, per batch row b
 * over the neurons whose req_mask has bit b, every vector dequantized at the
 * neuron's step tier; fp32 accumulation. The result is ADDED to y (a residual
 * stream); zero y first for the plain FFN output.
 *   x dev fp16 [batch][d_model];  y dev fp32 [batch][d_model], in/out.
 * `batch` (1..max_batch) must equal the batch given to the plan. Batch 1 is a
 * gather-dequant GEMV; larger batches run both contractions on the matrix
 * cores with fp32 accumulation: gate / up with the codes (exact as fp16) and
 * x, group scales applied in fp32; down with the codes and h times the group
 * scale, the latter split into an fp16 high and low part. They are never
 * bit-deterministic (the deterministic flag applies to batch 1). */
m2c_status m2c_sparse_ffn(m2c_layer* layer, const uint16_t* x, int32_t batch, const void* plan,
                          float* y, void* stream);

/* Make the cache cold again (all slots empty, stats zeroed, step history
 * cleared), on `stream`. */
m2c_status m2c_layer_reset_cache(m2c_layer* layer, void* stream);

/* Synchronizes the device, then reads the cumulative counters. Returns
 * M2C_ERR_CAPACITY (and clears the condition) if a cache plan since the last
 * call received a tier map with more active neurons than the layer's plan
 * capacity, min(d_ff, max_batch * k_max): such a plan is left empty and the
 * cache unchanged. Returns M2C_ERR_STATE (and clears the condition) if a
 * batch-1 sparse FFN gave up waiting for one of its own h values (its
 * workgroups could not all run, for instance because another kernel held the
 * GPU for a long time); that call's output is wrong. */
m2c_status m2c_layer_stats(const m2c_layer* layer, m2c_stats* out);

/* ------------------------------------------------------------------------
 * SSD -> DRAM tier (Sec. 5.4 "Pattern-Aware Preloading for SSD", Fig. 8)
 * ------------------------------------------------------------------------
 * Every layer's neuron records live in a file (the SSD). A two-level DRAM
 * cache holds the first `fixed_layers` layers in a fixed area, read once at
 * creation and never evicted (a new token does not reload them), and the
 * other layers in a dynamic area of `dynamic_slots` layer-sized buffers. A
 * loader thread reads whole layers ahead of use. When layer l is acquired,
 * the window l, l+1, ..., l+lookahead (mod n_layers) is made resident in
 * that order (the caller waits only for l); a missing layer takes the lowest
 * empty slot, else the slot of the loaded, unheld layer outside the window
 * whose next use in the cyclic layer order is furthest away (largest
 * (layer - l) mod n_layers); a look-ahead load with no slot to give up is
 * skipped. These decisions depend only on the order of acquires.
 *
 * File layout of one layer (what m2c_layer_write_store writes): the FP16,
 * INT8 and INT4 record arrays back to back (d_ff * record_stride[t] bytes
 * each), zero-padded to a multiple of 4096 bytes; layer_bytes is the
 * unpadded size. Layer offsets in the file are multiples of 4096. */
enum {
  M2C_DRAM_HOST_MEMORY = 1, /* plain host memory (no HIP calls; CPU-side use
                               and tests); default: pinned (hipHostMalloc) so
                               that the GPU fill reads it over the host link */
  M2C_DRAM_DIRECT_IO = 2    /* read with O_DIRECT (bypass the page cache);
                               falls back to buffered reads if the file system
                               refuses it (m2c_dram_stats.direct_io says) */
};
typedef struct {
  int32_t n_layers;      /* layers in the file                                 */
  int32_t fixed_layers;  /* fixed area: layers 0 .. fixed_layers-1             */
  int32_t dynamic_slots; /* dynamic area: >= lookahead + 1 unless every layer
                            is fixed                                          */
  int32_t lookahead;     /* layers loaded ahead of the one in use, >= 1        */
  int64_t layer_bytes;   /* bytes of one layer's records (unpadded)            */
  int32_t flags;         /* M2C_DRAM_*                                         */
  int32_t device;        /* device whose fills read the pinned buffers         */
} m2c_dram_desc;
typedef struct {
  int64_t acquires, hits;  /* hits: the layer was already in DRAM             */
  int64_t loads, evictions;
  int64_t bytes_read;      /* layer_bytes per load from the file              */
  int64_t fixed_bytes;     /* bytes of the fixed area                         */
  double read_seconds;     /* time the loader spent reading                   */
  double wait_seconds;     /* time acquires spent waiting for their layer     */
  int32_t direct_io;       /* 1 if reads bypass the page cache                */
} m2c_dram_stats;
typedef struct m2c_dram m2c_dram; /* opaque */

/* Write the layer's host store into `path` (created if missing) at `offset`
 * (a multiple of 4096), in the file layout above; *padded_bytes gets the
 * bytes written (layer_bytes rounded up to 4096). Synchronous. */
m2c_status m2c_layer_write_store(const m2c_layer* layer, const char* path, int64_t offset,
                                 int64_t* padded_bytes);

/* Open the cache over `path`; offsets[l] is layer l's offset. Reads the fixed
 * area before returning and starts the loader thread. */
m2c_status m2c_dram_create(const m2c_dram_desc* desc, const char* path, const int64_t* offsets,
                           m2c_dram** out);
/* Stops the loader, waits for the GPU readers of the buffers, frees them.
 * M2C_ERR_STATE while layers created on the cache still exist. */
m2c_status m2c_dram_destroy(m2c_dram* dram);
/* Host-side use: wait until `layer` is in DRAM, hold it, return its bytes. */
m2c_status m2c_dram_acquire(m2c_dram* dram, int32_t layer, const uint8_t** data);
/* Give up a hold taken by m2c_dram_acquire. */
m2c_status m2c_dram_release(m2c_dram* dram, int32_t layer);
m2c_status m2c_dram_get_stats(m2c_dram* dram, m2c_dram_stats* out);
/* Test support: the loads decided so far, in order (layer loaded, layer
 * evicted or -1); *count gets the total, at most `capacity` are copied. */
m2c_status m2c_dram_get_log(m2c_dram* dram, int32_t* loaded, int32_t* evicted, int32_t capacity,
                            int32_t* count);

/* Create a layer whose neuron records are layer `index` of a pinned DRAM
 * cache (same d_model / d_ff and device; dram layer_bytes must equal the
 * layer's record arrays). Its own predictor, slot cache and tables; each
 * m2c_cache_fill acquires the layer from the cache (waiting for the loader
 * if needed), enqueues the gather from those buffers and releases them
 * behind a HIP event, so the loader never overwrites bytes a fill still
 * reads. Fills of layers of one cache should be issued in layer order (the
 * cyclic order the look-ahead assumes). The cache must outlive the layer. */
m2c_status m2c_layer_create_from_dram(const m2c_layer_desc* desc, m2c_dram* dram, int32_t index,
                                      const uint16_t* pred_a, const uint16_t* pred_b,
                                      const float* score_bias, m2c_layer** out);

/* Offline neuron-ratio search (Sec. 5.2 "Offline Neuron Ratio Search",
 * Algorithm 1) on an FFN-error proxy of the paper's entropy estimate, which
 * needs a trained language model. Candidate i = 1, 2, ... has
 * n_high = i * step FP16 neurons and n_low = n_low0 - i * step * bit_ratio
 * low-precision ones (INT4 for bit_ratio 4, INT8 for bit_ratio 2), while
 * n_low >= 0: the bytes of the active neurons stay the same. Its score is
 *   uq = sum_t |y_t - y*_t|^2 / sum_t |y*_t|^2
 * over the T calibration tokens x (dev fp16 [T][d_model]): y_t is this
 * layer's sparse FFN with the top n_high + n_low neurons by predictor score,
 * the n_high best at FP16, the rest at the low tier; y*_t the FFN with every
 * neuron at FP16. Each FFN runs through the layer's predict, plan, fill and
 * FFN kernels on `stream`. The chosen candidate is the one with the lowest
 * score, a later one winning ties (the comparison UQ_best >= UQ_score).
 * Needs k_max == d_ff (the all-FP16 reference). Outputs (host, room for
 * max_candidates): n_high, n_low, uq per candidate, *count candidates,
 * *best the chosen index (-1 if none). Synchronous; allocates its buffers;
 * leaves the layer's cache cold (reset). */
m2c_status m2c_ratio_search(m2c_layer* layer, const uint16_t* x, int32_t T, int32_t n_low0,
                            int32_t step, int32_t bit_ratio, int32_t max_candidates,
                            int32_t* n_high, int32_t* n_low, double* uq, int32_t* count,
                            int32_t* best, void* stream);

/* Test support. Copies one record of the host store (no device work). */
m2c_status m2c_debug_read_record(const m2c_layer* layer, int32_t tier, int32_t neuron, void* out,
                                 size_t bytes);
/* Test support. Synchronizes the device, then copies slot `slot` (0..C+S-1;
 * at most its pool's stride with M2C_FLAG_TIER_POOLS). */
m2c_status m2c_debug_read_slot(const m2c_layer* layer, int32_t slot, void* out, size_t bytes);
/* Test support. Synchronizes the device, then copies the tables of tier
 * `tier`'s pool (M2C_FLAG_TIER_POOLS): slot_of int32 [d_ff] (pool-local
 * resident slot or -1), slot_key int32 [tier_slots[tier]], slot_last int32
 * [tier_slots[tier]]; any pointer may be NULL. */
m2c_status m2c_debug_read_pool_tables(const m2c_layer* layer, int32_t tier, int32_t* slot_of,
                                      int32_t* slot_key, int32_t* slot_last);

/* Test support. Synchronizes the device, then copies the slot tables; any
 * pointer may be NULL. slot_of int32 [d_ff] (-1 = not resident);
 * slot_key int32 [C] (-1 = empty); slot_tier uint8 [C]; slot_last int32 [C]. */
m2c_status m2c_debug_read_tables(const m2c_layer* layer, int32_t* slot_of, int32_t* slot_key,
                                 uint8_t* slot_tier, int32_t* slot_last);

/* Test support. Enqueues on `stream` a kernel that overwrites with 0xFF
 * bytes every slot the fill of `plan` writes (slot_bytes each), except the
 * slots whose INT8 / INT4 record the fill may make from the FP16 bytes
 * already there (fill_from == 3). Enqueued right before m2c_cache_fill on the
 * same stream, it makes ordering mistakes visible: an FFN that reads a slot
 * before its fill completes reads 0xFF bytes (NaN as fp16, code -1 as
 * INT8 / INT4 with a NaN scale), and a fill that starts while an earlier FFN
 * still reads the slot corrupts that FFN's output. */
m2c_status m2c_debug_poison_fill_slots(m2c_layer* layer, const void* plan, void* stream);

/* Test support. polls > 0: the layer's one-launch batch-1 sparse FFN (d_model
 * <= 8192, not deterministic) stops publishing its h values and its down
 * tasks give up after `polls` polls, so that every later call takes the
 * bounded-wait give-up path (h = 0, status word set, M2C_ERR_STATE from the
 * next m2c_layer_stats) while every kernel still exits normally. polls == 0
 * restores the normal behaviour. Host-side setting; affects launches made
 * after the call. */
m2c_status m2c_debug_ffn_withhold_h(m2c_layer* layer, int32_t polls);

/* Message of the last error on this thread ("" if none). */
const char* m2c_last_error(void);

/* Identifier of the sources the library was built from (16 hex digits of a
 * SHA-256 over the kernel sources and this header), so that a loader can
 * refuse a library built from other sources. Static string, never NULL. */
const char* m2c_build_id(void);

#ifdef __cplusplus
}
#endif
#endif /* M2C_H */
