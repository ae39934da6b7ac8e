// Sparse mixed-precision SwiGLU FFN for a batch of 2..32 tokens. The plan's
// required set is the union of the batch rows' active sets, each neuron at
// the highest tier any row asked for, with a row mask (the paper keeps batch
// 1, Sec. 5.5; this follows the union reading in include/m2c.h). Row b sums
// only the neurons whose mask has bit b:
//
//   y_b += sum_{i : mask_i bit b} silu(<g_i, x_b>) * <u_i, x_b> * d_i
//
// With several tokens the gate / up side is a real dense contraction, a
// gathered (2|R| x d) by (d x B) product, so it runs on the matrix cores:
//
//   ffn_bh_kernel   a workgroup takes a tile of 16 neurons of one tier (8 for
//                   FP16, padded with the zero slot); its 8
//                   waves split d by quantization group (group g to wave
//                   g % 8). For each group a wave issues four
//                   v_mfma_f32_16x16x32_f16 steps per row kind over the 128
//                   elements: A = the 16 neurons' codes (INT8 / INT4 unpacked
//                   to exact fp16), B = x of 16 batch rows (rows past the
//                   batch are zeros), read from the wave's LDS copy of the
//                   group's x rows. Which columns a lane takes in a step is
//                   chosen per tier so that every 16-byte record load of a
//                   wave covers 64 contiguous bytes of each row; both
//                   operands follow the same order. Each group's product is
//                   scaled by its fp16 scales in fp32 and added up, so the
//                   dequantization stays exact. The waves' partials meet in
//                   LDS; h_{b,i} = silu(a) * u, zero where row b did not
//                   select neuron i.
//   ffn_bdm_kernel  the down projection, also on the matrix cores, by
//                   quantization group and single-tier run (below).
#include "ffn_device.h"

namespace m2c {

typedef _Float16 half4v __attribute__((ext_vector_type(4)));
typedef float float4v __attribute__((ext_vector_type(4)));

constexpr int kBHThreads = 512;
constexpr int kBHWaves = kBHThreads / 64;

__device__ __forceinline__ half4v h4(uint32_t lo, uint32_t hi) {
  half4v r;
  const half2v a = as_h2(lo), b = as_h2(hi);
  r[0] = a[0];
  r[1] = a[1];
  r[2] = b[0];
  r[3] = b[1];
  return r;
}

// Four INT4 codes (16 bits, element e in bits 4e..4e+3) -> exact fp16 values.
__device__ __forceinline__ half4v i4x4_to_h4(uint32_t w16) {
  const uint32_t ob = w16 ^ 0x8888u;  // q + 8 per nibble
  const uint32_t lo = (ob & 0xfu) | ((ob & 0xf0u) << 12) | 0x64006400u;
  const uint32_t hi = ((ob >> 8) & 0xfu) | ((ob & 0xf000u) << 4) | 0x64006400u;
  const half2v bias = {(_Float16)1032.0f, (_Float16)1032.0f};
  const half2v a = as_h2(lo) - bias, b = as_h2(hi) - bias;
  half4v r;
  r[0] = a[0];
  r[1] = a[1];
  r[2] = b[0];
  r[3] = b[1];
  return r;
}

// Four INT8 codes (one word) -> exact fp16 values.
__device__ __forceinline__ half4v i8x4_to_h4(uint32_t w) {
  half2v a, b;
  i8x4_to_h2(w, a, b);
  half4v r;
  r[0] = a[0];
  r[1] = a[1];
  r[2] = b[0];
  r[3] = b[1];
  return r;
}

// Tile b: up to 16 consecutive work items of one tier. An FP16 tile takes 8
// items (the MFMA rows past them read the zero slot), so that it carries about
// as many record bytes as an INT8 tile of 16 and the workgroups finish
// together instead of the FP16 tiles trailing.
__device__ __forceinline__ void bh_tile(int b, int n3, int n2, int n1, int& tier, int& item0,
                                        int& nitems) {
  const int t3 = (n3 + 7) >> 3, t2 = (n2 + 15) >> 4, t1 = (n1 + 15) >> 4;
  if (b < t3) {
    tier = 3;
    item0 = 8 * b;
    nitems = min(8, n3 - item0);
  } else if (b < t3 + t2) {
    tier = 2;
    item0 = 16 * (b - t3);
    nitems = min(16, n2 - item0);
    item0 += n3;
  } else if (b < t3 + t2 + t1) {
    tier = 1;
    item0 = 16 * (b - t3 - t2);
    nitems = min(16, n1 - item0);
    item0 += n3 + n2;
  } else {
    tier = 0;
    item0 = nitems = 0;
  }
}

// One group (128 columns) of a tile on the matrix cores, as four
// v_mfma_f32_16x16x32_f16 steps per row kind (gate, up). Lane (row r, lane
// group j) supplies 8 codes of neuron row r per step; which 8 of the group's
// 128 columns a (j, step) pair takes is chosen per tier so that every 16-byte
// record load of a wave covers 64 contiguous bytes of each of its rows:
//
//   FP16  load e = step e:            columns 32 s + 8 j .. + 8
//   INT8  load e = steps 2e, 2e + 1:  columns 64 (s >> 1) + 16 j + 8 (s & 1) .. + 8
//   INT4  one load, word s = step s:  columns 32 j + 8 s .. + 8
//
// The B operand (x of the lane's batch column, same 8 columns) is read from
// the wave's copy of the group's x rows in LDS, so both operands pair the
// same columns whatever the mapping.
typedef _Float16 half8v __attribute__((ext_vector_type(8)));
constexpr int kBXRow = 136;  // halves per staged x row: 128 and a pad against bank conflicts
// halves per row of the staged gate and up scales (2 G, padded to 16 bytes)
__host__ __device__ constexpr int bh_scale_row(int G) { return 8 * ((G + 3) / 4); }

__device__ __forceinline__ half8v h8(half4v lo, half4v hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

template <int TIER>
__host__ __device__ constexpr int bh_xcol(int j, int s) {
  return TIER == 3 ? 32 * s + 8 * j : TIER == 2 ? 64 * (s >> 1) + 16 * j + 8 * (s & 1) : 32 * j + 8 * s;
}

template <int TIER>
struct GroupA {
  static constexpr int NV = TIER == 3 ? 4 : TIER == 2 ? 2 : 1;  // 16-byte loads per row
  uint4 g[NV], u[NV];
  __device__ __forceinline__ void load(const uint8_t* rec, int d, int grp, int j) {
    const int64_t row = TIER == 3 ? 2 * (int64_t)d : TIER == 2 ? d : (d >> 1);
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      const int64_t off = TIER == 3   ? 256 * (int64_t)grp + 64 * e + 16 * j
                          : TIER == 2 ? 128 * (int64_t)grp + 64 * e + 16 * j
                                      : 64 * (int64_t)grp + 16 * j;
      g[e] = *reinterpret_cast<const uint4*>(rec + off);
      u[e] = *reinterpret_cast<const uint4*>(rec + row + off);
    }
  }
  // the 8 codes of step s, as exact fp16 values
  __device__ __forceinline__ static half8v step(const uint4 (&v)[NV], int s) {
    if (TIER == 3) {
      return __builtin_bit_cast(half8v, v[s]);
    } else if (TIER == 2) {
      const uint4 c = v[s >> 1];
      return (s & 1) ? h8(i8x4_to_h4(c.z), i8x4_to_h4(c.w)) : h8(i8x4_to_h4(c.x), i8x4_to_h4(c.y));
    } else {
      const uint4 c = v[0];
      const uint32_t w = s == 0 ? c.x : s == 1 ? c.y : s == 2 ? c.z : c.w;
      return h8(i4x4_to_h4(w & 0xffffu), i4x4_to_h4(w >> 16));
    }
  }
};

// The global loads of one group: x rows 4 q + j (q < NXQ; 16-byte chunk
// col; rows past the batch re-read the last row, and are stored as zeros)
// and the records. Every load is unconditional.
template <int TIER, int NXQ>
struct BhLoads {
  GroupA<TIER> A;
  uint4 xr[NXQ];
  __device__ __forceinline__ void issue(const uint16_t* x, const uint8_t* rec, int d, int B,
                                        int grp, int lane) {
    const int j = lane >> 4, col = lane & 15;
#pragma unroll
    for (int q = 0; q < NXQ; ++q) {
      const int row = min(4 * q + j, B - 1);
      xr[q] = *reinterpret_cast<const uint4*>(x + (int64_t)row * d + 128 * grp + 8 * col);
    }
    A.load(rec, d, grp, j);
  }
  // the x rows into the wave's LDS copy (the asm makes the values used
  // whatever the row, so that no load of a row past the batch moves under
  // a branch)
  __device__ __forceinline__ void stage(uint16_t* s_xw, int B, int lane) {
    const int j = lane >> 4, col = lane & 15;
#pragma unroll
    for (int q = 0; q < NXQ; ++q)
      asm volatile("" : "+v"(xr[q].x), "+v"(xr[q].y), "+v"(xr[q].z), "+v"(xr[q].w));
#pragma unroll
    for (int q = 0; q < NXQ; ++q) {
      const int row = 4 * q + j;
      *reinterpret_cast<uint4*>(s_xw + row * kBXRow + 8 * col) =
          row < B ? xr[q] : make_uint4(0u, 0u, 0u, 0u);
    }
  }
};

// The arithmetic of one group, x staged in s_xw.
template <int TIER, int NT>
__device__ __forceinline__ void bh_compute(const GroupA<TIER>& A, const uint16_t* s_xw,
                                           const uint16_t* s_sc, int G, int grp, int lane,
                                           float4v (&acc_g)[NT], float4v (&acc_u)[NT]) {
  const int j = lane >> 4, col = lane & 15;
  float4v tg[NT], tu[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    tg[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
    tu[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const half8v ag = GroupA<TIER>::step(A.g, s), au = GroupA<TIER>::step(A.u, s);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const half8v bx = *reinterpret_cast<const half8v*>(s_xw + (16 * t + col) * kBXRow +
                                                          bh_xcol<TIER>(j, s));
      tg[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ag, bx, tg[t], 0, 0, 0);
      tu[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(au, bx, tu[t], 0, 0, 0);
    }
  }
  // rows 4j + i of the result: scale each by its neuron's group scale
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float sg = 1.0f, su = 1.0f;
    if (TIER != 3) {
      sg = h2f(s_sc[(4 * j + i) * bh_scale_row(G) + grp]);
      su = h2f(s_sc[(4 * j + i) * bh_scale_row(G) + G + grp]);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      acc_g[t][i] = fmaf(sg, tg[t][i], acc_g[t][i]);
      acc_u[t][i] = fmaf(su, tu[t][i], acc_u[t][i]);
    }
  }
}

// NT: 16-column tiles of the batch (1 for B <= 16, 2 for B <= 32); NXQ: x
// loads per lane and group (4 NXQ >= B). s_xw: this wave's x rows (16 NT of
// kBXRow halves; rows from 4 NXQ on are zero from the start). s_sc: the
// tile's gate and up group scales, [16][bh_scale_row(G)] halves. The wave's
// groups are w, w + 8, ...; the loads of the next one go out before the
// current one's arithmetic (past the last group the prefetch re-reads the
// current one, which keeps every load unconditional).
template <int TIER, int NT, int NXQ>
__device__ __forceinline__ void bh_tier(int lane, int w, int d, int G, int B, const uint16_t* x,
                                        const uint8_t* rec, uint16_t* s_xw, const uint16_t* s_sc,
                                        float4v (&acc_g)[NT], float4v (&acc_u)[NT]) {
  int grp = w;
  if (grp >= G) return;  // wave-uniform
  BhLoads<TIER, NXQ> L0, L1;
  L0.issue(x, rec, d, B, grp, lane);
  for (;;) {
    const int g1 = grp + kBHWaves;
    L1.issue(x, rec, d, B, g1 < G ? g1 : grp, lane);
    L0.stage(s_xw, B, lane);
    bh_compute<TIER, NT>(L0.A, s_xw, s_sc, G, grp, lane, acc_g, acc_u);
    if (g1 >= G) break;
    const int g2 = g1 + kBHWaves;
    L0.issue(x, rec, d, B, g2 < G ? g2 : g1, lane);
    L1.stage(s_xw, B, lane);
    bh_compute<TIER, NT>(L1.A, s_xw, s_sc, G, g1, lane, acc_g, acc_u);
    if (g2 >= G) break;
    grp = g2;
  }
}

// LDS of ffn_bh_kernel: the waves' x rows, then (after the main loop, over
// the same bytes) the waves' partial results; the tile's gate and up scales
// follow, [16][bh_scale_row(G)] halves (rows padded to 16 bytes; G <= 128).
template <int NT>
__host__ __device__ constexpr int bh_lds_words() {
  return (kBHWaves * 16 * NT * kBXRow * 2 + 16 * bh_scale_row(128) * 2) / 16;
}
static_assert(kBHWaves * 2 * 16 * 16 * 4 <= kBHWaves * 16 * kBXRow * 2, "partials fit over the x rows");

template <int NT, int NXQ>
__global__ __launch_bounds__(kBHThreads) void ffn_bh_kernel(
    const uint16_t* __restrict__ x, int d, int B, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ work_slot, const uint32_t* __restrict__ work_mask,
    const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap, int n_slots,
    float* __restrict__ hB) {
  __shared__ uint4 bh_lds[bh_lds_words<NT>()];
  __shared__ uint32_t s_mask[16];
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  int tier, item0, nitems;
  bh_tile(blockIdx.x, n3, n2, n1, tier, item0, nitems);
  if (nitems <= 0) return;  // workgroup-uniform
  const int G = d >> 7;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint16_t* s_x = reinterpret_cast<uint16_t*>(bh_lds);
  uint16_t* s_xw = s_x + w * 16 * NT * kBXRow;
  uint16_t* s_sc = s_x + kBHWaves * 16 * NT * kBXRow;
  // The tile's slot ids by scalar loads (a wave-uniform range, inside the
  // plan's spare work_slot entries past the list), which do not queue behind
  // other workgroups' vector loads; each lane then picks the ids it needs with
  // branch-free masks.
  int u[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int s = __builtin_amdgcn_readfirstlane(work_slot[item0 + k]);
    u[k] = k < nitems && s >= 0 && s < n_slots ? s : n_slots;  // zero slot for padding
  }
  int my_slot = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) my_slot |= u[k] & -((lane & 15) == k);
  const uint32_t my_mask = work_mask[min(item0 + (lane & 15), cap - 1)];  // stored after the main loop
  const uint8_t* rec = slots + (int64_t)my_slot * slot_bytes;
  // the tile's gate and up scales (4 G contiguous bytes per record) into LDS
  if (tier != 3) {
    const int cpr = bh_scale_row(G) / 8;  // 16-byte chunks per row (the last may pass 4 G bytes)
    const int r = threadIdx.x / cpr, c = threadIdx.x - r * cpr;
    if (r < 16) {
      int sr = 0;
#pragma unroll
      for (int k = 0; k < 16; ++k) sr |= u[k] & -(r == k);
      const int64_t sbase = tier == 1 ? 3 * (int64_t)(d >> 1) : 3 * (int64_t)d;
      reinterpret_cast<uint4*>(s_sc)[r * cpr + c] =
          *reinterpret_cast<const uint4*>(slots + (int64_t)sr * slot_bytes + sbase + 16 * c);
    }
  }
  // rows of the wave's x copy that the group loads never write stay zero
  for (int e = lane; e < (16 * NT - 4 * NXQ) * (kBXRow / 8); e += 64)
    reinterpret_cast<uint4*>(s_xw + 4 * NXQ * kBXRow)[e] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  float4v acc_g[NT], acc_u[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    acc_g[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
    acc_u[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  }
  if (tier == 3)
    bh_tier<3, NT, NXQ>(lane, w, d, G, B, x, rec, s_xw, s_sc, acc_g, acc_u);
  else if (tier == 2)
    bh_tier<2, NT, NXQ>(lane, w, d, G, B, x, rec, s_xw, s_sc, acc_g, acc_u);
  else
    bh_tier<1, NT, NXQ>(lane, w, d, G, B, x, rec, s_xw, s_sc, acc_g, acc_u);
  if (threadIdx.x < 16) s_mask[threadIdx.x] = my_slot < n_slots ? my_mask : 0u;
  __syncthreads();  // every wave is done with its x rows: the partials take their bytes
  // partials of the waves -> LDS: [w][gate/up][row][col]
  float* s_part = reinterpret_cast<float*>(bh_lds);
  const int j = lane >> 4, col = lane & 15;
  constexpr int NC = 16 * NT;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s_part[((w * 2 + 0) * 16 + 4 * j + i) * NC + 16 * t + col] = acc_g[t][i];
      s_part[((w * 2 + 1) * 16 + 4 * j + i) * NC + 16 * t + col] = acc_u[t][i];
    }
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * B; e += kBHThreads) {
    const int r = e / B, b = e % B;  // neuron row, batch row
    if (r >= nitems) continue;
    float a = 0.0f, u = 0.0f;
    for (int q = 0; q < kBHWaves; ++q) {  // waves in a fixed order
      a += s_part[((q * 2 + 0) * 16 + r) * NC + b];
      u += s_part[((q * 2 + 1) * 16 + r) * NC + b];
    }
    // zero where row b did not select neuron r (or its slot is invalid)
    hB[(int64_t)b * ((cap + 3) & ~3) + item0 + r] = (s_mask[r] >> b) & 1u ? silu_mul(a, u) : 0.0f;
  }
}

// ---------------------------------------------------------------------------
// Batched down projection on the matrix cores. The contraction runs over the
// neurons: for one quantization group of 128 columns,
//   y[b][c] += sum_n (h[b][n] s[n]) q[n][c],
// so each neuron's scale folds into the h side and the codes q enter the
// matrix cores exactly, as fp16. The h side is split into an fp16 high and low
// part (two MFMAs per tile) after a power-of-two normalisation per wave, which
// keeps the products at fp32-level precision whatever the magnitudes.
//
// Workgroup: one group by a run of one tier; its 8 waves take consecutive
// parts of the run, in steps of 16 neurons. In a step lane (x, j)
// (x = lane % 16, j = lane / 16) loads the 8 codes at columns 8x .. 8x + 7 of
// the group from neurons 4j .. 4j + 3; MFMA e (e = 0..7) takes code e of
// each, so that its 16 result columns are 8x + e, and the lane's A operand is
// h s of batch row x for the same four neurons.

constexpr int kDMThreads = 512;
constexpr int kDMWaves = kDMThreads / 64;
constexpr int kDMRegions = kDMWaves / 2;  // LDS partial results per workgroup
#ifndef M2C_DM_STEPS
#define M2C_DM_STEPS 1
#endif
// 16-neuron steps per wave: INT8 runs take twice and INT4 runs four times the
// FP16 count, so that every workgroup carries the same record bytes (32 KB).
template <int TIER>
__host__ __device__ constexpr int dm_steps() {
  return M2C_DM_STEPS << (3 - TIER);
}
template <int TIER>
__host__ __device__ constexpr int dm_run_len() {
  return kDMWaves * 16 * dm_steps<TIER>();
}

// a wave reads slot ids up to one run length past its run's first item
static_assert(dm_run_len<1>() <= kWorkSlotPad, "runs longer than the plan's spare work_slot entries");

// Run b of a group: up to dm_run_len<tier>() consecutive items of one tier.
__device__ __forceinline__ void dm_run(int b, int n3, int n2, int n1, int& tier, int& lo, int& hi) {
  constexpr int R3 = dm_run_len<3>(), R2 = dm_run_len<2>(), R1 = dm_run_len<1>();
  const int w3 = (n3 + R3 - 1) / R3, w2 = (n2 + R2 - 1) / R2, w1 = (n1 + R1 - 1) / R1;
  if (b < w3) {
    tier = 3;
    lo = b * R3;
    hi = min(lo + R3, n3);
  } else if (b < w3 + w2) {
    tier = 2;
    lo = n3 + (b - w3) * R2;
    hi = min(lo + R2, n3 + n2);
  } else if (b < w3 + w2 + w1) {
    tier = 1;
    lo = n3 + n2 + (b - w3 - w2) * R1;
    hi = min(lo + R1, n3 + n2 + n1);
  } else {
    tier = 0;
    lo = hi = 0;
  }
}

// The 8 codes of one neuron at the lane's columns: 16 bytes of FP16, 8 of
// INT8, 4 of INT4.
template <int TIER>
struct DmWord {
  typedef uint32_t T;
};
template <>
struct DmWord<3> {
  typedef uint4 T;
};
template <>
struct DmWord<2> {
  typedef uint2 T;
};

__device__ __forceinline__ uint32_t dm_dword(const uint4& v, int q) {
  return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
}
__device__ __forceinline__ uint32_t dm_dword(const uint2& v, int q) { return q == 0 ? v.x : v.y; }

// B operands of the 8 MFMAs of a step from the codes of the lane's neurons
// 4j + m (m = 0..3): element m of operand e is code e of neuron m, exact.
// INT8 / INT4 words arrive in offset binary (code + 128 per byte, code + 8
// per nibble); ORing the offset code under fp16 exponent 10 gives 1024 +
// offset code, and one packed subtraction restores the code.
template <int TIER>
__device__ __forceinline__ void dm_operands(const typename DmWord<TIER>::T (&c)[4],
                                            half4v (&bop)[8]) {
  if constexpr (TIER == 3) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;  // halves e & 1 of two words
      const int q = e >> 1;
      bop[e] = h4(__builtin_amdgcn_perm(dm_dword(c[1], q), dm_dword(c[0], q), sel),
                  __builtin_amdgcn_perm(dm_dword(c[3], q), dm_dword(c[2], q), sel));
    }
  } else if constexpr (TIER == 2) {
    const half4v bias = {(_Float16)1152.0f, (_Float16)1152.0f, (_Float16)1152.0f,
                         (_Float16)1152.0f};
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const int q = e >> 2;
      const uint32_t p = e & 3;
      // bytes (neuron 0 code e, neuron 1 code e, neuron 0 code e + 1, neuron 1 code e + 1)
      const uint32_t sel = p | ((4 + p) << 8) | ((p + 1) << 16) | ((5 + p) << 24);
      const uint32_t t01 = __builtin_amdgcn_perm(dm_dword(c[1], q), dm_dword(c[0], q), sel);
      const uint32_t t23 = __builtin_amdgcn_perm(dm_dword(c[3], q), dm_dword(c[2], q), sel);
      bop[e] = h4(__builtin_amdgcn_perm(0x64646464u, t01, 0x04010400u),
                  __builtin_amdgcn_perm(0x64646464u, t23, 0x04010400u)) -
               bias;
      bop[e + 1] = h4(__builtin_amdgcn_perm(0x64646464u, t01, 0x04030402u),
                      __builtin_amdgcn_perm(0x64646464u, t23, 0x04030402u)) -
                   bias;
    }
  } else {
    const half4v bias = {(_Float16)1032.0f, (_Float16)1032.0f, (_Float16)1032.0f,
                         (_Float16)1032.0f};
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const uint32_t p = e >> 1;
      // bytes (neuron 0 byte p, 0, neuron 1 byte p, 0): codes e (low nibbles) and e + 1 (high)
      const uint32_t sel = p | (0x0cu << 8) | ((4 + p) << 16) | (0x0cu << 24);
      const uint32_t t01 = __builtin_amdgcn_perm(c[1], c[0], sel);
      const uint32_t t23 = __builtin_amdgcn_perm(c[3], c[2], sel);
      bop[e] = h4((t01 & 0x000f000fu) | 0x64006400u, (t23 & 0x000f000fu) | 0x64006400u) - bias;
      bop[e + 1] = h4(((t01 >> 4) & 0x000f000fu) | 0x64006400u,
                      ((t23 >> 4) & 0x000f000fu) | 0x64006400u) -
                   bias;
    }
  }
}

__device__ __forceinline__ uint4 dm_offset(uint4 v) { return v; }
__device__ __forceinline__ uint2 dm_offset(uint2 v) {
  return make_uint2(v.x ^ 0x80808080u, v.y ^ 0x80808080u);
}
__device__ __forceinline__ uint32_t dm_offset(uint32_t v) { return v ^ 0x88888888u; }

// One wave's share of a run: neurons [first, first + 16 S) of the run's
// items, group grp; acc[t][e] gets the lane's D rows 16 t + 4 j + i of MFMA e.
// s_hw: the wave's LDS for its h values, 16 NT rows of 16 S floats.
typedef float float4u __attribute__((ext_vector_type(4), aligned(4)));
template <int TIER, int NT>
__device__ __forceinline__ void dm_wave(int first, int hi, int grp, int d, int G, int B, int cap,
                                        const int32_t* __restrict__ work_slot,
                                        const float* __restrict__ hB,
                                        const uint8_t* __restrict__ slots, int64_t slot_bytes,
                                        int n_slots, float* s_hw, float4v (&acc)[NT][8]) {
  constexpr int S = dm_steps<TIER>();
  typedef typename DmWord<TIER>::T Word;
  const int lane = threadIdx.x & 63, x = lane & 15, j = lane >> 4;
  // byte offsets in a record: the lane's 8 down codes of group grp, and the group's down scale
  const int64_t doff = TIER == 3   ? 4 * (int64_t)d + 2 * (128 * grp + 8 * x)
                       : TIER == 2 ? 2 * (int64_t)d + 128 * grp + 8 * x
                                   : (int64_t)d + 64 * grp + 4 * x;
  const int64_t soff = (TIER == 1 ? 3 * (int64_t)(d >> 1) : 3 * (int64_t)d) + 4 * G + 2 * grp;
  // Every vector load is unconditional (indices clamped into the run and the
  // batch, values masked afterwards), so that all of them are in flight at
  // once. The slot ids come first, through the scalar cache: the wave's 16
  // ids of a step are one wave-uniform range (inside the plan's spare
  // work_slot entries past the run), and a scalar load does not queue behind
  // the vector loads of other waves.
  int sl[S][4];
  // lane group j takes ids 4 j .. 4 j + 3 of each step (branch-free select)
  const int mj0 = -(j == 0), mj1 = -(j == 1), mj2 = -(j == 2), mj3 = -(j == 3);
#pragma unroll
  for (int st = 0; st < S; ++st) {
    int u[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) u[k] = __builtin_amdgcn_readfirstlane(work_slot[first + 16 * st + k]);
#pragma unroll
    for (int m = 0; m < 4; ++m)
      sl[st][m] = (u[m] & mj0) | (u[4 + m] & mj1) | (u[8 + m] & mj2) | (u[12 + m] & mj3);
  }
  // h of the wave's 16 S items for every batch row (rows cap rounded up to
  // 4 apart): 16-byte loads of 4 consecutive items, which run along a row,
  // staged through LDS; chunk e = 64 q + lane is row e / (4 S), items 4 (e %
  // (4 S)) .. + 4. Rows past the batch and items past the run are masked below.
  constexpr int CPR = 4 * S;  // 16-byte chunks per batch row
  const int hs = (cap + 3) & ~3;
  float4u hv[S * NT];
#pragma unroll
  for (int q = 0; q < S * NT; ++q) {
    const int e = 64 * q + lane, row = e / CPR, c = e - row * CPR;
    hv[q] = *reinterpret_cast<const float4u*>(hB + (int64_t)min(row, B - 1) * hs +
                                               min(first + 4 * c, hi - 1));
  }
  // phase 2: per neuron its group scale and its codes (the zero slot past the run)
  half2v sc[S][2];  // two fp16 scales per register
  Word cw[S][4];
#pragma unroll
  for (int st = 0; st < S; ++st)
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int s = first + 16 * st + 4 * j + m < hi ? sl[st][m] : -1;
      const uint8_t* rec = slots + (int64_t)(s >= 0 && s < n_slots ? s : n_slots) * slot_bytes;
      if (TIER != 3) sc[st][m >> 1][m & 1] = *reinterpret_cast<const _Float16*>(rec + soff);
      cw[st][m] = *reinterpret_cast<const Word*>(rec + doff);
    }
  __builtin_amdgcn_sched_barrier(0);  // keep every load issued before the first use
#pragma unroll
  for (int q = 0; q < S * NT; ++q) {
    const int e = 64 * q + lane, row = e / CPR, c = e - row * CPR;
    *reinterpret_cast<float4v*>(s_hw + row * 16 * S + 4 * c) = hv[q];
  }
  float a[S][NT][4];
#pragma unroll
  for (int st = 0; st < S; ++st)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float4v v = *reinterpret_cast<const float4v*>(s_hw + (16 * t + x) * 16 * S + 16 * st + 4 * j);
#pragma unroll
      for (int m = 0; m < 4; ++m) a[st][t][m] = v[m];
    }
  // h of rows past the batch and of items past the run is 0
#pragma unroll
  for (int st = 0; st < S; ++st)
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int t = 0; t < NT; ++t)
        if (16 * t + x >= B || first + 16 * st + 4 * j + m >= hi) a[st][t][m] = 0.0f;
  // A = h s, normalised so that the wave's largest |A| lies in [2^14, 2^15)
  float mx = 0.0f;
#pragma unroll
  for (int st = 0; st < S; ++st)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        if (TIER != 3) a[st][t][m] *= (float)sc[st][m >> 1][m & 1];
        mx = fmaxf(mx, fabsf(a[st][t][m]));
      }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  const int E = mx > 0.0f ? 15 - __builtin_amdgcn_frexp_expf(mx) : 0;
  half4v ahi[S][NT], alo[S][NT];
#pragma unroll
  for (int st = 0; st < S; ++st)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const float v = ldexpf(a[st][t][m], E);
        const _Float16 h = (_Float16)v;
        ahi[st][t][m] = h;
        alo[st][t][m] = (_Float16)(v - (float)h);
      }
#pragma unroll
  for (int st = 0; st < S; ++st) {
    Word c[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) c[m] = dm_offset(cw[st][m]);
    half4v bop[8];
    dm_operands<TIER>(c, bop);
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int t = 0; t < NT; ++t)
        acc[t][e] = __builtin_amdgcn_mfma_f32_16x16x16f16(ahi[st][t], bop[e], acc[t][e], 0, 0, 0);
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int t = 0; t < NT; ++t)
        acc[t][e] = __builtin_amdgcn_mfma_f32_16x16x16f16(alo[st][t], bop[e], acc[t][e], 0, 0, 0);
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[t][e][i] = ldexpf(acc[t][e][i], -E);
}

// NT: 16-row tiles of the batch (1 for B <= 16, 2 for B <= 32).
// blockIdx.x = group + G * run.
template <int NT>
__global__ __launch_bounds__(kDMThreads) void ffn_bdm_kernel(
    int d, int B, const int32_t* __restrict__ counts, const int32_t* __restrict__ work_slot,
    const float* __restrict__ hB, const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap,
    int n_slots, float* __restrict__ y) {
  constexpr int kRow = 132;  // 128 columns (in the order 16 e + x) and a pad against bank conflicts
  // [region][batch row][column]: waves 0..3 store their partial rows, then
  // waves 4..7 add theirs to them, so that every LDS word has one writer at a
  // time (LDS float atomics are slow)
  __shared__ float s_y[kDMRegions][16 * NT][kRow];
  static_assert(kDMWaves * 16 * dm_steps<1>() <= kDMRegions * kRow, "h staging fits in s_y");
  const int G = d >> 7;
  int grp = blockIdx.x % G;
  // Groups 2i and 2i + 1 of a run go to workgroup ids 8 apart: one XCD (ids
  // are dealt to the 8 XCDs in turn) and about the same start, so that a
  // 128-byte line of INT4 codes, which holds both groups of a neuron, is
  // fetched into that XCD's L2 once.
  if ((G & 15) == 0) {
    const int p = grp & 15;
    grp = (grp & ~15) + 2 * (p & 7) + (p >> 3);
  }
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  int tier, lo, hi;
  dm_run(blockIdx.x / G, n3, n2, n1, tier, lo, hi);
  if (lo >= hi) return;  // workgroup-uniform
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  float4v acc[NT][8];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[t][e] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  // the waves' h staging (16 NT rows of at most 16 dm_steps<1>() floats
  // each) lives in s_y until the partial results take it
  float* s_hw = &s_y[0][0][0] + w * 16 * NT * 16 * dm_steps<1>();
  if (tier == 3)
    dm_wave<3, NT>(lo + w * 16 * dm_steps<3>(), hi, grp, d, G, B, cap, work_slot, hB, slots,
                   slot_bytes, n_slots, s_hw, acc);
  else if (tier == 2)
    dm_wave<2, NT>(lo + w * 16 * dm_steps<2>(), hi, grp, d, G, B, cap, work_slot, hB, slots,
                   slot_bytes, n_slots, s_hw, acc);
  else
    dm_wave<1, NT>(lo + w * 16 * dm_steps<1>(), hi, grp, d, G, B, cap, work_slot, hB, slots,
                   slot_bytes, n_slots, s_hw, acc);
  __syncthreads();  // every wave's h staging is read
  const int lane = threadIdx.x & 63, x = lane & 15, j = lane >> 4;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (w / kDMRegions == pass) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 16 * t + 4 * j + i;
          if (row < B) {
            float* dst = &s_y[w % kDMRegions][row][x];
#pragma unroll
            for (int e = 0; e < 8; ++e) dst[16 * e] = pass ? dst[16 * e] + acc[t][e][i] : acc[t][e][i];
          }
        }
    }
    __syncthreads();
  }
  for (int q = threadIdx.x; q < B * 128; q += kDMThreads) {
    const int b = q >> 7, c = q & 127;
    float v = 0.0f;
#pragma unroll
    for (int r = 0; r < kDMRegions; ++r) v += s_y[r][b][16 * (c & 7) + (c >> 3)];
    atomicAdd(y + (int64_t)b * d + 128 * grp + c, v);
  }
}

static void launch_bdm(int d, int batch, int cap, hipStream_t stream, const int32_t* counts,
                       const int32_t* work_slot, const float* hB, const uint8_t* slots,
                       int64_t sb, int n_slots, float* y) {
  // runs of dm_run_len<tier>() items: at most ceil(cap / R_FP16) + 2 per group
  constexpr int R3 = dm_run_len<3>();
  const int runs = (cap + R3 - 1) / R3 + 2;
  const int G = d >> 7;
  if (batch <= 16)
    hipLaunchKernelGGL(ffn_bdm_kernel<1>, dim3(G * runs), dim3(kDMThreads), 0, stream, d, batch,
                       counts, work_slot, hB, slots, sb, cap, n_slots, y);
  else
    hipLaunchKernelGGL(ffn_bdm_kernel<2>, dim3(G * runs), dim3(kDMThreads), 0, stream, d, batch,
                       counts, work_slot, hB, slots, sb, cap, n_slots, y);
}

hipError_t launch_ffn_batch(m2c_layer* L, const uint16_t* x, int batch, const uint8_t* plan,
                            float* y, hipStream_t stream) {
  const int d = L->desc.d_model;
  const m2c_plan_layout& lay = L->layout;
  const int32_t* counts = reinterpret_cast<const int32_t*>(plan + lay.counts);
  const int32_t* work_slot = reinterpret_cast<const int32_t*>(plan + lay.work_slot);
  const uint32_t* work_mask = reinterpret_cast<const uint32_t*>(plan + lay.work_mask);
  const int64_t sb = L->info.slot_bytes;
  const int n_slots = L->desc.cache_slots + L->S;
  const int cap = L->cap;
  if (cap <= 0) return hipSuccess;
  float* hB = reinterpret_cast<float*>(L->ab);  // [batch][cap rounded up to 4]
  // tiles of 8 (FP16) and 16 items: at most ceil(cap/8) + 2 for any split into tiers
  const int tiles = (cap + 7) / 8 + 2;
  if (batch <= 8) {
    hipLaunchKernelGGL((ffn_bh_kernel<1, 2>), dim3(tiles), dim3(kBHThreads), 0, stream, x, d,
                       batch, counts, work_slot, work_mask, L->slots, sb, cap, n_slots, hB);
  } else if (batch <= 16) {
    hipLaunchKernelGGL((ffn_bh_kernel<1, 4>), dim3(tiles), dim3(kBHThreads), 0, stream, x, d,
                       batch, counts, work_slot, work_mask, L->slots, sb, cap, n_slots, hB);
  } else {
    hipLaunchKernelGGL((ffn_bh_kernel<2, 8>), dim3(tiles), dim3(kBHThreads), 0, stream, x, d,
                       batch, counts, work_slot, work_mask, L->slots, sb, cap, n_slots, hB);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  launch_bdm(d, batch, cap, stream, counts, work_slot, hB, L->slots, sb, n_slots, y);
  return hipGetLastError();
}

}  // namespace m2c
