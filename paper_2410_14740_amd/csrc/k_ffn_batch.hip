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
//   ffn_bh_kernel   a workgroup takes a tile of 16 neurons of one tier; its 8
//                   waves split d by quantization group (group g to wave
//                   g % 8). For each group a wave issues
//                   v_mfma_f32_16x16x16f16 over the 128 elements: A = the 16
//                   neurons' codes (INT8 / INT4 unpacked to exact fp16),
//                   B = x of 16 batch rows (rows past the batch read zeros).
//                   The order of k inside a group is permuted the same way on
//                   both operands, so that lane group j holds 32 consecutive
//                   elements -- one 16-byte INT4 load, two INT8, four FP16.
//                   Each group's product is scaled by its fp16 scales in fp32
//                   and added up, so the dequantization stays exact. The
//                   waves' partials meet in LDS; h_{b,i} = silu(a) * u, zero
//                   where row b did not select neuron i.
//   ffn_bdn_kernel  y by column slice and single-tier run of 128 neurons, on
//                   the VALU: a lane owns 8 columns and keeps one accumulator
//                   per batch row, so every down byte is loaded once and
//                   feeds B fused multiply-adds.
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

// Tile b of 16 consecutive work items of one tier.
__device__ __forceinline__ void bh_tile(int b, int n3, int n2, int n1, int& tier, int& item0,
                                        int& nitems) {
  const int t3 = (n3 + 15) >> 4, t2 = (n2 + 15) >> 4, t1 = (n1 + 15) >> 4;
  if (b < t3) {
    tier = 3;
    item0 = 16 * b;
    nitems = min(16, n3 - item0);
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

// A operand of one group: lane (row r, lane group j) holds the 32 codes at
// positions [32j, 32j + 32) of the group, for the gate and the up row.
template <int TIER>
struct GroupA {
  static constexpr int NV = TIER == 3 ? 4 : TIER == 2 ? 2 : 1;  // 16-byte loads per row
  uint4 g[NV], u[NV];
  __device__ __forceinline__ void load(const uint8_t* rec, int d, int grp, int j) {
    const int64_t row = TIER == 3 ? 2 * (int64_t)d : TIER == 2 ? d : (d >> 1);
    // byte offset of element 128 grp + 32 j in a row
    const int64_t off = TIER == 3 ? 2 * (int64_t)(128 * grp + 32 * j)
                        : TIER == 2 ? (int64_t)(128 * grp + 32 * j)
                                    : (int64_t)((128 * grp + 32 * j) >> 1);
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      g[e] = *reinterpret_cast<const uint4*>(rec + off + 16 * e);
      u[e] = *reinterpret_cast<const uint4*>(rec + row + off + 16 * e);
    }
  }
  // codes [4s, 4s + 4) of the lane's 32
  __device__ __forceinline__ static half4v step(const uint4 (&v)[NV], int s) {
    if (TIER == 3) {
      const uint4 c = v[s >> 1];  // 8 halves per 16 bytes: steps 2q, 2q + 1 in chunk q
      return (s & 1) ? h4(c.z, c.w) : h4(c.x, c.y);
    } else if (TIER == 2) {
      const uint4 c = v[s >> 2];  // 16 codes per 16 bytes: 4 steps per chunk
      const uint32_t w = (s & 3) == 0 ? c.x : (s & 3) == 1 ? c.y : (s & 3) == 2 ? c.z : c.w;
      return i8x4_to_h4(w);
    } else {
      const uint4 c = v[0];  // 32 codes: 8 steps, 4 codes (16 bits) each
      const uint32_t w = (s >> 1) == 0 ? c.x : (s >> 1) == 1 ? c.y : (s >> 1) == 2 ? c.z : c.w;
      return i4x4_to_h4((s & 1) ? (w >> 16) : (w & 0xffffu));
    }
  }
};

// NT: 16-column tiles of the batch (1 for B <= 16, 2 for B <= 32).
template <int TIER, int NT>
__device__ __forceinline__ void bh_tier(int lane, int w, int d, int G, int B, const uint16_t* x,
                                        const uint16_t* zero_row, const uint8_t* rec,
                                        const uint8_t* const (&srec)[4], float4v (&acc_g)[NT],
                                        float4v (&acc_u)[NT]) {
  const int j = lane >> 4, col = lane & 15;
  // scales of the lane's result rows 4j + i, read with the group's codes
  const int64_t sbase = TIER == 1 ? 3 * (int64_t)(d >> 1) : 3 * (int64_t)d;
  for (int grp = w; grp < G; grp += kBHWaves) {
    GroupA<TIER> A;
    A.load(rec, d, grp, j);
    uint32_t sgu[4][2];
    if (TIER != 3) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sgu[i][0] = *reinterpret_cast<const uint16_t*>(srec[i] + sbase + 2 * (int64_t)grp);
        sgu[i][1] = *reinterpret_cast<const uint16_t*>(srec[i] + sbase + 2 * (int64_t)(G + grp));
      }
    }
    uint4 xv[NT][4];  // x[n][128 grp + 32 j .. + 32] for the lane's batch column n
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int n = 16 * t + col;
      const uint16_t* xr = n < B ? x + (int64_t)n * d : zero_row;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        xv[t][e] = *reinterpret_cast<const uint4*>(xr + 128 * grp + 32 * j + 8 * e);
    }
    float4v tg[NT], tu[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tg[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
      tu[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const half4v ag = GroupA<TIER>::step(A.g, s), au = GroupA<TIER>::step(A.u, s);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint4 c = xv[t][s >> 1];
        const half4v bx = (s & 1) ? h4(c.z, c.w) : h4(c.x, c.y);
        tg[t] = __builtin_amdgcn_mfma_f32_16x16x16f16(ag, bx, tg[t], 0, 0, 0);
        tu[t] = __builtin_amdgcn_mfma_f32_16x16x16f16(au, bx, tu[t], 0, 0, 0);
      }
    }
    // rows 4j + i of the result: scale each by its neuron's group scale
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float sg = 1.0f, su = 1.0f;
      if (TIER != 3) {
        sg = h2f((uint16_t)sgu[i][0]);
        su = h2f((uint16_t)sgu[i][1]);
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        acc_g[t][i] = fmaf(sg, tg[t][i], acc_g[t][i]);
        acc_u[t][i] = fmaf(su, tu[t][i], acc_u[t][i]);
      }
    }
  }
}

template <int NT>
__global__ __launch_bounds__(kBHThreads) void ffn_bh_kernel(
    const uint16_t* __restrict__ x, int d, int B, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ work_slot, const uint32_t* __restrict__ work_mask,
    const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap, int n_slots,
    float* __restrict__ hB) {
  extern __shared__ float s_part[];  // [waves][2][16][16 NT]
  __shared__ int s_slot[16];
  __shared__ uint32_t s_mask[16];
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  int tier, item0, nitems;
  bh_tile(blockIdx.x, n3, n2, n1, tier, item0, nitems);
  if (nitems <= 0) return;  // workgroup-uniform
  const int G = d >> 7;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (threadIdx.x < 16) {
    const bool in = threadIdx.x < nitems;
    const int s = in ? work_slot[item0 + threadIdx.x] : -1;
    const bool ok = s >= 0 && s < n_slots;
    s_slot[threadIdx.x] = ok ? s : n_slots;  // zero slot for padding
    s_mask[threadIdx.x] = in && ok ? work_mask[item0 + threadIdx.x] : 0u;
  }
  __syncthreads();
  const uint8_t* rec = slots + (int64_t)s_slot[lane & 15] * slot_bytes;
  const uint8_t* srec[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) srec[i] = slots + (int64_t)s_slot[4 * (lane >> 4) + i] * slot_bytes;
  const uint16_t* zero_row = reinterpret_cast<const uint16_t*>(slots + (int64_t)n_slots * slot_bytes);
  float4v acc_g[NT], acc_u[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    acc_g[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
    acc_u[t] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  }
  if (tier == 3)
    bh_tier<3, NT>(lane, w, d, G, B, x, zero_row, rec, srec, acc_g, acc_u);
  else if (tier == 2)
    bh_tier<2, NT>(lane, w, d, G, B, x, zero_row, rec, srec, acc_g, acc_u);
  else
    bh_tier<1, NT>(lane, w, d, G, B, x, zero_row, rec, srec, acc_g, acc_u);
  // partials of the waves -> LDS: [w][gate/up][row][col]
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
    hB[(int64_t)b * cap + item0 + r] = (s_mask[r] >> b) & 1u ? silu_mul(a, u) : 0.0f;
  }
}

constexpr int kBDThreads = 256;
constexpr int kBDRounds = 8;   // rounds of neurons whose loads are in flight together
constexpr int kBDRun = 128;    // neurons per workgroup (one tier)

// Run b of a column slice: up to kBDRun consecutive items of one tier.
__device__ __forceinline__ void bdn_run(int b, int n3, int n2, int n1, int& tier, int& lo, int& hi) {
  const int w3 = (n3 + kBDRun - 1) / kBDRun, w2 = (n2 + kBDRun - 1) / kBDRun,
            w1 = (n1 + kBDRun - 1) / kBDRun;
  if (b < w3) {
    tier = 3;
    lo = b * kBDRun;
    hi = min(lo + kBDRun, n3);
  } else if (b < w3 + w2) {
    tier = 2;
    lo = n3 + (b - w3) * kBDRun;
    hi = min(lo + kBDRun, n3 + n2);
  } else if (b < w3 + w2 + w1) {
    tier = 1;
    lo = n3 + n2 + (b - w3 - w2) * kBDRun;
    hi = min(lo + kBDRun, n3 + n2 + n1);
  } else {
    tier = 0;
    lo = hi = 0;
  }
}

// Down projection of one tier over the run (s_slot / s_h hold its items,
// s_slot the zero slot past the run) for the lane's 8 columns from `col`.
// BT: batch rows of this pass (accumulators per lane: BT x 8); LPN lanes per
// neuron.
template <int TIER, int BT, int LPN>
__device__ __forceinline__ void bdn_tier(int nrun, int col, int d, int G, int nb,
                                         const int* s_slot, const float* s_h, const uint8_t* slots,
                                         int64_t slot_bytes, float (&acc)[BT][8]) {
  constexpr int NPR = kBDThreads / LPN;
  const int r = threadIdx.x / LPN;
  for (int base = 0; base < nrun; base += NPR * kBDRounds) {
    uint4 v[kBDRounds];
    float sc[kBDRounds];
#pragma unroll
    for (int q = 0; q < kBDRounds; ++q) {
      const int ii = base + q * NPR + r;  // < kBDRun, so s_slot[ii] exists
      const uint8_t* rec = slots + (int64_t)s_slot[ii] * slot_bytes;
      if (TIER == 3) {
        v[q] = *reinterpret_cast<const uint4*>(rec + 4 * (int64_t)d + 2 * (int64_t)col);
        sc[q] = 1.0f;
      } else if (TIER == 2) {
        const uint2 t = *reinterpret_cast<const uint2*>(rec + 2 * (int64_t)d + col);
        v[q] = make_uint4(t.x, t.y, 0u, 0u);
        sc[q] = h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)d + 4 * G + 2 * (col >> 7)));
      } else {
        const uint32_t t = *reinterpret_cast<const uint32_t*>(rec + (int64_t)d + (col >> 1));
        v[q] = make_uint4(t, 0u, 0u, 0u);
        sc[q] = h2f(*reinterpret_cast<const uint16_t*>(rec + 3 * (int64_t)(d >> 1) + 4 * G +
                                                       2 * (col >> 7)));
      }
    }
#pragma unroll
    for (int q = 0; q < kBDRounds; ++q) {
      float wv[8];
      if (TIER == 3) {
        const uint32_t ws[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          wv[2 * u] = h2f((uint16_t)(ws[u] & 0xffffu));
          wv[2 * u + 1] = h2f((uint16_t)(ws[u] >> 16));
        }
      } else if (TIER == 2) {
        const uint32_t ws[2] = {v[q].x, v[q].y};
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int bb = 0; bb < 4; ++bb) wv[4 * u + bb] = (float)(int8_t)((ws[u] >> (8 * bb)) & 0xffu);
      } else {
#pragma unroll
        for (int n = 0; n < 8; ++n) {
          const int nib = (int)((v[q].x >> (4 * n)) & 0xfu);
          wv[n] = (float)(nib >= 8 ? nib - 16 : nib);
        }
      }
      // items past the run read the zero slot: data 0, scale 0, h 0
      const int ii = base + q * NPR + r;
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        if (b < nb) {
          const float c = sc[q] * s_h[b * kBDRun + ii];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[b][e] = fmaf(c, wv[e], acc[b][e]);
        }
      }
    }
  }
}

// SW: slice width (128 or 256 columns); blockIdx.x = slice + n_slices * run.
template <int BT, int SW>
__global__ __launch_bounds__(kBDThreads) void ffn_bdn_kernel(
    int d, int B, const int32_t* __restrict__ counts, const int32_t* __restrict__ work_slot,
    const float* __restrict__ hB, const uint8_t* __restrict__ slots, int64_t slot_bytes, int cap,
    int n_slots, float* __restrict__ y) {
  constexpr int LPN = SW / 8;  // lanes per neuron, 8 columns each
  constexpr int NW = kBDThreads / 64;
  extern __shared__ float s_mem[];
  int* s_slot = reinterpret_cast<int*>(s_mem);  // [kBDRun]
  float* s_h = s_mem + kBDRun;                  // [BT][kBDRun]
  float* s_row = s_h;                           // [NW][BT][SW], after s_h is read
  const int n_slices = d / SW;
  const int slice = blockIdx.x % n_slices;
  int n3, n2, n1;
  work_counts(counts, cap, n3, n2, n1);
  int tier, lo, hi;
  bdn_run(blockIdx.x / n_slices, n3, n2, n1, tier, lo, hi);
  if (lo >= hi) return;  // workgroup-uniform
  const int G = d >> 7;
  const int m = threadIdx.x % LPN;
  const int col = slice * SW + 8 * m;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nrun = hi - lo;
  for (int t = threadIdx.x; t < kBDRun; t += kBDThreads) {
    const int s = t < nrun ? work_slot[lo + t] : -1;
    s_slot[t] = s >= 0 && s < n_slots ? s : n_slots;
  }
  for (int b0 = 0; b0 < B; b0 += BT) {
    const int nb = min(BT, B - b0);
    for (int t = threadIdx.x; t < BT * kBDRun; t += kBDThreads) {
      const int b = t / kBDRun, i = t % kBDRun;
      s_h[t] = b < nb && i < nrun ? hB[(int64_t)(b0 + b) * cap + lo + i] : 0.0f;
    }
    __syncthreads();
    float acc[BT][8];
#pragma unroll
    for (int b = 0; b < BT; ++b)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[b][e] = 0.0f;
    if (tier == 3)
      bdn_tier<3, BT, LPN>(nrun, col, d, G, nb, s_slot, s_h, slots, slot_bytes, acc);
    else if (tier == 2)
      bdn_tier<2, BT, LPN>(nrun, col, d, G, nb, s_slot, s_h, slots, slot_bytes, acc);
    else
      bdn_tier<1, BT, LPN>(nrun, col, d, G, nb, s_slot, s_h, slots, slot_bytes, acc);
    // lanes m, m + LPN, ... of a wave share columns; then the waves via LDS
#pragma unroll
    for (int off = LPN; off < 64; off <<= 1)
#pragma unroll
      for (int b = 0; b < BT; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[b][e] += __shfl_xor(acc[b][e], off);
    __syncthreads();  // every wave is done with s_h, which s_row overlays
    if (lane < LPN) {
#pragma unroll
      for (int b = 0; b < BT; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e) s_row[(w * BT + b) * SW + 8 * lane + e] = acc[b][e];
    }
    __syncthreads();
    for (int t = threadIdx.x; t < nb * SW; t += kBDThreads) {
      const int b = t / SW, c = t % SW;
      float v = s_row[b * SW + c];
#pragma unroll
      for (int q = 1; q < NW; ++q) v += s_row[(q * BT + b) * SW + c];
      atomicAdd(y + (int64_t)(b0 + b) * d + slice * SW + c, v);
    }
    __syncthreads();  // s_h and s_row are reused by the next batch chunk
  }
}

template <int BT>
static void launch_bdn(int d, int batch, int cap, hipStream_t stream, const int32_t* counts,
                       const int32_t* work_slot, const float* hB, const uint8_t* slots,
                       int64_t sb, int n_slots, float* y) {
  // runs of kBDRun items: at most ceil(cap / kBDRun) + 2 per slice
  const int runs = (cap + kBDRun - 1) / kBDRun + 2;
  // 16 batch rows per pass use 128-column slices to stay within 64 KB of LDS
  const int sw = (d % 256 == 0 && BT <= 8) ? 256 : 128;
  const int hrow = BT * kBDRun, rrow = (kBDThreads / 64) * BT * sw;
  const size_t lds = (size_t)(kBDRun + (hrow > rrow ? hrow : rrow)) * 4;
  if (sw == 256)
    hipLaunchKernelGGL((ffn_bdn_kernel<BT, 256>), dim3((d / 256) * runs), dim3(kBDThreads), lds,
                       stream, d, batch, counts, work_slot, hB, slots, sb, cap, n_slots, y);
  else
    hipLaunchKernelGGL((ffn_bdn_kernel<BT, 128>), dim3((d / 128) * runs), dim3(kBDThreads), lds,
                       stream, d, batch, counts, work_slot, hB, slots, sb, cap, n_slots, y);
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
  float* hB = reinterpret_cast<float*>(L->ab);  // [batch][cap]
  // tiles of 16 items: at most ceil(cap/16) + 2 for any split into tiers
  const int tiles = (cap + 15) / 16 + 2;
  if (batch <= 16) {
    const size_t lds = (size_t)kBHWaves * 2 * 16 * 16 * 4;
    hipLaunchKernelGGL(ffn_bh_kernel<1>, dim3(tiles), dim3(kBHThreads), lds, stream, x, d, batch,
                       counts, work_slot, work_mask, L->slots, sb, cap, n_slots, hB);
  } else {
    const size_t lds = (size_t)kBHWaves * 2 * 16 * 32 * 4;
    hipLaunchKernelGGL(ffn_bh_kernel<2>, dim3(tiles), dim3(kBHThreads), lds, stream, x, d, batch,
                       counts, work_slot, work_mask, L->slots, sb, cap, n_slots, hB);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (batch <= 8)
    launch_bdn<8>(d, batch, cap, stream, counts, work_slot, hB, L->slots, sb, n_slots, y);
  else
    launch_bdn<16>(d, batch, cap, stream, counts, work_slot, hB, L->slots, sb, n_slots, y);
  return hipGetLastError();
}

}  // namespace m2c
