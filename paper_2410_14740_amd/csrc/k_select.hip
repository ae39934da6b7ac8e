// Top-k selection and score-rank precision tiers (Sec. 5.2: the top-k scored
// neurons are active, and the higher the score the higher the precision).
//
// One workgroup per token. Neurons are ranked by (score descending, id
// ascending) with scores compared as order-preserving u32 keys. Three rank
// boundaries are needed -- n_fp16, n_fp16 + n_int8 and k -- and each is found
// by an MSD radix select over the keys (digits of 12, 12 and 8 bits) that
// runs all three targets through the same passes. A final pass assigns
// tiers; neurons whose key equals a boundary key are admitted in ascending
// id, using a block-wide scan of the equal-key counts.
#include "m2c_internal.h"

namespace m2c {

constexpr int kSelThreads = 1024;
constexpr int kSelBins = 4096;

__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ scores,
                                                             int d_ff, int k, int n16, int n8,
                                                             uint8_t* __restrict__ tier_map) {
  __shared__ uint32_t hist[3][kSelBins];
  __shared__ uint32_t s_prefix[3], s_remain[3];
  __shared__ uint32_t scan32[kSelThreads / 64 + 1];
  __shared__ unsigned long long scan64[kSelThreads / 64 + 1];
  const float* s = scores + (int64_t)blockIdx.x * d_ff;
  uint8_t* out = tier_map + (int64_t)blockIdx.x * d_ff;
  const int tid = threadIdx.x;
  const int R[3] = {n16, n16 + n8, k};
  if (tid < 3) {
    s_prefix[tid] = 0;
    s_remain[tid] = (uint32_t)R[tid];
  }
  const int widths[3] = {12, 12, 8};
  const int shifts[3] = {20, 8, 0};
  for (int pass = 0; pass < 3; ++pass) {
    const int width = widths[pass], shift = shifts[pass];
    const int nbins = 1 << width;
    for (int t = 0; t < 3; ++t)
      for (int b = tid; b < nbins; b += kSelThreads) hist[t][b] = 0;
    __syncthreads();
    const int top = shift + width;  // bits above this digit are the prefix
    for (int i = tid; i < d_ff; i += kSelThreads) {
      const uint32_t key = score_key(s[i]);
      const uint32_t dig = (key >> shift) & (uint32_t)(nbins - 1);
      if (pass == 0) {
        atomicAdd(&hist[0][dig], 1u);  // no prefix yet: one histogram serves all targets
      } else {
        for (int t = 0; t < 3; ++t)
          if (R[t] > 0 && (key >> top) == (s_prefix[t] >> top)) atomicAdd(&hist[t][dig], 1u);
      }
    }
    __syncthreads();
    // For every target, find the digit whose bin holds the R-th largest key:
    // threads cover bins from the highest down, a block scan gives the count
    // of keys in higher bins.
    const int bpt = nbins >= kSelThreads ? nbins / kSelThreads : 1;
    const int hi_bin = nbins - tid * bpt;  // this thread owns bins [hi_bin - bpt, hi_bin)
    for (int t = 0; t < 3; ++t) {
      if (R[t] == 0) continue;  // uniform
      const uint32_t* h = hist[pass == 0 ? 0 : t];
      uint32_t c = 0;
      if (hi_bin > 0)
        for (int b = hi_bin - 1; b >= hi_bin - bpt; --b) c += h[b];
      const uint32_t rem = s_remain[t];  // read before the scan's barriers
      uint32_t tot;
      const uint32_t above = block_exclusive_scan<uint32_t>(c, scan32, &tot);
      if (hi_bin > 0 && above < rem && above + c >= rem) {
        uint32_t cum = above;
        for (int b = hi_bin - 1; b >= hi_bin - bpt; --b) {
          if (cum + h[b] >= rem) {
            s_prefix[t] |= (uint32_t)b << shift;
            s_remain[t] = rem - cum;
            break;
          }
          cum += h[b];
        }
      }
      __syncthreads();
    }
  }
  // Tier pass. T[t] = boundary key, need[t] = how many keys equal to T[t]
  // are admitted (the lowest ids among them).
  uint32_t T[3], need[3];
  for (int t = 0; t < 3; ++t) {
    T[t] = s_prefix[t];
    need[t] = s_remain[t];
  }
  const int per = (d_ff + kSelThreads - 1) / kSelThreads;
  const int i0 = tid * per < d_ff ? tid * per : d_ff;
  const int i1 = i0 + per < d_ff ? i0 + per : d_ff;
  unsigned long long eq = 0;
  for (int i = i0; i < i1; ++i) {
    const uint32_t key = score_key(s[i]);
    for (int t = 0; t < 3; ++t)
      if (R[t] > 0 && key == T[t]) eq += 1ull << (21 * t);
  }
  unsigned long long tot64;
  const unsigned long long before = block_exclusive_scan<unsigned long long>(eq, scan64, &tot64);
  uint32_t rank[3];
  for (int t = 0; t < 3; ++t) rank[t] = (uint32_t)((before >> (21 * t)) & 0x1fffffu);
  for (int i = i0; i < i1; ++i) {
    const uint32_t key = score_key(s[i]);
    bool in[3];
    for (int t = 0; t < 3; ++t) {
      in[t] = false;
      if (R[t] > 0) {
        if (key > T[t]) {
          in[t] = true;
        } else if (key == T[t]) {
          in[t] = rank[t] < need[t];
          rank[t]++;
        }
      }
    }
    out[i] = in[0] ? 3 : in[1] ? 2 : in[2] ? 1 : 0;
  }
}

// Register-resident variant for d_ff <= 32768: every thread loads its keys
// once (neuron t + 1024 j for chunk j, so the loads are coalesced and all in
// flight together), the three radix passes read them from registers, the
// three targets share one block scan per pass (counts packed in 21-bit
// fields), and ranks among keys equal to a boundary key are computed only
// when such ties straddle a boundary (from wave ballots, in ascending id).
constexpr int kSelJ = 32;  // most chunks of 1024 neurons held in registers

__device__ __forceinline__ unsigned long long pack3(uint32_t a, uint32_t b, uint32_t c) {
  return (unsigned long long)a | ((unsigned long long)b << 21) | ((unsigned long long)c << 42);
}
__device__ __forceinline__ uint32_t field3(unsigned long long v, int t) {
  return (uint32_t)((v >> (21 * t)) & 0x1fffffu);
}

// J: chunks per thread, J >= ceil(d_ff / 1024).
template <int J>
__global__ __launch_bounds__(kSelThreads) void select_reg_kernel(const float* __restrict__ scores,
                                                                 int d_ff, int k, int n16, int n8,
                                                                 uint8_t* __restrict__ tier_map) {
  __shared__ uint32_t hist[3][kSelBins];
  __shared__ unsigned long long scan64[kSelThreads / 64 + 1];
  __shared__ uint32_t s_prefix[3], s_remain[3], s_eqtot[3];
  __shared__ uint32_t s_cnt[3][J][kSelThreads / 64];
  const float* sc = scores + (int64_t)blockIdx.x * d_ff;
  uint8_t* out = tier_map + (int64_t)blockIdx.x * d_ff;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R[3] = {n16, n16 + n8, k};
  uint32_t key[J];
#pragma unroll
  for (int j = 0; j < J; ++j) key[j] = score_key(sc[min(tid + 1024 * j, d_ff - 1)]);
  auto valid = [&](int j) { return tid + 1024 * j < d_ff; };
  if (tid < 3) {
    s_prefix[tid] = 0;
    s_remain[tid] = (uint32_t)R[tid];
  }
  // three MSD passes: 12 bits (one histogram for every target), 12, 8
  const int widths[3] = {12, 12, 8};
  const int shifts[3] = {20, 8, 0};
  for (int pass = 0; pass < 3; ++pass) {
    const int width = widths[pass], shift = shifts[pass];
    const int nbins = 1 << width;
    const int nh = pass == 0 ? 1 : 3;
    for (int t = 0; t < nh; ++t)
      for (int b = tid; b < nbins; b += kSelThreads) hist[t][b] = 0;
    __syncthreads();
    const int top = shift + width;
    uint32_t pre[3];
#pragma unroll
    for (int t = 0; t < 3; ++t) pre[t] = s_prefix[t] >> top;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (!valid(j)) continue;
      const uint32_t dig = (key[j] >> shift) & (uint32_t)(nbins - 1);
      if (pass == 0) {
        atomicAdd(&hist[0][dig], 1u);
      } else {
#pragma unroll
        for (int t = 0; t < 3; ++t)
          if (R[t] > 0 && (key[j] >> top) == pre[t]) atomicAdd(&hist[t][dig], 1u);
      }
    }
    __syncthreads();
    // thread tid owns bins [hi_bin - bpt, hi_bin), highest first
    const int bpt = nbins >= kSelThreads ? nbins / kSelThreads : 1;
    const int hi_bin = nbins - tid * bpt;
    uint32_t c[3] = {0u, 0u, 0u};
    if (hi_bin > 0) {
      for (int t = 0; t < nh; ++t)
        for (int b = hi_bin - 1; b >= hi_bin - bpt; --b) c[t] += hist[t][b];
    }
    if (pass == 0) c[1] = c[2] = c[0];
    uint32_t rem[3];
#pragma unroll
    for (int t = 0; t < 3; ++t) rem[t] = s_remain[t];  // read before the scan's barriers
    unsigned long long tot;
    const unsigned long long above = block_exclusive_scan<unsigned long long>(
        pack3(c[0], c[1], c[2]), scan64, &tot);
    if (hi_bin > 0) {
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const uint32_t ab = field3(above, t);
        if (R[t] > 0 && ab < rem[t] && ab + c[t] >= rem[t]) {
          const uint32_t* h = hist[pass == 0 ? 0 : t];
          uint32_t cum = ab;
          for (int b = hi_bin - 1; b >= hi_bin - bpt; --b) {
            if (cum + h[b] >= rem[t]) {
              s_prefix[t] |= (uint32_t)b << shift;
              s_remain[t] = rem[t] - cum;
              if (pass == 2) s_eqtot[t] = h[b];
              break;
            }
            cum += h[b];
          }
        }
      }
    }
    __syncthreads();
  }
  // Boundary key T[t]: every key above it is in; need[t] of the keys equal
  // to it are in, the lowest ids first. Targets from the widest (k) to the
  // narrowest (n_fp16), each overwriting the tier of the keys it admits.
  uint32_t tier[J];
#pragma unroll
  for (int j = 0; j < J; ++j) tier[j] = 0;
  const unsigned long long lt = (1ull << lane) - 1ull;
  for (int t = 2; t >= 0; --t) {
    if (R[t] == 0) continue;  // workgroup-uniform
    const uint32_t T = s_prefix[t], need = s_remain[t];
    const bool ordered = need < s_eqtot[t];  // ties across the boundary: workgroup-uniform
    if (ordered) {
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const unsigned long long bal = __ballot(valid(j) && key[j] == T);
        if (lane == 0) s_cnt[t][j][wave] = (uint32_t)__popcll(bal);
      }
      __syncthreads();
      if (tid == 0) {  // exclusive prefix over (chunk, wave): ascending id
        uint32_t run = 0;
        for (int jj = 0; jj < J; ++jj)
          for (int w = 0; w < kSelThreads / 64; ++w) {
            const uint32_t v = s_cnt[t][jj][w];
            s_cnt[t][jj][w] = run;
            run += v;
          }
      }
      __syncthreads();
    }
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const bool eq = valid(j) && key[j] == T;
      bool in = key[j] > T || eq;
      if (ordered) {
        const unsigned long long bal = __ballot(eq);
        in = key[j] > T || (eq && s_cnt[t][j][wave] + (uint32_t)__popcll(bal & lt) < need);
      }
      if (in) tier[j] = 3 - t;
    }
  }
#pragma unroll
  for (int j = 0; j < J; ++j)
    if (valid(j)) out[tid + 1024 * j] = (uint8_t)tier[j];
}

hipError_t launch_select(const float* scores, int batch, int d_ff, int k, int n16, int n8,
                         uint8_t* tier_map, hipStream_t stream) {
  const int J = (d_ff + kSelThreads - 1) / kSelThreads;
#define M2C_SEL(JJ)                                                                            \
  hipLaunchKernelGGL(select_reg_kernel<JJ>, dim3(batch), dim3(kSelThreads), 0, stream, scores, \
                     d_ff, k, n16, n8, tier_map)
  if (J <= 4)
    M2C_SEL(4);
  else if (J <= 8)
    M2C_SEL(8);
  else if (J <= 12)
    M2C_SEL(12);
  else if (J <= 16)
    M2C_SEL(16);
  else if (J <= 24)
    M2C_SEL(24);
  else if (J <= kSelJ)
    M2C_SEL(32);
#undef M2C_SEL
  else
    hipLaunchKernelGGL(select_kernel, dim3(batch), dim3(kSelThreads), 0, stream, scores, d_ff, k,
                       n16, n8, tier_map);
  return hipGetLastError();
}

}  // namespace m2c
