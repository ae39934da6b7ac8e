// Low-rank neuron predictor (Sec. 1 "Active Neuron Identification"; Sec. 5.2:
// the predictor gives every FFN neuron a score): z = A x, s = B z + bias.
//
// Every dot product follows one fixed fp32 order so the scores -- and the
// top-k ids chosen from them -- are reproducible bit for bit: chunks of 8
// consecutive elements, chunk c feeds partial c % L with
// L = min(64, largest power of two <= n/8); each partial is an fmaf chain in
// ascending order from +0; then p[l] += p[l ^ off] for off = L/2 .. 1. On the
// GPU partial l is lane l of a group of L lanes, so a wave serves 64/L rows.
#include "m2c_internal.h"

namespace m2c {

constexpr int kPredBatch = 8;  // batch rows per kernel pass

__host__ __device__ inline int canon_lanes(int n) {
  int chunks = n / 8, L = 1;
  while (L * 2 <= chunks && L < 64) L *= 2;
  return L;
}

__device__ __forceinline__ void unpack8(const uint4 v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    f[2 * q] = h2f((uint16_t)(w[q] & 0xffffu));
    f[2 * q + 1] = h2f((uint16_t)(w[q] >> 16));
  }
}

// z[b][j] for rows b < nb (x, z already offset to the first row of the pass).
__global__ __launch_bounds__(256) void pred_z_kernel(const uint16_t* __restrict__ A,
                                                     const uint16_t* __restrict__ x, int d, int r,
                                                     int nb, int L, float* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  // wave index as a scalar: loops and shuffles below stay wave-uniform
  const int gw = __builtin_amdgcn_readfirstlane((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
  const int sl = lane & (L - 1);
  const int j = gw * (64 / L) + lane / L;
  const bool valid = j < r;
  float acc[kPredBatch];
#pragma unroll
  for (int b = 0; b < kPredBatch; ++b) acc[b] = 0.0f;
  if (valid) {
    const uint4* arow = reinterpret_cast<const uint4*>(A + (int64_t)j * d);
    const int chunks = d >> 3;
#pragma unroll 2
    for (int c = sl; c < chunks; c += L) {
      float af[8];
      unpack8(arow[c], af);
#pragma unroll
      for (int b = 0; b < kPredBatch; ++b) {
        if (b < nb) {
          float xf[8];
          unpack8(reinterpret_cast<const uint4*>(x + (int64_t)b * d)[c], xf);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[b] = __builtin_fmaf(af[e], xf[e], acc[b]);
        }
      }
    }
  }
  for (int off = L >> 1; off >= 1; off >>= 1) {
#pragma unroll
    for (int b = 0; b < kPredBatch; ++b) acc[b] = acc[b] + __shfl_xor(acc[b], off);
  }
  if (valid && sl == 0) {
#pragma unroll
    for (int b = 0; b < kPredBatch; ++b)
      if (b < nb) z[(int64_t)b * r + j] = acc[b];
  }
}

// s[b][i] = dot(B[i], z[b]) (+ bias[i]); z of the pass staged in LDS.
__global__ __launch_bounds__(256) void pred_s_kernel(const uint16_t* __restrict__ Bm,
                                                     const float* __restrict__ z,
                                                     const float* __restrict__ bias, int d_ff,
                                                     int r, int nb, int L, int64_t s_stride,
                                                     float* __restrict__ s) {
  extern __shared__ float zs[];  // [nb][r]
  for (int t = threadIdx.x; t < nb * r; t += blockDim.x) zs[t] = z[t];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int rpw = 64 / L;
  const int sl = lane & (L - 1);
  const int gw = __builtin_amdgcn_readfirstlane((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
  const int nw = (gridDim.x * blockDim.x) >> 6;
  const int chunks = r >> 3;
  for (int base = gw * rpw; base < d_ff; base += nw * rpw) {
    const int i = base + lane / L;
    const bool valid = i < d_ff;
    float acc[kPredBatch];
#pragma unroll
    for (int b = 0; b < kPredBatch; ++b) acc[b] = 0.0f;
    if (valid) {
      const uint4* brow = reinterpret_cast<const uint4*>(Bm + (int64_t)i * r);
      for (int c = sl; c < chunks; c += L) {
        float bf[8];
        unpack8(brow[c], bf);
#pragma unroll
        for (int b = 0; b < kPredBatch; ++b) {
          if (b < nb) {
            const float* zb = zs + b * r + 8 * c;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[b] = __builtin_fmaf(bf[e], zb[e], acc[b]);
          }
        }
      }
    }
    for (int off = L >> 1; off >= 1; off >>= 1) {
#pragma unroll
      for (int b = 0; b < kPredBatch; ++b) acc[b] = acc[b] + __shfl_xor(acc[b], off);
    }
    if (valid && sl == 0) {
#pragma unroll
      for (int b = 0; b < kPredBatch; ++b) {
        if (b < nb) {
          float v = acc[b];
          if (bias) v = v + bias[i];
          s[(int64_t)b * s_stride + i] = v;
        }
      }
    }
  }
}

hipError_t launch_predict(const m2c_layer* L, const uint16_t* x, int batch, float* scores,
                          hipStream_t stream) {
  const int d = L->desc.d_model, r = L->desc.pred_rank, d_ff = L->desc.d_ff;
  const int Lz = canon_lanes(d), Ls = canon_lanes(r);
  for (int b0 = 0; b0 < batch; b0 += kPredBatch) {
    const int nb = batch - b0 < kPredBatch ? batch - b0 : kPredBatch;
    const int rows_z = 64 / Lz;
    const int waves_z = (r + rows_z - 1) / rows_z;
    hipLaunchKernelGGL(pred_z_kernel, dim3((waves_z + 3) / 4), dim3(256), 0, stream, L->pred_a,
                       x + (int64_t)b0 * d, d, r, nb, Lz, L->z + (int64_t)b0 * r);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int rows_s = 64 / Ls;
    int waves_s = (d_ff + rows_s - 1) / rows_s;
    int blocks = (waves_s + 3) / 4;
    const int cap = 8 * L->num_cus;
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL(pred_s_kernel, dim3(blocks), dim3(256), (size_t)nb * r * sizeof(float),
                       stream, L->pred_b, L->z + (int64_t)b0 * r, L->bias, d_ff, r, nb, Ls,
                       (int64_t)d_ff, scores + (int64_t)b0 * d_ff);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace m2c
