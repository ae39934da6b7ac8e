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
// A lane's partial takes chunks sl, sl + L, ... of its row: all of them are
// loaded before the first fmaf (NCH >= chunks / L per lane), x of the pass
// is staged in LDS, and the fmaf chain then runs in the canonical order, so
// the wave costs one memory round trip instead of one per chunk.
template <int NCH>
__global__ __launch_bounds__(256) void pred_z_kernel(const uint16_t* __restrict__ A,
                                                     const uint16_t* __restrict__ x, int d, int r,
                                                     int nb, int L, float* __restrict__ z) {
  extern __shared__ uint4 xs[];  // [nb][d / 8]
  const int lane = threadIdx.x & 63;
  // wave index as a scalar: loops and shuffles below stay wave-uniform
  const int gw = __builtin_amdgcn_readfirstlane((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
  const int sl = lane & (L - 1);
  const int j = gw * (64 / L) + lane / L;
  const bool valid = j < r;
  const int chunks = d >> 3;
  const uint4* arow = reinterpret_cast<const uint4*>(A + (int64_t)(valid ? j : 0) * d);
  uint4 av[NCH];
#pragma unroll
  for (int q = 0; q < NCH; ++q) av[q] = arow[min(sl + q * L, chunks - 1)];
  for (int c = threadIdx.x; c < nb * chunks; c += blockDim.x)
    xs[c] = reinterpret_cast<const uint4*>(x)[c];
  __syncthreads();
  float acc[kPredBatch];
#pragma unroll
  for (int b = 0; b < kPredBatch; ++b) acc[b] = 0.0f;
#pragma unroll
  for (int q = 0; q < NCH; ++q) {
    const int c = sl + q * L;
    if (c < chunks) {
      float af[8];
      unpack8(av[q], af);
#pragma unroll
      for (int b = 0; b < kPredBatch; ++b) {
        if (b < nb) {
          float xf[8];
          unpack8(xs[b * chunks + c], xf);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[b] = __builtin_fmaf(af[e], xf[e], acc[b]);
        }
      }
    }
  }
  for (int off = L >> 1; off >= 1; off >>= 1) {
#pragma unroll
    for (int b = 0; b < kPredBatch; ++b)
      if (b < nb) acc[b] = acc[b] + __shfl_xor(acc[b], off);  // rows of the pass only
  }
  if (valid && sl == 0) {
#pragma unroll
    for (int b = 0; b < kPredBatch; ++b)
      if (b < nb) z[(int64_t)b * r + j] = acc[b];
  }
}

// s[b][i] = dot(B[i], z[b]) (+ bias[i]); z of the pass staged in LDS. A
// wave takes RB row groups (64 / L rows each) in one pass: their rows' loads
// go out before z is staged, so the two share one memory round trip. A row
// has at most 2 L chunks (r <= 1024): a lane's chunks are sl and, when it
// exists, sl + L, in that order (the canonical order of its partial).
template <int kPredRB>
__global__ __launch_bounds__(256) void pred_s_kernel(const uint16_t* __restrict__ Bm,
                                                     const float* __restrict__ z,
                                                     const float* __restrict__ bias, int d_ff,
                                                     int r, int nb, int L, int64_t s_stride,
                                                     float* __restrict__ s) {
  extern __shared__ float zs[];  // [nb][r]
  const int lane = threadIdx.x & 63;
  const int rpw = 64 / L;
  const int sl = lane & (L - 1);
  const int gw = __builtin_amdgcn_readfirstlane((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
  const int chunks = r >> 3;
  const bool two = sl + L < chunks;
  uint4 bv[kPredRB][2];
  int row[kPredRB];
#pragma unroll
  for (int rb = 0; rb < kPredRB; ++rb) {
    row[rb] = (gw * kPredRB + rb) * rpw + lane / L;
    const uint4* brow =
        reinterpret_cast<const uint4*>(Bm + (int64_t)min(row[rb], d_ff - 1) * r);
    bv[rb][0] = brow[sl];
    bv[rb][1] = brow[two ? sl + L : sl];
  }
  for (int t = threadIdx.x; t < nb * r; t += blockDim.x) zs[t] = z[t];
  __syncthreads();
#pragma unroll
  for (int rb = 0; rb < kPredRB; ++rb) {
    float acc[kPredBatch];
#pragma unroll
    for (int b = 0; b < kPredBatch; ++b) acc[b] = 0.0f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h == 1 && !two) break;
      const int c = sl + h * L;
      float bf[8];
      unpack8(bv[rb][h], bf);
#pragma unroll
      for (int b = 0; b < kPredBatch; ++b) {
        if (b < nb) {
          const float* zb = zs + b * r + 8 * c;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[b] = __builtin_fmaf(bf[e], zb[e], acc[b]);
        }
      }
    }
    for (int off = L >> 1; off >= 1; off >>= 1) {
#pragma unroll
      for (int b = 0; b < kPredBatch; ++b)
        if (b < nb) acc[b] = acc[b] + __shfl_xor(acc[b], off);  // rows of the pass only
    }
    const int i = row[rb];
    if (i < d_ff && sl == 0) {
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

template <int NCH>
static void launch_z(int blocks, size_t lds, hipStream_t stream, const uint16_t* A,
                     const uint16_t* x, int d, int r, int nb, int L, float* z) {
  hipLaunchKernelGGL(pred_z_kernel<NCH>, dim3(blocks), dim3(256), lds, stream, A, x, d, r, nb, L,
                     z);
}

hipError_t launch_predict(const m2c_layer* L, const uint16_t* x, int batch, float* z,
                          float* scores, hipStream_t stream) {
  const int d = L->desc.d_model, r = L->desc.pred_rank, d_ff = L->desc.d_ff;
  const int Lz = canon_lanes(d), Ls = canon_lanes(r);
  const int nch = ((d >> 3) + Lz - 1) / Lz;  // chunks per lane of the z kernel
  // rows per pass: at most kPredBatch, and x of the pass within 64 KB of LDS
  int per_pass = 32768 / d;
  if (per_pass > kPredBatch) per_pass = kPredBatch;
  if (per_pass < 1) per_pass = 1;
  for (int b0 = 0; b0 < batch; b0 += per_pass) {
    const int nb = batch - b0 < per_pass ? batch - b0 : per_pass;
    const int rows_z = 64 / Lz;
    const int waves_z = (r + rows_z - 1) / rows_z;
    const int bz = (waves_z + 3) / 4;
    const size_t lz = (size_t)nb * d * 2;
    const uint16_t* xb = x + (int64_t)b0 * d;
    float* zb = z + (int64_t)b0 * r;
    if (nch <= 1)
      launch_z<1>(bz, lz, stream, L->pred_a, xb, d, r, nb, Lz, zb);
    else if (nch <= 2)
      launch_z<2>(bz, lz, stream, L->pred_a, xb, d, r, nb, Lz, zb);
    else if (nch <= 4)
      launch_z<4>(bz, lz, stream, L->pred_a, xb, d, r, nb, Lz, zb);
    else if (nch <= 8)
      launch_z<8>(bz, lz, stream, L->pred_a, xb, d, r, nb, Lz, zb);
    else if (nch <= 16)
      launch_z<16>(bz, lz, stream, L->pred_a, xb, d, r, nb, Lz, zb);
    else
      launch_z<32>(bz, lz, stream, L->pred_a, xb, d, r, nb, Lz, zb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // RB row groups per wave, every wave makes a single pass; two when the
    // grid would otherwise hold many more workgroups than the chip (70B:
    // 54.5 -> 52.0 us per predict call; 7B, with fewer rows, is faster with one)
    const int rows_s = 64 / Ls;
    const int groups = (d_ff + rows_s - 1) / rows_s;
    const int rb = groups >= 16384 ? 2 : 1;
    const int waves_s = (groups + rb - 1) / rb;
    const int blocks = (waves_s + 3) / 4;
    if (rb == 2)
      hipLaunchKernelGGL(pred_s_kernel<2>, dim3(blocks), dim3(256), (size_t)nb * r * sizeof(float),
                         stream, L->pred_b, zb, L->bias, d_ff, r, nb, Ls, (int64_t)d_ff,
                         scores + (int64_t)b0 * d_ff);
    else
      hipLaunchKernelGGL(pred_s_kernel<1>, dim3(blocks), dim3(256), (size_t)nb * r * sizeof(float),
                         stream, L->pred_b, zb, L->bias, d_ff, r, nb, Ls, (int64_t)d_ff,
                         scores + (int64_t)b0 * d_ff);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace m2c
