// Create-time kernels: W_down transpose and the per-neuron record builder.
//
// A neuron is row i of W_gate and W_up plus column i of W_down (Sec. 1
// footnote); lower-scored neurons are loaded at lower precision (Sec. 5.2).
// The INT8 / INT4 copies use symmetric group-128 quantization with fp16
// scales: s = fp16_rne(fp32(amax) / qmax), q = clamp(rne(w / s)).
#include "quant_device.h"

namespace m2c {

// out[c][r] = in[r][c]; 64x64 tiles through LDS.
__global__ __launch_bounds__(256) void transpose_u16_kernel(const uint16_t* __restrict__ in,
                                                            uint16_t* __restrict__ out, int rows,
                                                            int cols) {
  __shared__ uint16_t tile[64][66];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4
  for (int r = ty; r < 64; r += 4) {
    int gr = r0 + r, gc = c0 + tx;
    tile[r][tx] = (gr < rows && gc < cols) ? in[(int64_t)gr * cols + gc] : 0;
  }
  __syncthreads();
  for (int c = ty; c < 64; c += 4) {
    int gc = c0 + c, gr = r0 + tx;
    if (gc < cols && gr < rows) out[(int64_t)gc * rows + gr] = tile[tx][c];
  }
}

// One wave per (neuron, vector). Lane l owns elements 2l and 2l+1 of every
// 128-element group. Records are written into chunk buffers that hold
// neurons i0 .. i0+n-1 (record index = neuron - i0).
__global__ __launch_bounds__(64) void quantize_records_kernel(
    const uint16_t* __restrict__ wg, const uint16_t* __restrict__ wu,
    const uint16_t* __restrict__ wdT, int d, int i0, uint8_t* __restrict__ r16, int64_t st16,
    uint8_t* __restrict__ r8, int64_t st8, uint8_t* __restrict__ r4, int64_t st4) {
  const int local = blockIdx.x;
  const int64_t i = (int64_t)i0 + local;
  const int v = blockIdx.y;  // 0 gate, 1 up, 2 down
  const int lane = threadIdx.x;
  const int G = d / 128;
  const uint16_t* src = (v == 0 ? wg : v == 1 ? wu : wdT) + i * d;
  uint8_t* f16 = r16 + local * st16 + (int64_t)v * 2 * d;
  uint8_t* c8 = r8 + local * st8 + (int64_t)v * d;
  uint8_t* s8p = r8 + local * st8 + 3 * (int64_t)d + (int64_t)v * 2 * G;
  uint8_t* c4 = r4 + local * st4 + (int64_t)v * (d / 2);
  uint8_t* s4p = r4 + local * st4 + 3 * (int64_t)(d / 2) + (int64_t)v * 2 * G;
  for (int g = 0; g < G; ++g) {
    const uint32_t pair = *reinterpret_cast<const uint32_t*>(src + g * 128 + 2 * lane);
    *reinterpret_cast<uint32_t*>(f16 + 2 * (g * 128 + 2 * lane)) = pair;
    const float amax = group_amax(pair);
    uint16_t s8, s4b;
    *reinterpret_cast<uint16_t*>(c8 + g * 128 + 2 * lane) = int8_codes(pair, amax, s8);
    c4[g * 64 + lane] = int4_codes(pair, amax, s4b);
    if (lane == 0) {
      *reinterpret_cast<uint16_t*>(s8p + 2 * g) = s8;
      *reinterpret_cast<uint16_t*>(s4p + 2 * g) = s4b;
    }
  }
}

hipError_t launch_transpose_u16(const uint16_t* in, uint16_t* out, int rows, int cols,
                                hipStream_t stream) {
  dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  hipLaunchKernelGGL(transpose_u16_kernel, grid, dim3(256), 0, stream, in, out, rows, cols);
  return hipGetLastError();
}

hipError_t launch_quantize_records(const uint16_t* wg, const uint16_t* wu, const uint16_t* wdT,
                                   int d, int i0, int n, uint8_t* r16, int64_t st16, uint8_t* r8,
                                   int64_t st8, uint8_t* r4, int64_t st4, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(quantize_records_kernel, dim3(n, 3), dim3(64), 0, stream, wg, wu, wdT, d, i0,
                     r16, st16, r8, st8, r4, st4);
  return hipGetLastError();
}

}  // namespace m2c
