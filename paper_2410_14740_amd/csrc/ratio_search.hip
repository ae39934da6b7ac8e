// Offline neuron-ratio search (Sec. 5.2 "Offline Neuron Ratio Search",
// Algorithm 1) on an FFN-error proxy.
//
// Algorithm 1 starts with no high-precision neurons and r_low low-precision
// ones; each iteration adds s high-precision neurons and removes s * n
// low-precision ones, where n is the ratio of their bit widths, so the bytes
// of the active neurons stay the same; every ratio is scored by an
// uncertainty estimate and the best one is kept (a later ratio wins ties).
// The paper's estimate is the entropy of a language model's token
// distributions on wikitext, which needs a trained model; here the score is
// the FFN's output error against the all-FP16 FFN over calibration tokens,
//     UQ = sum_t |y_t - y*_t|^2 / sum_t |y*_t|^2,
// where y_t is the sparse mixed-precision FFN at the ratio (top n_high +
// n_low neurons by predictor score, the n_high best at FP16, the rest at the
// low tier) and y*_t the FFN with every neuron at FP16. Every FFN runs
// through the layer's own predict / plan / fill / FFN kernels; a one-
// workgroup kernel accumulates both sums in fp64 in a fixed order.
#include <vector>

#include "m2c_internal.h"

namespace m2c {

constexpr int kErrThreads = 1024;

// acc[0] += sum_j (y_j - r_j)^2, acc[1] += sum_j r_j^2 (fp64, fixed order:
// thread strides, then a tree over the threads).
__global__ __launch_bounds__(kErrThreads) void sq_error_kernel(const float* __restrict__ y,
                                                               const float* __restrict__ ref,
                                                               int d, double* __restrict__ acc) {
  __shared__ double s_num[kErrThreads], s_den[kErrThreads];
  double num = 0.0, den = 0.0;
  for (int j = threadIdx.x; j < d; j += kErrThreads) {
    const double e = (double)y[j] - (double)ref[j];
    num += e * e;
    den += (double)ref[j] * (double)ref[j];
  }
  s_num[threadIdx.x] = num;
  s_den[threadIdx.x] = den;
  __syncthreads();
  for (int off = kErrThreads / 2; off >= 1; off >>= 1) {
    if ((int)threadIdx.x < off) {
      s_num[threadIdx.x] += s_num[threadIdx.x + off];
      s_den[threadIdx.x] += s_den[threadIdx.x + off];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    acc[0] += s_num[0];
    acc[1] += s_den[0];
  }
}

}  // namespace m2c

namespace {

struct DevBuf {
  void* p = nullptr;
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
};

}  // namespace

extern "C" m2c_status m2c_ratio_search(m2c_layer* L, const uint16_t* x, int32_t T, int32_t n_low0,
                                       int32_t step, int32_t bit_ratio, int32_t max_candidates,
                                       int32_t* n_high, int32_t* n_low, double* uq,
                                       int32_t* count, int32_t* best, void* stream) {
  if (!L || !x || !count || !best) return m2c::api_fail(M2C_ERR_INVALID_ARG, "NULL argument");
  const int d = L->desc.d_model, d_ff = L->desc.d_ff;
  if (T < 1) return m2c::api_fail(M2C_ERR_INVALID_ARG, "T %d: need at least one token", T);
  if (bit_ratio != 2 && bit_ratio != 4)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "bit_ratio %d: 2 (FP16 vs INT8) or 4 (FP16 vs INT4)",
                         bit_ratio);
  if (step < 1 || n_low0 < 0 || n_low0 > d_ff)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "step %d / n_low0 %d out of range", step, n_low0);
  if (L->desc.k_max != d_ff)
    return m2c::api_fail(M2C_ERR_CAPACITY, "the search runs the all-FP16 FFN as its reference: "
                         "create the layer with k_max = d_ff (%d)", d_ff);
  int n_cand = 0;
  while ((int64_t)n_low0 - (int64_t)(n_cand + 1) * step * bit_ratio >= 0) ++n_cand;
  *count = n_cand;
  *best = -1;
  if (n_cand > max_candidates || (n_cand > 0 && (!n_high || !n_low || !uq)))
    return m2c::api_fail(M2C_ERR_CAPACITY, "%d candidates; room for %d", n_cand, max_candidates);
  if (n_cand == 0) return M2C_OK;
  hipStream_t s = (hipStream_t)stream;
  int prev = -1;
  if (hipGetDevice(&prev) != hipSuccess) prev = -1;
  if (hipSetDevice(L->desc.device) != hipSuccess)
    return m2c::api_fail(M2C_ERR_HIP, "hipSetDevice(%d) failed", L->desc.device);
  struct Restore {
    int dev;
    ~Restore() {
      if (dev >= 0) (void)hipSetDevice(dev);
    }
  } restore{prev};
  DevBuf plan, tiers, yref, y, acc;
  hipError_t e = hipMalloc(&plan.p, (size_t)L->info.plan_bytes);
  if (e == hipSuccess) e = hipMalloc(&tiers.p, (size_t)d_ff);
  if (e == hipSuccess) e = hipMalloc(&yref.p, (size_t)T * d * 4);
  if (e == hipSuccess) e = hipMalloc(&y.p, (size_t)d * 4);
  if (e == hipSuccess) e = hipMalloc(&acc.p, (size_t)n_cand * 2 * sizeof(double));
  if (e == hipSuccess) e = hipMemsetAsync(yref.p, 0, (size_t)T * d * 4, s);
  if (e == hipSuccess) e = hipMemsetAsync(acc.p, 0, (size_t)n_cand * 2 * sizeof(double), s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return m2c::api_fail(e == hipErrorOutOfMemory ? M2C_ERR_OUT_OF_MEMORY : M2C_ERR_HIP,
                         "ratio search buffers: %s", hipGetErrorString(e));
  }
  uint8_t* tm = (uint8_t*)tiers.p;
  m2c_status rc = M2C_OK;
  // one token through predict -> plan -> fill -> FFN into out (zeroed here)
  auto ffn = [&](int t, int k, int n16, int n8, float* out) -> m2c_status {
    const uint16_t* xt = x + (int64_t)t * d;
    m2c_status r = m2c_predict_rank(L, xt, 1, k, n16, n8, nullptr, tm, s);
    if (r == M2C_OK) r = m2c_cache_plan(L, tm, 1, L->last_step + 1, plan.p, s);
    if (r == M2C_OK) r = m2c_cache_fill(L, plan.p, s);
    if (r == M2C_OK && hipMemsetAsync(out, 0, (size_t)d * 4, s) != hipSuccess)
      r = m2c::api_fail(M2C_ERR_HIP, "clear the FFN output");
    if (r == M2C_OK) r = m2c_sparse_ffn(L, xt, 1, plan.p, out, s);
    return r;
  };
  for (int t = 0; t < T && rc == M2C_OK; ++t)
    rc = ffn(t, d_ff, d_ff, 0, (float*)yref.p + (int64_t)t * d);
  for (int i = 0; i < n_cand && rc == M2C_OK; ++i) {
    const int nh = (i + 1) * step, nl = n_low0 - (i + 1) * step * bit_ratio;
    n_high[i] = nh;
    n_low[i] = nl;
    for (int t = 0; t < T && rc == M2C_OK; ++t) {
      // the nh best at FP16, the next nl at the low tier (INT8 or INT4)
      rc = ffn(t, nh + nl, nh, bit_ratio == 2 ? nl : 0, (float*)y.p);
      if (rc == M2C_OK) {
        hipLaunchKernelGGL(m2c::sq_error_kernel, dim3(1), dim3(m2c::kErrThreads), 0, s,
                           (const float*)y.p, (const float*)yref.p + (int64_t)t * d, d,
                           (double*)acc.p + 2 * i);
        if (hipGetLastError() != hipSuccess) rc = m2c::api_fail(M2C_ERR_HIP, "error kernel launch");
      }
    }
  }
  std::vector<double> sums((size_t)n_cand * 2);
  if (rc == M2C_OK) {
    e = hipMemcpyAsync(sums.data(), acc.p, sums.size() * sizeof(double), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      rc = m2c::api_fail(M2C_ERR_HIP, "ratio search: %s", hipGetErrorString(e));
    }
  } else {
    (void)hipStreamSynchronize(s);
  }
  // leave the cache cold: the search's plans are not a decode history
  if (m2c_layer_reset_cache(L, s) != M2C_OK && rc == M2C_OK) rc = M2C_ERR_HIP;
  (void)hipStreamSynchronize(s);
  if (rc != M2C_OK) return rc;
  double uq_best = 0.0;
  for (int i = 0; i < n_cand; ++i) {
    uq[i] = sums[2 * i + 1] > 0.0 ? sums[2 * i] / sums[2 * i + 1] : 0.0;
    if (*best < 0 || uq_best >= uq[i]) {  // a later ratio wins ties
      uq_best = uq[i];
      *best = i;
    }
  }
  return M2C_OK;
}
