// m2c_predict_rank_noalloc: the predictor + top-k entry point for callers
// that cannot allocate device memory. Its scratch lives in one fixed device
// array per GPU instead of the layer's buffers; the call allocates nothing.
#include <mutex>

#include "m2c_internal.h"

namespace {

// The scratch of every m2c_predict_rank_noalloc call on a GPU: z of the
// batch (fp32 [batch][pred_rank], 256-byte aligned) and, when the caller
// passes no scores buffer, the scores (fp32 [batch][d_ff]) right after it.
// Each GPU the library runs on holds its own copy until the process ends.
static __device__ __align__(256) uint8_t scratch[M2C_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
uint8_t* g_scratch[kMaxDevices] = {};  // device address of `scratch`, per device

// Device address of this device's `scratch`, looked up once per device with
// the device current. In host code the name `scratch` is only a host-side
// handle: kernels get this address, never the name.
m2c_status scratch_address(int device, uint8_t** out) {
  if (device < 0 || device >= kMaxDevices)
    return m2c::api_fail(M2C_ERR_INVALID_ARG, "device %d: at most %d devices", device,
                         kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return m2c::api_fail(M2C_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", device,
                           hipGetErrorString(e));
    }
    g_scratch[device] = (uint8_t*)p;
  }
  *out = g_scratch[device];
  return M2C_OK;
}

struct CurrentDevice {
  int prev = -1;
  bool ok = false;
  explicit CurrentDevice(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    ok = hipSetDevice(dev) == hipSuccess;
  }
  ~CurrentDevice() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

}  // namespace

extern "C" m2c_status m2c_predict_rank_noalloc(m2c_layer* L, const uint16_t* x, int32_t batch,
                                               int32_t k, int32_t n_fp16, int32_t n_int8,
                                               float* scores, uint8_t* tier_map, void* stream) {
  m2c_status rc = m2c::check_predict_args(L, x, batch, k, n_fp16, n_int8, tier_map);
  if (rc != M2C_OK) return rc;
  const int64_t z_bytes = ((int64_t)batch * L->desc.pred_rank * 4 + 255) / 256 * 256;
  const int64_t s_bytes = scores ? 0 : (int64_t)batch * L->desc.d_ff * 4;
  if (z_bytes + s_bytes > (int64_t)M2C_NOALLOC_SCRATCH_BYTES)
    return m2c::api_fail(M2C_ERR_CAPACITY,
                         "scratch of %lld bytes (z%s) exceeds M2C_NOALLOC_SCRATCH_BYTES = %lld; "
                         "pass a scores buffer or a smaller batch",
                         (long long)(z_bytes + s_bytes), scores ? "" : " and scores",
                         (long long)M2C_NOALLOC_SCRATCH_BYTES);
  CurrentDevice g(L->desc.device);
  if (!g.ok) return m2c::api_fail(M2C_ERR_HIP, "hipSetDevice(%d) failed", L->desc.device);
  uint8_t* base = nullptr;
  rc = scratch_address(L->desc.device, &base);
  if (rc != M2C_OK) return rc;
  float* z = reinterpret_cast<float*>(base);
  float* sc = scores ? scores : reinterpret_cast<float*>(base + z_bytes);
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = m2c::launch_predict(L, x, batch, z, sc, s);
  if (e == hipSuccess) e = m2c::launch_select(sc, batch, L->desc.d_ff, k, n_fp16, n_int8, tier_map, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return m2c::api_fail(M2C_ERR_HIP, "predictor launch: %s", hipGetErrorString(e));
  }
  return M2C_OK;
}
