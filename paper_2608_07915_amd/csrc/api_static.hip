// The decode step for callers that cannot allocate device memory: its split-K
// partials live in a file-scope device array of fixed size instead of a
// caller-provided workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "host_common.hpp"

namespace {

// One array per GPU the library runs on, held until the process ends.
__device__ __attribute__((aligned(256))) unsigned char scratch[SPECTRA_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch` on each GPU (host stand-in never used)

// Device address of this GPU's array, taken once per device with the device current.
spectra_status device_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return spectra::fail(SPECTRA_EHIP, "decode_step_static: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return spectra::fail(SPECTRA_EUNSUPPORTED, "decode_step_static: device index %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return spectra::fail(SPECTRA_EHIP, "decode_step_static: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return SPECTRA_OK;
}

}  // namespace

extern "C" spectra_status spectra_decode_step_static(const spectra_codec* ck, const spectra_codec* cv,
                                                     uint32_t* packed_k, uint32_t* packed_v, int64_t t_capacity,
                                                     int64_t t, const void* k_new, const void* v_new,
                                                     spectra_dtype kv_dt, const void* q, spectra_dtype q_dt,
                                                     int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                                     float softmax_scale, float* out, void* stream) {
  if (t < 0 || t >= t_capacity)
    return spectra::fail(SPECTRA_EINVAL, "decode_step_static: slot t=%lld outside [0, t_capacity)", (long long)t);
  const size_t need = spectra_attention_workspace_bytes(batch, n_q_heads, n_kv_heads, t + 1);
  if (need == 0) return spectra::fail(SPECTRA_EINVAL, "decode_step_static: batch and head counts must be positive");
  if (need > (size_t)SPECTRA_STATIC_SCRATCH_BYTES)
    return spectra::fail(SPECTRA_EWORKSPACE, "decode_step_static: %zu bytes of partials exceed the static %zu bytes",
                         need, (size_t)SPECTRA_STATIC_SCRATCH_BYTES);
  void* ws = nullptr;
  const spectra_status st = device_scratch(&ws);
  if (st != SPECTRA_OK) return st;
  // the partials are written before they are read, so nothing needs clearing
  return spectra_decode_step(ck, cv, packed_k, packed_v, t_capacity, t, k_new, v_new, kv_dt, q, q_dt, batch, n_q_heads,
                             n_kv_heads, softmax_scale, out, ws, (size_t)SPECTRA_STATIC_SCRATCH_BYTES, stream);
}
