// sirius_ffn_cats_noalloc: the threshold-sparse FFN of sirius_ffn_cats for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc). Its workspace is `scratch`, a fixed device array of this library: each GPU
// the library runs on holds its own copy from module load until the process ends.
//
// In host code `scratch` names a host-side stand-in, not the device array, so its device
// address is taken once per device with hipGetSymbolAddress (on the first call that runs on
// that device, with the device current) and only that address is ever handed to kernels.
//
// The kernels are those of sirius_ffn_cats, which read nothing of the workspace they did not
// write earlier in the same call, so the array needs no clearing between calls. Calls that
// overlap on one GPU (two streams, two threads) share the array and race.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "sirius.h"
#include "kernels.h"
#include "profile.h"

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[SIRIUS_NOALLOC_SCRATCH_BYTES];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch` on each device, once taken

int noalloc_fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int noalloc_fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  sirius::set_last_error(buf);
  return code;
}

// The device `stream` launches on (the current device for the NULL stream).
hipError_t stream_device(hipStream_t stream, int* dev) {
  if (stream == nullptr) return hipGetDevice(dev);
  return hipStreamGetDevice(stream, dev);
}

// Device address of `scratch` on device `dev`, taken once with that device current.
int scratch_on(const char* fn, int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices)
    return noalloc_fail(SIRIUS_EINVAL, "%s: device %d outside [0, %d)", fn, dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_scratch[dev] == nullptr) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur >= 0 && cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess || p == nullptr)
      return noalloc_fail(SIRIUS_EHIP, "%s: scratch address on device %d: HIP error %d (%s)", fn, dev,
                          (int)e, hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return SIRIUS_OK;
}

}  // namespace

extern "C" int sirius_ffn_cats_noalloc(const float* x, int B, const uint16_t* w_gate,
                                       const uint16_t* w_up, const uint16_t* w_down, int d_model,
                                       int d_ff, float t, float norm_eps, const float* resid,
                                       float* y, int32_t* active_idx, int32_t* active_cnt,
                                       void* stream) {
  const char* fn = "sirius_ffn_cats_noalloc";
  size_t need = 0;
  int rc = sirius::ffn_cats_validate(fn, x, B, w_gate, w_up, w_down, d_model, d_ff, t, norm_eps,
                                     resid, y, active_idx, active_cnt, &need);
  if (rc) return rc;
  if (B == 0) return SIRIUS_OK;
  if (need > SIRIUS_NOALLOC_SCRATCH_BYTES)
    return noalloc_fail(SIRIUS_EWORKSPACE,
                        "%s: B=%d, d_model=%d, d_ff=%d needs %zu workspace bytes, above the fixed "
                        "scratch of %zu bytes (use sirius_ffn_cats with a workspace)",
                        fn, B, d_model, d_ff, need, (size_t)SIRIUS_NOALLOC_SCRATCH_BYTES);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = -1;
  const hipError_t e = stream_device(s, &dev);
  if (e != hipSuccess)
    return noalloc_fail(SIRIUS_EHIP, "%s: device of the stream: HIP error %d (%s)", fn, (int)e,
                        hipGetErrorString(e));
  void* ws = nullptr;
  if ((rc = scratch_on(fn, dev, &ws))) return rc;
  // per-kernel timing would create events; this path creates nothing
  sirius::ProfSuppress quiet;
  return sirius::ffn_cats_run(fn, x, B, w_gate, w_up, w_down, d_model, d_ff, t, norm_eps, resid, y,
                              active_idx, active_cnt, ws, stream);
}
