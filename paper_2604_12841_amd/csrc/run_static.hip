// run_static.hip -- predecoder_run_static: the whole path of predecoder_run
// with its workspace in a fixed device array of the library instead of the
// handle's, so that a call allocates nothing (for callers that cannot
// allocate: code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).
//
// The array is a file-scope __device__ variable: every device the library
// runs on holds its own copy, at its own address, until the process ends.
// In host code its name stands for a host-side shadow, not a device address,
// so the device address is looked up once per device (with that device
// current) and only that address is handed to the kernels.  Every call on a
// device shares its array, which keeps the last call's contents: the call
// clears what must start at zero, and calls that overlap on one device race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/predecoder.h"
#include "internal.h"

static __device__ __align__(256) unsigned char scratch[PD_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch` per device, once looked up

// The device address of the current device's array (looked up on the first
// call on that device).
pd_status scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return PD_ERR_DEVICE;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return PD_ERR_DEVICE;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PD_OK;
}

}  // namespace

extern "C" pd_status predecoder_run_static(pd_predecoder* h, void* hip_stream, const uint64_t* det, int32_t batch,
                                           uint64_t* flips, uint64_t* residual, float* logits) {
  if (!h || !det || !flips || !residual || batch < 1) return PD_ERR_INVALID_ARG;
  void* base = nullptr;
  const pd_status s = scratch_of_current_device(&base);
  if (s != PD_OK) return s;
  return pd::run_in_region(h, (hipStream_t)hip_stream, det, batch, flips, residual, logits, base,
                           (size_t)PD_STATIC_SCRATCH_BYTES);
}
