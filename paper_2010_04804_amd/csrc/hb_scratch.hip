// hb_scratch.hip -- hb_predict_scratch: hb_predict_ws with the library's own
// static device scratch as the workspace, for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops).
#include <mutex>
#include <string>

#include "hb_internal.h"

namespace {

// The scratch: a file-scope device array, one copy on every GPU the library
// runs on, held until the process ends. In host code its name is only a
// stand-in for the symbol; kernels get its device address, looked up once
// per device with hipGetSymbolAddress.
__device__ __align__(256) unsigned char scratch[HB_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];

// The device address of `scratch` on `device` (looked up once, with that
// device current); nullptr after an error, with the message set.
void *scratch_on(int device) {
  if (device < 0 || device >= kMaxDevices) {
    hb::set_error(HB_ERR_INVALID_ARG, "device id out of range for the static scratch");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[device]) return g_scratch[device];
  int prev = -1;
  if (hipGetDevice(&prev) != hipSuccess) {
    hb::set_error(HB_ERR_HIP, "hipGetDevice failed");
    return nullptr;
  }
  if (prev != device && hipSetDevice(device) != hipSuccess) {
    hb::set_error(HB_ERR_HIP, "hipSetDevice failed");
    return nullptr;
  }
  void *p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (prev != device) (void)hipSetDevice(prev);
  if (e != hipSuccess || !p) {
    hb::set_error(HB_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    return nullptr;
  }
  g_scratch[device] = p;
  return p;
}

}  // namespace

extern "C" {

int hb_predict_scratch(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids, int strategy,
                       void *stream, int64_t scratch_bytes) {
  if (scratch_bytes < 0 || scratch_bytes > HB_SCRATCH_BYTES)
    return hb::set_error(HB_ERR_INVALID_ARG, "scratch_bytes " + std::to_string(scratch_bytes) +
                                                 " outside [0, HB_SCRATCH_BYTES = " +
                                                 std::to_string((long long)HB_SCRATCH_BYTES) + "]");
  if (!h) return hb::set_error(HB_ERR_INVALID_ARG, "handle is NULL");
  const int device = hb::handle_device(h);
  if (device < 0) return hb::set_error(HB_ERR_INVALID_ARG, "host-only handle: compile with a device to predict");
  void *ws = nullptr;
  if (scratch_bytes > 0 && !(ws = scratch_on(device))) return HB_ERR_HIP;
  return hb_predict_ws(h, X, n_rows, scores, leaf_ids, strategy, stream, ws, scratch_bytes);
}

}  // extern "C"
