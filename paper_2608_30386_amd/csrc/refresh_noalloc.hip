// dasc_refresh_noalloc: the bounded-suffix refresh of dasc_refresh for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).
//
// The only scratch the refresh kernels use is the GDN factor record of each 32-token
// chunk (dk = dv = 128 GDN heads; KDA heads and other shapes need none).  Here it lives
// in a file-scope device array of fixed size instead of a caller workspace.  Each device
// the library runs on holds its own copy of the array, at its own address, until the
// process ends.  The array's name in host code is a host-side stand-in, never a device
// address: its device address is looked up once per device with hipGetSymbolAddress, on
// the entry point's first call with that device current, and only that address is handed
// to the kernels.
//
// Every call on one device shares that device's array and leaves the last call's
// records in it.  Nothing in it must start at zero: the factor kernel writes every record
// the recurrence later reads in the same call.  Calls that overlap on one device (on
// different streams, or from different threads without ordering) race on the array.

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "dasc.h"
#include "dasc_testing.h"
#include "launch_common.h"
#include "refresh_kernels.h"

static __device__ __attribute__((aligned(256))) unsigned char scratch[DASC_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};   // device address of `scratch`, per device

// The current device's copy of the scratch array (looked up on first use).
int current_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return DASC_E_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return DASC_E_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return DASC_E_HIP;
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DASC_OK;
}

}  // namespace

extern "C" int dasc_refresh_noalloc(const dasc_shape* shape, int32_t layer,
                                    const int32_t* inv_row, float* states, int64_t n_pool,
                                    const int32_t* slot, const uint16_t* k, const uint16_t* v,
                                    const float* g, const float* beta, int32_t n_req, int32_t W,
                                    int32_t init_mode, dasc_stream_t stream) {
  if (!shape) return DASC_E_INVAL;
  size_t need = 0;
  const int rc = dasc_refresh_workspace_bytes(shape, n_req, W, &need);
  if (rc != DASC_OK) return rc;
  if (need > size_t(DASC_NOALLOC_SCRATCH_BYTES)) return DASC_E_SCRATCH;
  void* ws = nullptr;
  if (need > 0) {
    const int rs = current_scratch(&ws);
    if (rs != DASC_OK) return rs;
  }
  return dasc::refresh_impl(shape, layer, inv_row, states, n_pool, slot, k, v, g, beta, n_req, W,
                            init_mode, ws, need, DASC_REFRESH_KERNEL_AUTO, stream);
}
