// The rate estimate for callers that cannot allocate device memory (code under
// graph capture, serving loops, harnesses that forbid hipMalloc): no context,
// no workspace.  Its partial sums live in a file-scope device array, one copy
// per GPU, whose address is taken once per device with hipGetSymbolAddress.
#include <mutex>
#include <string>

#include "../../include/ncodec.h"
#include "common.hpp"
#include "internal.hpp"

namespace {

// kBitsBlocks partial sums of k_bits (8 KiB); every launch of k_bits writes all
// of them before k_reduce reads them, so no clearing is needed.
static __device__ __align__(256) double scratch[nc::kBitsBlocks];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
double* g_scratch[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (the host-side name is
// not a device address).  Taken once per device, with that device current.
hipError_t scratch_ptr(int dev, double** out) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = (double*)p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" ncodec_status ncodec_estimate_bits_noalloc(const int16_t* d_q, const float* d_sigma, int64_t n,
                                                      double* d_bits, void* hip_stream) {
  if (!d_bits) return nc::set_error(NCODEC_EINVAL, "estimate_bits_noalloc: d_bits is NULL");
  if (n < 0 || n >= ((int64_t)1 << 31))
    return nc::set_error(NCODEC_EINVAL, "estimate_bits_noalloc: n = " + std::to_string(n) +
                                            " is outside [0, 2^31), the largest count the fixed " +
                                            std::to_string(nc::kBitsBlocks) + "-partial scratch serves");
  if (n > 0 && (!d_q || !d_sigma)) return nc::set_error(NCODEC_EINVAL, "estimate_bits_noalloc: d_q and d_sigma must be non-NULL");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess && (dev < 0 || dev >= kMaxDevices)) e = hipErrorInvalidDevice;
  if (e == hipSuccess) e = hipGetLastError();  // an earlier asynchronous failure
  double* part = nullptr;
  if (e == hipSuccess) e = scratch_ptr(dev, &part);
  if (e == hipSuccess) e = nc::launch_estimate_bits(d_q, d_sigma, nullptr, n, part, d_bits, (hipStream_t)hip_stream);
  if (e != hipSuccess) return nc::set_error(NCODEC_EHIP, std::string("estimate_bits_noalloc: ") + hipGetErrorString(e));
  return NCODEC_OK;
}
