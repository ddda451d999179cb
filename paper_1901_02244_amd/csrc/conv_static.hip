// conv_static.hip -- cb_test_conv for callers that cannot allocate.
//
// Code under HIP graph capture, tight serving loops and harnesses that
// forbid allocation cannot hand over scratch memory of their own.  This
// entry point runs exactly cb_test_conv, with the weight-gradient split
// partials (the only scratch its kernels use) in a device array of the
// library's own: one copy per GPU, kept until the process ends.  Every
// partial the reduction reads is written earlier in the same call (each
// (replica, split) block of the weight-gradient kernels stores its whole
// tile), so the array needs no clearing; calls that overlap on one GPU share
// it and race.
#include "crossbow_sma.h"
#include "kernels.hpp"

#include <mutex>

namespace {

__device__ __align__(256) unsigned char scratch[CB_STATIC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void* g_scratch_dev[MAX_DEVICES] = {};  // the array's address on each device

// The array's device address on the current device.  Its name in host code
// is only a host-side stand-in, so the address is looked up once per
// device, with that device current, and kept.
int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return CB_EDEVICE;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CB_EDEVICE;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return CB_OK;
}

}  // namespace

extern "C" {

int cb_test_conv_static(int k, int b, int Ci, int H, int W, int Co, int R, int stride, int pad,
                        int relu, int has_bias, const float* x, const float* params,
                        int64_t pstride, float* y, double* stats, const float* dy, float* dx,
                        float* grads, void* stream) {
  const size_t need = cb_test_conv_scratch_bytes(k, b, Ci, H, W, Co, R, stride, pad);
  if (need == 0) return CB_EINVAL;
  if (need > CB_STATIC_SCRATCH_BYTES) {
    cbk::note_error("cb_test_conv_static: the layer's weight-gradient partials need " +
                    std::to_string(need) + " bytes, more than the " +
                    std::to_string((size_t)CB_STATIC_SCRATCH_BYTES) +
                    " the library holds (use cb_test_conv with caller scratch)");
    return CB_ENOMEM;
  }
  void* p = nullptr;
  if (int rc = scratch_address(&p)) {
    cbk::note_error("cb_test_conv_static: hipGetSymbolAddress of the library's scratch failed");
    return rc;
  }
  return cb_test_conv(k, b, Ci, H, W, Co, R, stride, pad, relu, has_bias, x, params, pstride, y,
                      stats, dy, dx, grads, p, CB_STATIC_SCRATCH_BYTES, stream);
}

}  // extern "C"
