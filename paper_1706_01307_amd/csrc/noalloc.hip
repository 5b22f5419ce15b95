// Weight and bias gradients that allocate nothing: the per-chunk partial sums
// of the weight gradient and the per-row-chunk partials of the bias gradient
// go to a fixed device array of the library (one per GPU, kept until the
// process ends) instead of a caller-provided workspace.  The kernels are the
// ones spconv_backward_weight runs; they take the array's device address as
// their workspace argument.
#include <mutex>

#include "internal.h"

namespace {

using namespace spc;

constexpr size_t kScratchBytes = size_t(SPCONV_NOALLOC_SCRATCH_BYTES);

// Every partial the kernels read is written by them first in the same call,
// so nothing here needs clearing between calls.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];   // the array's device address on each device, once looked up

// The device address of `scratch` on device `dev`, which must be the current
// device.  In host code the array's name is a host-side stand-in, never a
// device address: only this looked-up pointer is handed to kernels.
int scratch_on(int dev, void** p) {
  if (dev < 0 || dev >= kMaxDevices) return SPCONV_EINVAL;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) {
      (void)hipGetLastError();
      return SPCONV_EHIP;
    }
    g_scratch[dev] = q;
  }
  *p = g_scratch[dev];
  return SPCONV_OK;
}

}  // namespace

extern "C" int spconv_backward_weight_noalloc(spconv_rulebook rb, int op, int dt, const void* x,
                                              const void* dy, float* dw, float* db, int C_in,
                                              int C_out, void* stream) {
  if (!rb || C_in < 1 || C_out < 1) return SPCONV_EINVAL;
  size_t need = 0;
  int st = spconv_backward_weight_workspace(rb, op, C_in, C_out, &need);
  if (st != SPCONV_OK) return st;
  if (need > kScratchBytes) return SPCONV_ESCRATCH;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return SPCONV_EHIP;
  }
  if (dev != rb->device) return SPCONV_EINVAL;
  void* ws = nullptr;
  st = scratch_on(dev, &ws);
  if (st != SPCONV_OK) return st;
  return spconv_backward_weight(rb, op, dt, x, dy, dw, db, C_in, C_out, ws, need, stream);
}
