// Dispatch of the output-stationary multiply-add kernels (kernels in
// forward_kernels.h, one object file per weight mode).
#include <cstdlib>
#include <cstring>

#include "internal.h"

namespace spc {

FwdView view_of(spconv_rulebook rb) {
  FwdView v;
  v.gmap = rb->gmap;
  v.perm = rb->perm;
  v.gstride = rb->gstride;
  v.hdr = rb->hdr;
  v.n_cap = rb->n_cap;
  v.K = rb->K;
  v.n_src = rb->n_in;
  v.seg = nullptr;
  return v;
}

int forward_view(const FwdView& v, int wmode, int in_dt, const void* x, const void* w,
                 const float* bias, int out_dt, void* y, int C_in, int C_out,
                 hipStream_t stream, const Epilogue& epi) {
  if (v.n_cap == 0) return SPCONV_OK;
  FwdCall c{v, x, 0u, w, bias, y, C_out, stream, epi};
  if (!x) c.v.n_src = 0;   // no source rows (the map then names none): every gather reads 0
  bool done = false;
  switch (wmode) {
    case 0: done = forward_run_w0(c, in_dt, out_dt, C_in); break;
    case 1: done = forward_run_w1(c, in_dt, out_dt, C_in); break;
    case 2: done = forward_run_w2(c, in_dt, out_dt, C_in); break;
    default: return SPCONV_EINVAL;
  }
  if (!done) return kNotSingle;           // a segmented view with no matrix-core kernel
  return hipGetLastError() == hipSuccess ? SPCONV_OK : SPCONV_EHIP;
}

int forward(spconv_rulebook rb, int in_dt, const void* x, const void* w, const float* bias,
            int out_dt, void* y, int C_in, int C_out, hipStream_t stream) {
  return forward_view(view_of(rb), 0, in_dt, x, w, bias, out_dt, y, C_in, C_out, stream);
}

}  // namespace spc
