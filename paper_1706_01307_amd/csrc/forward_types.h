// Types the forward kernels are compiled from: the device header of a rule
// book, the view of a gather map, and a forward call with its epilogue.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace spc {

struct DeviceHeader {          // first bytes of the rule book's allocation
  uint32_t status;             // kSt* bits
  uint32_t pad;
  int64_t n_out;               // output rows (SC: computed on the device)
};

// Forward (forward.hip).  A view names the gather map the output-stationary
// kernels walk: for output position p (rows perm[p], p < hdr->n_out <= n_cap)
// and offset i, gmap[i * gstride + p] = 1 + source row (0: none); n_src rows
// of the source features.
struct FwdView {
  const int32_t* gmap;
  const int32_t* perm;
  int64_t gstride;
  const DeviceHeader* hdr;
  int64_t n_cap;
  int64_t K;
  int64_t n_src;
  // Segmented single-offset views (K = 1): position chunks of kSegRows rows
  // belong to one offset each, seg[chunk] naming which W^i they take; a
  // position whose perm entry is negative is padding.  NULL otherwise.
  const int32_t* seg = nullptr;
};
constexpr int kSegRows = 256;
// Optional epilogue of a forward.  The networks of Section 5 follow each
// convolution with batch normalisation (at inference a per-channel affine
// map), add the block input back in residual blocks, and apply a ReLU, all at
// the active output sites; fused here into the single store of the output:
//   out[r][n] = act(acc[r][n] * scale[n] + bias[n] + res[r][n])
// scale NULL = 1, res NULL = 0 (res has the output's dtype and layout),
// relu 0 = identity, 1 = max(., 0) with NaN kept.
struct Epilogue {
  const float* scale = nullptr;
  const void* res = nullptr;
  int relu = 0;
};
struct FwdCall {
  FwdView v;
  const void* x;
  uint32_t x_bytes;
  const void* w;
  const float* bias;
  void* y;
  int C_out;
  hipStream_t stream;
  Epilogue epi;
};
// Each returns false when the view is segmented and no matrix-core kernel
// fits the shape (nothing is launched then).
bool forward_run_w0(const FwdCall& c, int in_dt, int out_dt, int C_in);
bool forward_run_w1(const FwdCall& c, int in_dt, int out_dt, int C_in);
bool forward_run_w2(const FwdCall& c, int in_dt, int out_dt, int C_in);

}  // namespace spc
