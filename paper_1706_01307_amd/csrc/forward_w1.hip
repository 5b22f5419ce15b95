// Matrix-core and vector kernels of weight mode 1 (the VSC input gradient, W^i = w[K-1-i]^T).
// One translation unit per weight mode keeps the library build parallel.
#include "forward_kernels.h"

namespace spc {

bool forward_run_w1(const FwdCall& c, int in_dt, int out_dt, int C_in) {
  return run<1>(c, in_dt, out_dt, C_in);
}

}  // namespace spc
