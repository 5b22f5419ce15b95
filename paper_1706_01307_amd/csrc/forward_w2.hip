// Matrix-core and vector kernels of weight mode 2 (the SC / DC input gradients and DC, W^i = w[i]^T).
// One translation unit per weight mode keeps the library build parallel.
#include "forward_kernels.h"

namespace spc {

bool forward_run_w2(const FwdCall& c, int in_dt, int out_dt, int C_in) {
  return run<2>(c, in_dt, out_dt, C_in);
}

}  // namespace spc
