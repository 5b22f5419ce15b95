// Matrix-core and vector kernels of weight mode 0 (the forward, W^i = w[i]).
// One translation unit per weight mode keeps the library build parallel.
#include "forward_kernels.h"

namespace spc {

bool forward_run_w0(const FwdCall& c, int in_dt, int out_dt, int C_in) {
  return run<0>(c, in_dt, out_dt, C_in);
}

}  // namespace spc
