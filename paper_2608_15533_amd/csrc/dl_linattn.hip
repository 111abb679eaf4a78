// Linear-attention instantiations of the DeltaLog decode kernels.
#include "dl_launch.hpp"

namespace dl {
hipError_t launch_linattn(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                          hipStream_t s) {
  return launch_op<OP_LINATTN>(mode, dk, dv, bf16, state_bf16, p, s);
}
}  // namespace dl
