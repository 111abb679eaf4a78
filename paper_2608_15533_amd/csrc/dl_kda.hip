// KDA instantiations of the DeltaLog decode kernels.
#include "dl_launch.hpp"
#include "dl_tiled.hpp"

namespace dl {
hipError_t launch_kda(int mode, int dk, int dv, bool bf16, bool state_bf16, const KParams& p,
                      hipStream_t s) {
  return launch_op<OP_KDA>(mode, dk, dv, bf16, state_bf16, p, s);
}
hipError_t launch_tiled_kda(int dk, int dv, bool bf16, int nv, bool split, const KParams& p,
                            float* coef, hipStream_t s) {
  return launch_tiled_op<OP_KDA>(dk, dv, bf16, nv, split, p, coef, s);
}
}  // namespace dl
