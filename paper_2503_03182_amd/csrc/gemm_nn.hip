// NN instantiations of the GEMM family (kernel in gemm_impl.h).
#include "gemm_impl.h"

namespace tps {
hipError_t gemm_launch_nn(int dtype, GemmArgs g, hipStream_t stream) {
  return launch_layout<TPS_GEMM_NN>(dtype, g, stream);
}
}  // namespace tps
