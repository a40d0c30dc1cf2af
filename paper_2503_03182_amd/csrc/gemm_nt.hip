// NT instantiations of the GEMM family (kernel in gemm_impl.h).
#include "gemm_impl.h"

namespace tps {
hipError_t gemm_launch_nt(int dtype, GemmArgs g, hipStream_t stream) {
  return launch_layout<TPS_GEMM_NT>(dtype, g, stream);
}
}  // namespace tps
