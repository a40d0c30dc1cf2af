// TN instantiations of the GEMM family (kernel in gemm_impl.h).
#include "gemm_impl.h"

namespace tps {
hipError_t gemm_launch_tn(int dtype, GemmArgs g, hipStream_t stream) {
  return launch_layout<TPS_GEMM_TN>(dtype, g, stream);
}
}  // namespace tps
