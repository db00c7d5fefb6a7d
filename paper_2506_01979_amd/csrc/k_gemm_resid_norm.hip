// GEMM kernels with the residual projection fused with the following RMSNorm epilogue.
#include "sb_gemm_kernel.h"

namespace sb {

hipError_t launch_gemm_resid_norm(const GemmArgs &a, const GemmPlan &p, hipStream_t s) {
  return launch_epi<EPI_RESID_NORM>(a, p, s);
}

}  // namespace sb
