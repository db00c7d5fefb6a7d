// GEMM kernels with the residual projection, split K: delta slices for the next RMSNorm epilogue.
#include "sb_gemm_kernel.h"

namespace sb {

hipError_t launch_gemm_resid(const GemmArgs &a, const GemmPlan &p, hipStream_t s) {
  return launch_epi<EPI_RESID>(a, p, s);
}

}  // namespace sb
