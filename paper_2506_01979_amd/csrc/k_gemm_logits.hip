// GEMM kernels with the LM head: fp32 logits epilogue.
#include "sb_gemm_kernel.h"

namespace sb {

hipError_t launch_gemm_logits(const GemmArgs &a, const GemmPlan &p, hipStream_t s) {
  return launch_epi<EPI_LOGITS>(a, p, s);
}

}  // namespace sb
