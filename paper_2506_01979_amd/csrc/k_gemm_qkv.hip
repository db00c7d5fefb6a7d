// GEMM kernels with the QKV projection: RoPE on q and k, q / K / V^T writes epilogue.
#include "sb_gemm_kernel.h"

namespace sb {

hipError_t launch_gemm_qkv(const GemmArgs &a, const GemmPlan &p, hipStream_t s) {
  return launch_epi<EPI_QKV>(a, p, s);
}

}  // namespace sb
