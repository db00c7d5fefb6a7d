// GEMM kernels with the gate/up projection: SwiGLU into the packed activation (optionally after the RMSNorm scale) epilogue.
#include "sb_gemm_kernel.h"

namespace sb {

hipError_t launch_gemm_swiglu(const GemmArgs &a, const GemmPlan &p, hipStream_t s) {
  return launch_epi<EPI_SWIGLU>(a, p, s);
}

}  // namespace sb
