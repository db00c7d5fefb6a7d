// Launch of the persistent bf16 forward (kernels in sb_persist_kernel.h,
// instantiated per token-tile count in k_persist_t*.hip) and the kernel that
// writes its layer table.
#include "sb_internal_fwd.h"

namespace sb {

// Kernel of a signature (k_persist_t*.hip): rt = 16-row query tiles of an
// attention block, special = the 7B-shaped tiles-per-pass set.
const void *pk_kernel_t1(int rt, bool special);
const void *pk_kernel_t2(int rt, bool special);
const void *pk_kernel_t3(int rt, bool special);
const void *pk_kernel_t4(int rt, bool special);

namespace {

__global__ void k_pk_table(PkTableArgs t) {
  const int i = threadIdx.x;
  if (i < t.n) t.dst[i] = t.layer[i];
  if (t.sync)
    for (int j = threadIdx.x; j < (int)(sizeof(PkSync) / 4); j += blockDim.x)
      ((unsigned *)t.sync)[j] = 0u;
}

}  // namespace

int pk_attn_chunks(int n_kv, int nkeys, int nwg) {
  const int steps = (nkeys + 31) / 32;
  int c = (steps + kPkAttnMaxSteps - 1) / kPkAttnMaxSteps;  // at most 16 steps per item
  const int fill = nwg / n_kv;                               // one item per workgroup
  if (c < fill) c = fill < steps ? fill : steps;
  return c < 1 ? 1 : c;
}

hipError_t launch_pk_table(const PkTableArgs &t, hipStream_t s) {
  hipLaunchKernelGGL(k_pk_table, dim3(1), dim3(256), 0, s, t);
  return hipGetLastError();
}

const void *pk_kernel(int tt, int rt, bool special) {
  switch (tt) {
    case 1: return pk_kernel_t1(rt, special);
    case 2: return pk_kernel_t2(rt, special);
    case 3: return pk_kernel_t3(rt, special);
    case 4: return pk_kernel_t4(rt, special);
    default: return nullptr;
  }
}

hipError_t launch_persist(const PkArgs &a, const void *kernel, int grid, hipStream_t s) {
  if (!kernel) return hipErrorInvalidValue;
  void *args[] = {(void *)&a};
  return hipLaunchCooperativeKernel(kernel, dim3(grid), dim3(kPkThreadsHost), args, 0, s);
}

}  // namespace sb
