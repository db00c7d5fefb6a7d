// The persistent forward's kernels for 1 token tile(s) of 16 rows.
#include "sb_persist_kernel.h"

namespace sb {

// rt: 16-row query tiles per attention block (1, or 4 with grouped
// queries); special: the 7B-shaped tiles per pass (3 token tiles only).
const void *pk_kernel_t1(int rt, bool special) {
  if (special) return nullptr;
  if (rt == 1) return (const void *)k_persist<PkSig<1, 1, 4, 4, 8, 4, 8>>;
  if (rt == 4) return (const void *)k_persist<PkSig<1, 4, 4, 4, 8, 4, 8>>;
  return nullptr;
}

}  // namespace sb
