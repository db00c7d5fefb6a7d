// The persistent forward's kernels for 2 token tile(s) of 16 rows.
#include "sb_persist_kernel.h"

namespace sb {

// rt: 16-row query tiles per attention block (2, or 4 with grouped
// queries); special: the 7B-shaped tiles per pass (3 token tiles only).
const void *pk_kernel_t2(int rt, bool special) {
  if (special) return nullptr;
  if (rt == 2) return (const void *)k_persist<PkSig<2, 2, 4, 4, 8, 4, 8>>;
  if (rt == 4) return (const void *)k_persist<PkSig<2, 4, 4, 4, 8, 4, 8>>;
  return nullptr;
}

}  // namespace sb
