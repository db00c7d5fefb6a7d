// The persistent forward's kernels for 3 token tile(s) of 16 rows.
#include "sb_persist_kernel.h"

namespace sb {

// rt: 16-row query tiles per attention block (3, or 4 with grouped
// queries); special: the 7B-shaped tiles per pass (3 token tiles only).
const void *pk_kernel_t3(int rt, bool special) {
  if (special) return rt == 3 ? (const void *)k_persist<PkSig<3, 3, 3, 4, 6, 4, 8>> : nullptr;
  if (rt == 3) return (const void *)k_persist<PkSig<3, 3, 4, 4, 8, 4, 8>>;
  if (rt == 4) return (const void *)k_persist<PkSig<3, 4, 4, 4, 8, 4, 8>>;
  return nullptr;
}

}  // namespace sb
