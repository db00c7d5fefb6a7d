// The persistent forward's kernels for 4 token tile(s) of 16 rows.
#include "sb_persist_kernel.h"

namespace sb {

// rt: 16-row query tiles per attention block (4, or 4 with grouped
// queries); special: the 7B-shaped tiles per pass (3 token tiles only).
const void *pk_kernel_t4(int rt, bool special) {
  if (special) return nullptr;
  return rt == 4 ? (const void *)k_persist<PkSig<4, 4, 4, 4, 8, 4, 8>> : nullptr;
}

}  // namespace sb
