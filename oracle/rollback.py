"""Oracle KV rollback / compaction (test infrastructure only).

After verification the paper keeps the selected branch and discards the
other branches together with their KV cache (Section "Branch Resampling",
"Branch Verification").  The verify step wrote tree row i's K/V to slot
kv_len + i; compaction moves the rows on the accepted path (root, then the
accepted drafts in depth order) to the contiguous slots kv_len, kv_len+1, ...
and the cache length becomes kv_len + len(path).
"""
from __future__ import annotations

import numpy as np


def kv_rollback(K: np.ndarray, V: np.ndarray, kv_len: int, path):
    """K, V: [n_layers][n_kv][capacity][d].  Returns compacted copies and the
    new length.  Copies run in ascending j; the source row path[j] >= j, so a
    slot is never read after it has been overwritten."""
    K = K.copy()
    V = V.copy()
    for j, src in enumerate(path):
        K[:, :, kv_len + j] = K[:, :, kv_len + int(src)]
        V[:, :, kv_len + j] = V[:, :, kv_len + int(src)]
    return K, V, kv_len + len(path)
