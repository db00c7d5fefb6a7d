"""MI355X-native branch-verification step of SpecBranch (arXiv 2506.01979).

The hot path -- one target-model forward over a token tree that shares a
prefix KV cache, row softmax statistics, the lossless accept/resample walk
(the paper's Branch Speculative Sampling at multi-child nodes and chain
speculative sampling below them) and KV rollback -- runs in hand-written HIP
kernels for gfx950 behind the C ABI declared in ``include/sb.h``.

``paper_2506_01979_amd.api`` is the thin Python binding (argument marshalling
only); ``paper_2506_01979_amd.synth`` holds the seeded synthetic inputs.
Importing this package loads nothing native; ``api`` loads ``libsb.so`` and
raises if it is missing.
"""

__all__ = ["api", "synth", "configs"]
