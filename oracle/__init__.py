"""Oracle for the branch-verification step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct CPU implementation (numpy) of what the
MI355X path computes, written from the paper:

* ``oracle.tree``     -- tree bookkeeping (parents, depths, ancestors);
* ``oracle.decoder``  -- the target forward over a token tree that shares a
  prefix KV cache (plain definition of a Llama-style decoder with a
  branch-causal key set), in float64, float32 or bfloat16 emulation;
* ``oracle.sampling`` -- row softmax statistics, target distributions, the
  speculative accept test min(1, p/q) with residual norm(max(0, p - q))
  (Preliminaries, "Speculative Decoding"), Branch Speculative Sampling
  (Appendix, Algorithm 1) at multi-child nodes, and inverse-CDF draws;
* ``oracle.rollback`` -- KV compaction to the accepted path;
* ``oracle.branching`` -- branch-point candidates (Section "Branch
  Resampling"): B = max(1, floor(k_max (1 - q(x_b)))), TopK / i.i.d. /
  without-replacement draws, each with the q row it carries;
* ``oracle.drafting`` -- the draft side of a round: the draft's float32 q
  rows and their draws, and a drafting phase with a branch point after the
  root (Section "Branch Resampling") on the same decoder definition;
* ``oracle.spec_round`` -- one whole round of Algorithm 2: the drafting
  phase, the target's chain test over the confident drafts, Algorithm 1 at
  the branch point when the chain is accepted, and both caches rolled back;
* ``oracle.hrad``     -- H-RAD's length predictor (Section "H-RAD"): the
  last K layers' hidden states and the new token's embedding through a
  256/64/3 ReLU MLP, s_t = argmax.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU baseline
may import this package.  It shares no code with the HIP path and imports
nothing from it; the product path never calls it.

Every function is pinned by ``-m "not gpu"`` tests to something other than
itself (an independent library implementation, exact enumeration of the
output distribution, closed forms printed in the paper, hand-worked golden
cases).  Nothing here is "parity unpinned".
"""

from . import tree, decoder, sampling, rollback, hrad, branching, drafting, spec_round  # noqa: F401
