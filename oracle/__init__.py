"""Float64 CPU oracle for the GliDe + CaPE hot path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct restatement of what the paper
"GliDe with a CaPE: A Low-Hassle Method to Accelerate Speculative Decoding"
(arXiv 2402.02082) computes on the decoding hot path:

* ``attention``  -- softmax attention of candidate-tree queries against a KV
                    cache under the CaPE verification mask (Sec. 4.2,
                    "Verification of Expanded Proposals", the mask_CaPE
                    equation) and the unmasked GliDe cross-attention head
                    (Sec. 4.1, the MultiHead / hd_j equations).
* ``cape``       -- confidence-aware proposal expansion into a parent-indexed
                    tree (Sec. 4.2, "Proposal Expansion", the S(p) table) and
                    its linearisation (Sec. 4.2, "Verification of Expanded
                    Proposals").
* ``verify``     -- greedy acceptance of the longest matching root path
                    (Sec. 3, speculative decoding with greedy acceptance;
                    Sec. 5.1, "Experiment design").
* ``cross_block`` -- the GliDe cross-attention sub-layer with its query and
                    output projections (Sec. 4.1, the Q^{m,j} and MultiHead
                    equations).
* ``spec_sampling`` -- chain verification with speculative sampling (Sec. 3;
                    Sec. 5.1, the GliDe-only experiments) and the expected
                    speedup model (Sec. 5.1, Metrics).
* ``block_attention`` -- the block-wise masked cross-attention of draft
                    training (Sec. 4.1, "Block-wise Attention Mask").
* ``commit``     -- the accepted path's keys and values moved behind the
                    prefix in every layer's cache, the rest discarded, and the
                    new length (Sec. 3; Sec. 4.1, the cache kept after a
                    verification step).

Only the test-suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import this package.  The HIP library never calls it and
shares no code with it; the only thing both sides share is the seeded input
generator module ``synth``, which holds none of the method's arithmetic.

Pins: every function here is checked against something other than itself in
``tests/test_oracle_*.py`` (brute force over explicit root paths with a library
causal-attention routine, the paper's own mask formula, closed forms, boundary
tables and hand-derived golden fixtures).  No function is "parity unpinned".
"""

from . import attention, block_attention, cape, commit, cross_block, spec_sampling, verify  # noqa: F401
