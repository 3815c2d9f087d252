"""CPU oracle for the ACE token-adaptive MoE layer — TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 numpy implementation of what the paper's method computes
(ACE: Adaptive Calibration-Free Expert Skipping, arxiv 2609.05228).  It exists
to check the HIP path and nothing else: only the tests, the package's
``smoke()`` check and the CPU-baseline leg of the benchmark may import it.
The product path never calls it and shares no code with it.

Modules
  forward  RMSNorm, router, softmax/top-k, Alg. 4 (online conservative
           skipping), the sparsified output (Eq. ace_sparse_output).
  tables   Alg. 2 (Global Spectral Proxy) and Alg. 3 (Router-Conditioned
           Refinement) offline amplification tables.
  tau      App. C.1 budget-to-threshold mapping.
  plan     The expected dispatch plan (counts, offsets, permutation) derived
           by sorting kept (expert, token) pairs.
  ties     Decision margins, tie accounting and admissibility of decisions
           taken inside the 1e-6 tie band.

Pinning status: every function is pinned by `tests/test_oracle_*.py` against
closed forms, invariants the paper proves, brute force on tiny inputs, the
hand-derived Alg. 4 worked example in `tests/golden/`, or (the tie checker)
hand-built tokens with known margins and known admissible decisions.  The absolute values
of the GSP/RCR tables for the paper's real models are parity unpinned (the
paper prints none); only their structural properties are pinned.
"""
from . import forward, plan, tables, tau, ties  # noqa: F401
