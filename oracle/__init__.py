"""CPU oracle for the TPP-SD hot path: TEST INFRASTRUCTURE ONLY.

A plain, slow float64 implementation of what the sampler computes, written
from the paper (CDF-based Transformer TPP of §4.2, TPP-SD of §4.3,
Theorem 1, Algorithm 1, App. A.1-A.3), used to check the HIP path. It shares
no code with the HIP path and imports nothing from it. Only tests/,
__graft_entry__.smoke() and bench.py's cpu_baseline leg may import it; the
product path never calls it.

Modules:
  philox   - Philox4x64-10 counter-based uniforms (pinned to numpy's Philox)
  numerics - bf16 rounding emulation, log-softmax / logsumexp
  model    - encoder (temporal encoding, type embedding, causal Transformer)
             and decoder (log-normal mixture + categorical type head)
  sampler  - naive AR sampling and the TPP-SD round (draft, verify, accept,
             adjusted-distribution replacement, bonus, commit)

Parity status: every function is pinned by a CPU test (tests/test_oracle_*.py)
against a library routine, a closed form, an invariant or brute-force
enumeration; the absolute outputs of the randomly initialised models have no
printed worked example in the paper ("parity unpinned" beyond those pins).
"""
