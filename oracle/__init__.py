"""fp64 CPU oracle for the M-FAC IHVP hot path.

TEST INFRASTRUCTURE. Only tests/, __graft_entry__.smoke() and the cpu_baseline
leg of bench.py import it. The library (paper_2107_03356_amd) never imports,
links or calls anything here, and nothing here imports the library: the two
share no code. Inputs come from the caller as exact fp32 values; every
arithmetic step runs in float64 with numpy/LAPACK.

Modules:
  dynamic     plain definition of F^-1 x for the sliding window, through the
              Woodbury identity (Section 2, eq. 2; Theorem 1's F)
  recursions  the paper's own recursions: the static V/q precompute (eq. 3-4,
              Algorithm 3), the dynamic D/B/q recursions (eq. 7-8,
              Algorithms 1 and 2), the row-selected diagonal (Appendix C)
  static      block-wise inverse diagonal of F_b (Section 3.1, block-wise
              variant) through Woodbury per block
  mask        OBD saliency and the global keep-mask (Section 4.1)
  bruteforce  explicit d x d Fisher and dense solves, for tiny d only

Every function is pinned by a test in tests/test_oracle_*.py against something
other than itself (brute force, closed forms, invariants); see the docstrings.
"""

from . import bruteforce, dynamic, mask, recursions, static  # noqa: F401
