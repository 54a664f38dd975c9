"""CPU oracle of the tree-replay round (plan -> replay -> verify).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT. Only the test suite, the smoke
check of the entry module and the CPU-baseline leg of the benchmark may
import, call or execute anything in this package. The HIP library and its
Python binding never depend on it, and it never depends on them: the two
share no code, headers, tables or constants. Only the seeded input
generators (the `workloads` package, which holds none of the method's
arithmetic) serve both.

Plain, slow, binary64 NumPy, one request and one step at a time, following
the paper (Tsubame: Tree Replay for Diffusion-Based Speculative Decoding):
  philox    counter-based RNG (Salmon et al. SC'11), uniforms, Gumbel noise
  rowstats  temperature scaling, log-sum-exp, planning candidates (Section 3.1)
  planner   lazy best-first topology planning (Section 3.1, Appendix B.3)
  replay    Gumbel-top-k refill of the frozen topology (Section 3.2, eq. (2))
  verify    WoR recursive rejection sampling + bonus (eq. (1), Appendix A)
  traversal traversal verification: sequence-level RRS over the tree
            (Appendix A, Table 2)
  step      one full round per request
  exact     exact law of a round by enumeration (Section 3.3, Proposition 1)

Pins (what ties each function to something other than itself) are listed in
the tests under tests/test_oracle_*.py. The Philox stream is pinned by the
published known-answer vectors and by an independent implementation; every
other function is pinned by closed forms, brute force or exact enumeration.
Exact token outputs on the large synthetic workloads have no pin beyond
these: they are checked only as GPU-versus-oracle agreement.
"""
