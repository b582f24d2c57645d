"""CPU fp64 oracle for the SLORR regularizer hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product library (the HIP path and its
Python binding) may import, call or link anything in this package; only the
test-suite, the smoke check and the CPU-baseline leg of the benchmark use it.

Contents
  pe_schedule  greedy minimax odd-polynomial schedule of Polar Express
               (Sec. 3 "Computing the polar factor"; App. E.1: l = 1e-3, d = 5)
  slorr        the approximate forward + backward of SLORR-Hoyer and SLORR-Nuc,
               step by step as Sec. 3 and Listing 1 define it, in float64
  exact        SVD-based exact quantities used only to pin the oracle
               (Eq. SLORR_grads, Prop. 1, Prop. 2)

Everything is plain NumPy in float64. No blocking, fusion or reordering beyond
what the paper's definitions state.
"""
