"""Plain CPU oracle for speculative diffusion sampling with block verification.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package; only the test suite, the smoke check and the CPU
baseline leg of the benchmark do.  It shares no code with the HIP library and
imports nothing from it.

Everything is NumPy float64, written to be read against the paper
("Accelerating Speculative Diffusions via Block Verification"):

  philox     counter-based RNG (Philox4x32-10, Salmon et al. SC'11), the one
             random stream both sides implement from its published definition
  schedule   VP-SDE coefficients of the Euler-Maruyama chain
             (Sec. 2, eqs. forward-process / backward-process / target-distribution)
  gmm        closed-form Gaussian-mixture score, the target model q
  verify     log density ratios (App. A.2), token verification (Alg. 2),
             block verification (Alg. 6)
  residual   the U-distribution psi_alpha and its CDF (Prop. 1, eq. u-cdf),
             U-sampling by doubling + bisection (Alg. 7, App. A.1),
             the Decomposition residual (Alg. 5)
  sampler    the full round loop (Alg. 8, App. B) with the Free Drafter
             (Sec. 3.3) and plain Euler-Maruyama ("DDPM")

Parity status of each function is stated in its module header.
"""
