"""CPU oracle for the block-scaled e4m3 Strassen-type product.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call,
link or execute anything in this package; only the test suite, the smoke
check and the benchmark's CPU-baseline leg use it.  It shares no code,
table or constant with the GPU library: it rebuilds every realization,
quantizer and product from the paper's definitions.

Modules
-------
``realizations``  exact and binary64 coefficient algebra (Section 2.1,
                  Section 3, Appendix A): the four named realizations, the
                  change-of-basis action (eq. A.1), the canonical rebalanced
                  gauge, Phi, Gamma, Brent residuals, Kronecker flattening.
``e4m3``          the OCP E4M3 codec and the block-scale rules (Appendix E.2's
                  quantization semantics), vectorised in numpy float64 where
                  every step is exact, plus a brute-force nearest-code search
                  over exact rationals for tiny inputs.
``fmm``           the fused block-scaled evaluation of a realization
                  (Assumption 1's encode -> quantize -> multiply order):
                  combine in float32, quantize, float64 sub-products,
                  W-combine, the float64 reference product and the error
                  statistics.
``model``         the second-moment model of Section 2.2 / Appendix D.
``e4m3_ref.c``    the same codec in plain C, for the exhaustive sweep over
                  all float32 bit patterns.

Every function says which passage of the paper it follows.  Where the paper
leaves a detail open (combine order, scale rule for power-of-two scales,
clamp target, sign of zero) the reading is stated where it is used.
"""
