"""CPU oracle for Speculative Rejection (Sun et al., NeurIPS 2024).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously-correct
re-statement of what the hot path computes.  Only the test-suite, the smoke
check and the CPU-baseline leg of the benchmark may import it; the product
library never does, and it shares no code with the GPU path.

Contents, each citing the passage it follows:

* ``philox``      -- Philox4x32-10 counter-based generator (SC'11 paper).
* ``sampler``     -- softmax sampling of the next token, eq. (auto-regressive)
                     of section 3, as an exact integer inverse CDF.
* ``transformer`` -- the decoder-only generator p and the reward model s of
                     section 3, in float64.
* ``specrej``     -- Best-of-N (section 3) and Speculative Rejection
                     (section 4.2, Algorithm 1 and eqs. partial-reward-set,
                     cutoff-threshold, accepted-set, output).
* ``diagnostics`` -- improvement score and relative compute (section 5),
                     Pearson and Kendall correlation (Appendix B).

Precision: the paper fixes none.  Model arithmetic is float64 on the given
weights; the sampler's decision (float logits -> integer token) is taken in
float32, the precision of the GPU kernel, as both sides must take it alike.
"""

