"""CPU oracle for one batched denoising step of Ripple-Pivot Search (RPS).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
float64 numpy implementation of what the GPU library computes.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it.  It
shares no code with the HIP library and never imports it; both sides receive
their inputs from the seeded generators in ``synth``.

Modules
  model   - the bidirectional masked-diffusion transformer forward (the dLLM
            p_theta of the paper's Notation paragraph, Section 3); the paper does
            not fix an architecture, the one used here is stated in ``model``.
  stats   - per-position predictive statistics: entropy H(p_i), confidence
            P_i^max, argmax and top-K (Section 3, Notation).
  rps     - the scheduler: confidence-aware commit (Eq. 1 and Eq. 2, third
            case), pivot selection (Eq. 3), adaptive candidate set, lookahead
            scoring (Eq. 4), commit/abstain and carry-over (Section 4.1).
  decode  - the semi-autoregressive RPS decoding loop (Algorithm 1, Appendix A).

Where the paper is silent or ambiguous the reading taken is stated in the
function that depends on it.
"""
