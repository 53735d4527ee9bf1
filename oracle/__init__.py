"""CPU oracle for multi-token prediction with Viterbi-based speculative decoding.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
reference that the HIP path is checked against.  Only the test suite, the
package smoke check and the benchmark's CPU-baseline leg may import it; the
product path never calls it and shares no code with it.

Contents (paper: "Accelerating Codec-based Speech Synthesis with Multi-Token
Prediction and Speculative Decoding", arXiv 2410.13839):

  decoder.py    -- the AR module theta_AR (Sec. 3.1, Eq. 1): a decoder-only
                   Transformer over [phonemes; acoustic prompt; generated
                   tokens] with a KV cache, and the n prediction heads on the
                   last hidden state (Sec. 3.2).  float64.
  selection.py  -- emission scores S_t from each head, per-head top_k
                   candidates (Fig. 2 step 1-2), the Viterbi recursion over
                   Q(a_i, a_j) * S_t(a_j) (Sec. 3.3) and the accept rule.
                   float32, the precision the GPU takes its decisions in.
  sampling.py   -- top_k sampling inside the lattice (Fig. 2 caption): the
                   path drawn from prod exp(e_t / tau) Q by forward filtering,
                   backward sampling, with Philox4x64-10 uniforms; float32
                   arithmetic every IEEE implementation reproduces exactly.
  brute.py      -- exhaustive search over every candidate path; the definition
                   the Viterbi recursion must reproduce, and the enumerated
                   path distribution the sampler must draw from.
  generate.py   -- the AR loop: n tokens per step (Fig. 1b, Sec. 3.2).
  nar.py        -- the NAR module (Sec. 3.1, Eq. 2): codec layers 2..8 in one
                   bidirectional pass each, conditioned on the phonemes, the
                   whole prompt and the known lower layers.  float64.
  qestimate.py  -- the transition table Q from a token corpus (Sec. 3.3):
                   bigram counts within utterances, row-normalised with
                   additive smoothing, log Q in float32.

Parity status: every function is pinned by tests under tests/ (closed forms,
brute force, library routines, invariants).  The paper prints no worked
numeric example, so no value is pinned to a printed number.
"""
