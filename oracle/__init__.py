"""CPU oracle for one WINO decoding step and the semi-autoregressive decode.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this
package: only the test suite, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP library; the only common module is
the seeded input generator ``wino_inputs``.

Everything is plain numpy in float64, computed straight from the definitions:

* ``model``    - the masked-diffusion backbone forward over the extended
                 sequence [Y_left, Y_cur, Y_right, Y_shad] with the shadow
                 block's position ids and attention mask (Sec. 4.2.2).
* ``wino``     - confidences, the draft rule (Eq. 2), the verify rule (Eq. 3),
                 the overall update (Eq. 4), the block loop (Sec. 4.2.3) and the
                 semi-autoregressive decode (Sec. 3).
* ``epilogue`` - the decision taken directly from given logits of the current
                 and shadow blocks (the standalone epilogue workload).
* ``losses``   - per-row entropy, target log-likelihood and greedy confidence
                 of a WINO+ training state (Sec. 5.2-5.3).

Readings of points the paper leaves open are stated where they are used.
"""
from . import model, wino, epilogue, losses  # noqa: F401
