"""CPU oracle of the masked co-adaptive MoE layer -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct float64 (NumPy) and pure-Python statement of
what the masked MoE hot path computes, written from the paper:

* ``routing``  -- router logits and softmax (Section 3.1), Top-K with the
  plain rule (Eq. 1), the hard binary mask of training (Eq. 2) and the soft
  prior of inference (Eq. 4), the two gate rules (Section 3.1);
* ``ffn``      -- the expert FFN (SwiGLU) and the gate-weighted combine with
  shared experts (Eq. 1 and Section 3.1), and the same with the low-rank
  adapters of Stage 2 (Section 3.2, Appendix B);
* ``cache``    -- the per-layer expert cache of the trace simulator and the
  hit-rate / fetches-per-token metrics (Section 4.1, Eq. 5);
* ``offload``  -- a batch-1 offloaded decode of one layer: the experts each
  step fetches and evicts, and the layer output (Section 1, Section 3.1,
  Section 4.1);
* ``train``    -- Stage 1 of the fine-tuning: mask sampling without
  replacement (Eq. 2), the gradients of the gate values with respect to the
  mask and the router, the straight-through mask-logit gradient (Eq. 3), and
  the experts' backward through their SwiGLU.

It shares no code with the HIP path and imports nothing from it. Only the
tests, the smoke check and the benchmark's CPU-baseline leg may import it;
the product path never does.

Parity pins: every function here is pinned by the CPU test suite
(brute-force Top-K, closed forms, invariants, library routines,
hand-worked cache traces, finite differences of the forward for the
gradients and exact enumerated inclusion probabilities for the sampler). The fetch counts of synthetic traces at
particular prior strengths have no value printed in the paper to compare
with; they are pinned only through the cache rules above.
"""

from . import cache, ffn, offload, routing, train  # noqa: F401
