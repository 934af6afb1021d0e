"""CPU oracle for the ProMoE hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct NumPy (float64) implementations of what the GPU
path computes, written from the paper (ProMoE: Fast MoE-based LLM Serving
using Proactive Caching, arXiv 2410.22134):

* ``router``    -- gate logits, softmax, top-k, renormalised weights
                   (Background, "Mixture-of-Experts (MoE) based LLMs");
* ``predictor`` -- look-ahead predictor logits, per-token top-k, vote
                   (Sec. "Learning-based Predictor", "Stride Prefetching");
* ``ffn``       -- SwiGLU experts and the weighted combine (Background);
* ``cache``     -- the logical per-layer LRU expert cache with speculative and
                   precise plans and reordered inference (Sec. "Coordination of
                   Prefetching and Inference", Alg. 1 and Alg. 2, Sec.
                   "Cache Implementation");
* ``stack``     -- harness ops around the MoE block (RMSNorm, a linear
                   attention surrogate, residual adds);
* ``quant``     -- decoding of group-quantised 4-bit expert weights (the
                   paper's bits-per-weight study): (code - 8) x scale per
                   group of 128 weights of a row;
* ``brute``     -- brute-force checkers used only to pin the oracle itself.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU path
(the seeded input generator in ``synth`` is the only common module, and it
holds none of the method's arithmetic).

Parity pins: every function here is pinned by ``tests/test_oracle_*.py``
against brute force, closed forms, the paper's worked example and invariants.
Parity unpinned: predictor *accuracy* against the paper's trained-predictor
figures, and all physical timing (bytes copied before a purge, stall time) --
those are reported, not parity-checked.
"""
from . import bf16, router, predictor, ffn, cache, stack, brute, quant  # noqa: F401
