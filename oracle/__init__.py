"""CPU oracle for RIS sparse attention (prefill hot path and decode step).

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
definition that the GPU library is checked against.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it.  The
product path (the HIP library and its Python binding) never imports, links or
calls anything here, and nothing here imports the product path: the two share
no code, headers, tables or constants.

Modules, in the order the method runs:

* ``philox``   -- Philox4x64-10 (Salmon et al., SC'11), the counter-based hash
                  keyed by (seed) and fed (query, kv-head, layer).
* ``prp``      -- the keyed Feistel permutation (16-bit multiply-xorshift
                  rounds) with cycle walking: an exact-k uniform draw without
                  replacement.
* ``geometry`` -- density -> per-row count, Stochastic and Structural sets,
                  the seed-ensemble union and its CSR (Methods, "Memory-Bounded
                  Geometry Generation" and "Sampling Modes").
* ``rope``     -- RoPE with plain, linear and YaRN frequencies (Methods,
                  "Dynamic RoPE Scaling"; Results, "RoPE Scaling").
* ``attention``-- one softmax over the unified index set (PFUS, Methods,
                  "Hybrid Anchor and Pre-Fusion Unified Softmax") and PV.
* ``decode``   -- the Hybrid-Anchor generation step: frozen stochastic anchor
                  plus sliding local window, merged, one softmax (same passage).
* ``model``    -- a LLaMA / Qwen2 decoder stack around the RIS attention
                  (model-level prefill; Methods, "The RIS Implementation").

Every floating-point step runs in float64.  Readings of the paper where it is
silent or ambiguous are listed in the module that takes them.
"""

from . import philox, prp, geometry, rope, attention, decode, model  # noqa: F401
