"""CPU oracle of the expert-slot-cache MoE FFN (MawForge, arXiv 2607.09686).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (the HIP library and its Python binding) never
does, and shares no code with it.

What it computes, in plain fp64 numpy, one obviously-correct step at a time:

* GGUF-style Q8_0 / Q4_0 block decoding          (``numerics``, ``quant``)
* router logits, top-k and renormalised softmax   (``router``)
* the per-layer LRU expert-slot table with hit / miss / eviction accounting
  and materialised-byte counters                  (``lru``)
* the SwiGLU expert FFN and the weighted combine  (``ffn``)
* a whole MoE layer call and the residual stack   (``layer``)
* the prefill variant that rounds weights, inputs and activations to bf16
  where the MFMA path does                        (``layer.moe_layer_bf16``)
* the static budget planner: slots per layer from a cache budget and the
  lower bound C + E(p) + K(n) against the serving target   (``planner``)

The paper (its Native Serving Path section) fixes only the mechanism: a fixed
set of slots per layer for the routed experts, filled on a miss, with a map from experts
to slots.  Every finer point (eviction rule, hit granularity, tie-breaks, FFN
form, block formats) is a stated reading; each function names the one it uses.
"""
from . import numerics, quant, router, lru, ffn, layer, planner  # noqa: F401
