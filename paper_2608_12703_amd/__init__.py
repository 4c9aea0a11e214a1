"""MI355X-native batched speculative-verify step for single-model ASR speculative decoding.

The verify step scores a drafted block against a paged self-attention KV cache and
precomputed encoder cross-attention K/V, takes the greedy argmax of the tied LM head,
accepts the longest greedy-matching prefix and commits the KV cache (paper: section 3,
"Speculative Loop"; appendix "Real cached loop").

Submodules are imported explicitly so that importing the input generators does not load
the HIP library:

* ``configs`` -- the five workload presets (shapes, draft lengths, acceptance laws).
* ``synth``   -- seeded synthetic inputs (weights, encoder states, KV prefixes, drafts).
* ``ad``      -- ctypes binding over ``libad.so`` (the C-ABI in ``include/ad.h``).
"""
