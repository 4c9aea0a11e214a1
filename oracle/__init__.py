"""CPU oracle for the batched speculative-verify step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py``
may import or run anything in this package.  It shares no code with the HIP path (no
kernels, headers, helpers or constants); its inputs come from
``paper_2608_12703_amd.synth``, which draws random numbers and holds none of the
decoder's arithmetic.

What it computes (float64 throughout, written for reading, not speed):

* ``decoder``  -- the Whisper-shape pre-LN decoder, the cross-K/V prefill, one-pass
  verification of a drafted block and plain autoregressive greedy decoding
  (paper: section 3, "Speculative Loop"; appendix "Real cached loop").
* ``accept``   -- the longest greedy-matching prefix and the commit rule.
* ``metrics``  -- survival s_k, conditional acceptance a_k^c and mean accepted length L
  (section 3, "Speculative Loop"; appendix "Acceptance measures").
* ``numerics`` -- storage rounding (bf16 / fp32).
* ``draft``    -- the audio-conditioned draft step (section 3, "Models and Protocol";
  appendix "Draft architecture", "Window geometry").
* ``anchor_loss`` -- the AnchorDraft training objective (section "Correction and Cost",
  paragraph "AnchorDraft Training Objective"; appendix "Training Correction with
  AnchorDraft").
* Tree verification and the verification-attention anchor live in ``decoder``
  (appendix "Tree-decoder implementation check"; section "Correction and Cost",
  paragraph "Verification-Attention Correction").

Pins: every function is checked in ``tests/test_oracle_*.py`` against something other
than itself (library routines, closed forms, brute force, the paper's printed tables).
"""
