"""Plain CPU oracle for the ADT-Tree draft-then-verify step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or link
anything under ``oracle/``: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library; both take their inputs from the ``synth`` generators.

Everything is NumPy in float64, slow and written to be checked by eye against
the paper (arXiv 2512.21857).  For bf16 model configurations the oracle rounds to
the nearest bfloat16 value exactly where such a model stores bf16 tensors (norm
outputs, rotated Q and cached K/V, attention output, SwiGLU product, features);
residual stream, logits and scores stay float64.

Modules:
  numerics  -- bf16 rounding, RMSNorm, RoPE, SiLU, Philox4x32-10
  tree      -- ancestor sets and packed ancestor bitmasks of a parent array
  attention -- tree attention over an explicit key set per node
  model     -- target transformer and EAGLE-style draft head, row by row
  schedule  -- adjacent initialisation + bisectional adaptation (Sec. 4.1, 4.2, Eq. 2)
  expand    -- EAGLE-2 dynamic expansion and top-N rerank (Sec. 3.1, Sec. 4.2, Eq. 3-5)
  accept    -- greedy, exact and relaxed acceptance along the tree (Sec. 3.1, Eq. 1)
  decode    -- prefill, the per-cycle step, KV compaction, and the plain AR reference
"""
