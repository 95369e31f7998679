"""Plain, slow CPU oracle for the layer-shard training step of arXiv 2411.06465.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it, to check the HIP library against
an independent restatement of the paper's method.  It shares no code with
``paper_2411_06465_amd`` (no kernels, headers, helpers or tables), and it does
not import the seeded input generators either: callers hand it arrays.

Modules
  memory   -- the closed-form byte counts of Sec. 3 (Eqs. 1-18), exact rationals
  layer    -- one GPU's shard of a Llama decoder layer, forward and backward,
              float64 numpy with bf16 rounding at the tensors the layer stores
  lm_head  -- the tensor-parallel LM head with vocabulary-parallel cross-entropy
  ends     -- the vocabulary-parallel embedding and the LM-head block (final
              RMSNorm, linear, FP32 softmax cross-entropy), forward and backward
  optim    -- one Adam step over a shard of the 18-bytes-per-parameter layout
  bf16     -- round-to-nearest-even onto the bfloat16 grid (the oracle's own)
"""
from . import bf16, memory, layer, lm_head, ends, optim  # noqa: F401
