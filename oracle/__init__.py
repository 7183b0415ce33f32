"""CPU oracle for the self-speculative draft-verify step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import or run anything in this package;
the product path (the HIP library and its Python binding) never does.

Plain, slow, float64 numpy written from the paper's definitions:

* ``attention``  block-causal (hybrid) masked softmax attention over a paged KV
  cache (Preliminaries, "Block Diffusion"; Method, "Joint AR-Diffusion
  Training"; appendix "Self-Speculative Decoding and KV-Cache Update",
  items Draft forward / Verify forward).
* ``decode``     top-1 selection, greedy longest-prefix acceptance, commit and
  KV rollback with a deterministic page allocator (Method, "Self-Speculative
  Decoding"; appendix items Accept / Cache update / Next round).
* ``model``      a random-init pre-norm decoder (layers the paper does not
  specify are read as documented in ``model``), greedy AR decoding
  (Preliminaries, eq. ``eq:ar``) and fused self-speculative decoding, whose
  committed streams must coincide (appendix "AR-Equivalence and Equality
  Testing", Argument), the paper's two-forward round, and direct
  block-diffusion decoding (appendix "Direct Block-Diffusion Decoding":
  confidence-threshold reveal, cache-write forward, block commit).

It shares no code with the HIP path and imports nothing from it.  Inputs come
from the seeded generators, passed in as arrays.
"""
