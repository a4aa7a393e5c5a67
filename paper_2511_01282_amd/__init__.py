"""MI355X (gfx950) draft-tree verification for retrieval-enhanced speculative decoding.

The product is the C-ABI library ``librespec_verify.so`` (``include/respec_verify.h``),
built from ``csrc/`` by ``build.py``; ``binding`` marshals torch tensors into its
calls.  ``runner`` turns a synthetic workload into device tensors and runs a step.
"""
