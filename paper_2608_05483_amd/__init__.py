"""MI355X-native batched heterogeneous-adapter LoRA apply (PLoRA's hot path).

The product is the C-ABI shared library built from ``csrc/`` (declared in
``include/plora.h``); ``plora`` is its thin Python binding and ``workloads``
draws the seeded synthetic inputs.  Importing this package loads nothing:
``from paper_2608_05483_amd import plora`` loads the HIP library and fails
loudly if it has not been built.
"""
__all__ = ["plora", "workloads", "build"]
