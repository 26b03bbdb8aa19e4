"""Grouped (shared-prefix) causal attention for AMD MI355X (gfx950).

The compute lives in the HIP library ``libpg_attn.so`` (C ABI declared in
``include/pg_attn.h``); ``paper_2506_05433_amd.binding`` marshals torch
tensors into it. Importing this package does not load the library, so the
seeded input generator (``paper_2506_05433_amd.inputs``) stays usable on a
machine without a GPU.
"""

__all__ = ["binding", "inputs"]
