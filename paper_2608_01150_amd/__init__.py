"""Packed whole+shard attention for MI355X (gfx950).

The product is the C-ABI library ``libzl_attn.so`` (header
``include/zl_attn.h``); ``paper_2608_01150_amd.api`` is its thin Python
binding and raises on import if the library is not built.
``paper_2608_01150_amd.workloads`` describes the synthetic batches and draws
their inputs.
"""
