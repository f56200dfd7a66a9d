"""kvx: MI355X-native store/load of paged KV state to a pinned host chunk pool.

The product is the HIP library ``libkvx.so`` (C ABI in ``include/kvx.h``);
``paper_2609_15021_amd.kvx`` is its Python binding.  Importing the binding
requires the built library and fails loudly without it.
"""
__all__ = ["kvx"]
