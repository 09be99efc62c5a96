"""Unified, batch-invariant causal GQA attention for MI355X (gfx950).

The HIP library (``libuattn.so``) is loaded lazily by ``paper_2609_35140_amd.uattn``;
importing this package alone touches no GPU.
"""
