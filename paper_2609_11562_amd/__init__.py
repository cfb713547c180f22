"""MI355X (gfx950) GEMM + tile-reduce: one tensor-parallel rank's share of a
row-parallel GEMM-ReduceScatter with interleaved tile production, per-tile
ready flags and a concurrent reduction kernel on a budget of workgroups.

The compute path lives in the HIP library ``libentwine.so`` (C ABI declared
in ``include/entwine.h``); ``paper_2609_11562_amd.entwine`` is a thin ctypes
binding over it.  Importing this package does not load the library.
"""
