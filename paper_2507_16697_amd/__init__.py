"""Ring-chunked bidirectional attention for MI355X (gfx950): one GPU's share of a RingX ring.

The compute lives in the HIP library ``libringx.so`` (C ABI declared in ``include/ringx.h``);
``paper_2507_16697_amd.ringx`` is its thin ctypes binding and ``paper_2507_16697_amd.inputs``
the seeded synthetic input generators.  Importing this package loads nothing.
"""
