"""Resettable memoroid scans for AMD MI355X (gfx950).

The compute lives in ``libmemoroid.so`` (hand-written HIP, C ABI declared in
``include/memoroid.h``).  ``paper_2402_09900_amd.binding`` marshals torch
tensors into that ABI; ``paper_2402_09900_amd.tapes`` draws seeded synthetic
tapes.  Importing this package does not load the shared library: the first
call into ``binding`` does, and raises if it is missing.
"""
__all__ = ["binding", "tapes"]
