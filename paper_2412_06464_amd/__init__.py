"""MI355X-native chunkwise gated delta rule (Gated DeltaNet, arXiv 2412.06464).

The compute path is the C-ABI library ``libgdn.so`` built from ``csrc/``
(hand-written HIP kernels for gfx950).  ``gdn`` is a thin ctypes binding with
the same entry-point names; ``inputs`` holds the seeded synthetic workloads.
Submodules are imported lazily so that the input generator can be used
without loading the HIP library.
"""
__all__ = ["gdn", "inputs"]
