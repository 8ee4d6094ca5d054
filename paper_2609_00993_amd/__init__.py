"""libmoepd: one GPU's share of a phase-owned MoE expert layer on MI355X (gfx950).

The compute path is the HIP library ``libmoepd.so`` (C ABI in
``include/moepd.h``); :mod:`paper_2609_00993_amd.moepd` is its ctypes binding.
"""

__all__ = ["moepd"]
