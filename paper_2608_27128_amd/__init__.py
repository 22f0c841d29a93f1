"""TwinKV pairwise key redundancy + budget-preserving repair on MI355X (gfx950).

The compute path is the HIP library ``libtwinkv.so`` (C ABI declared in
``include/twinkv.h``); ``paper_2608_27128_amd.binding`` marshals torch device
tensors into it.  ``paper_2608_27128_amd.synth`` generates seeded inputs.
The library is loaded lazily on first use and a missing build raises.
"""
__version__ = "0.1.0"
