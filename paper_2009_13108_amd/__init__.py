"""MI355X-native NITI hot path: int8 MFMA contractions with fused block-
exponent pseudo-stochastic rounding, integer loss gradient and update.

The compute runs in the HIP library ``libniti.so`` behind a C ABI
(``include/niti.h``); :mod:`paper_2009_13108_amd.niti` is its ctypes binding.
Importing this package does not load the library; the first call does, and
it raises if the library has not been built.
"""
__all__ = ["niti", "inputs"]
