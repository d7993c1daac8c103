"""Relaxed online long convolution (Flash Inference mixer path) on AMD MI355X.

The computation runs in the HIP library ``liblcsm.so`` (C ABI in
``include/lcsm.h``); :mod:`paper_2410_12982_amd.lcsm` is its Python binding.
"""
__all__ = ["lcsm"]
