"""MI355X-native streaming Skip-Convolution layer (Habibian et al., CVPR 2021).

The compute path lives in the HIP library ``libskipconv.so`` (built from
``csrc/``); ``skipconv`` holds the thin ctypes binding. Importing this package
loads nothing; the library is loaded on first use and a missing library is an
error, never a fallback.
"""
__all__ = ["skipconv", "synthetic"]
