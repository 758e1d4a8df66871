"""Sentinel-token context compression (Ren, Jia and Zhu, 2023) on MI355X.

The compute path is the HIP library ``libsckv.so`` (see ``csrc/``); the
Python side only marshals arguments into its C ABI (``binding``).
"""
__all__ = ["workload"]
