"""MI355X-native fused mini-batch SGD for the d-h-1 ReLU/MSE network.

The compute path is the HIP library ``libmlp.so`` (C ABI in include/mlp.h);
``paper_2606_30497_amd.mlp`` is its thin ctypes binding. Importing this package
does not load the library; the first call into the binding does, and fails
loudly if it is missing.
"""
__all__ = ["mlp", "build"]
