"""MI355X-native local SGD / post-local SGD hot path.

The compute path is liblsgd.so (HIP kernels for gfx950 behind the C ABI in
include/lsgd.h); ``paper_1808_07217_amd.lsgd`` is its ctypes binding. Import
the binding explicitly; this package initialiser loads nothing.
"""
__all__ = ["lsgd", "build"]
