"""SAGA-NN message-passing layer for AMD Instinct MI355X (gfx950).

The compute path is libsaga.so (HIP kernels behind the C ABI of
include/saga.h); ``saga`` is its ctypes binding and ``layers`` composes the
workloads' models from it.
"""
__all__ = ["saga", "layers", "build"]
