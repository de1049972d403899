"""Baton's re-batched decode step on MI355X: HIP kernels behind a C ABI (libbaton.so).

`baton` is the ctypes binding of include/baton.h; `cache.BatonCache` wraps one
handle together with the device buffers it uses (PyTorch supplies the device
memory and the stream).
"""
