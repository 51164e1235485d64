"""MI355X-native collective copy/reduce kernels with XCD-aware placement.

The compute path is the HIP library ``libnuna.so`` (C ABI declared in
``include/nuna.h``).  ``paper_2608_00867_amd.nuna`` is the thin ctypes binding
over it; importing this package loads nothing, so host-only modules such as
``workloads`` can be imported on machines without the library.
"""
__all__ = ["nuna", "workloads"]
