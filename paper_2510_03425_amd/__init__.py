"""MeBP checkpointed LoRA training step for AMD Instinct MI355X (gfx950).

``libmebp.so`` (C ABI, ``include/mebp.h``) holds the whole hot path as hand-written HIP
kernels; ``_lib`` is its ctypes binding (same function names) and ``device`` the torch
plumbing that places inputs in device memory. Importing this package loads nothing;
``_lib.lib()`` loads the library and raises if it has not been built.
"""
__all__ = ["_lib", "device", "build"]
