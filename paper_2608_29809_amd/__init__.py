"""Region-reuse DiT denoising step (RegionCache) on MI355X.

The compute path is libregioncache.so: hand-written HIP kernels for gfx950
behind the C ABI in include/regioncache.h.  `abi` binds that ABI with ctypes
(argument marshalling only), `runtime` adds device-memory plumbing with
PyTorch, and `schedule` drives multi-turn editing (Eq. 1, Eq. 2) on the
library's verbs.  Importing any of them without the built library raises
ImportError.
"""
__all__ = ["abi", "runtime", "schedule", "build"]
