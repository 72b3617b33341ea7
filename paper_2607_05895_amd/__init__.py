"""MI355X-native owner-local Muon / AdamW step (MatrixFSDP's per-GPU optimizer work).

The computation lives in ``libmfsdp.so`` (hand-written HIP kernels for gfx950 behind the C ABI in
``include/mfsdp.h``); ``native`` is its ctypes binding.
"""
from . import native  # noqa: F401

__all__ = ["native"]
