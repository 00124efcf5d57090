"""MI355X (gfx950) batched speculative-verify library.

The compute path is libsdverify.so (HIP kernels + C ABI, include/sd_verify.h);
``sdverify`` binds it with ctypes and ``verifier.Verifier`` marshals torch
device buffers into it.
"""
from . import sdverify  # noqa: F401
