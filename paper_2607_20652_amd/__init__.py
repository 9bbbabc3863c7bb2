"""MI355X-native Deep Parity Bottleneck (DPB): encode, decode, decode-backward.

The compute lives in `libdpb.so` (hand-written HIP kernels for gfx950 behind a
C ABI declared in `include/dpb.h`); `binding.py` marshals torch tensors into
that ABI.  Importing this package does not load the library; the first call
that needs it does, and fails loudly if it has not been built.
"""
from __future__ import annotations

__all__ = ["Plan", "encode", "decode", "decode_bwd", "forward", "lib_path"]


def __getattr__(name):
    if name in ("Plan", "encode", "decode", "decode_bwd", "forward", "lib_path", "DPBError"):
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
