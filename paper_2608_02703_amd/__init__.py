"""ARCHead packed LM-head forward for AMD Instinct MI355X (gfx950).

The compute path is the C-ABI library libarchead.so (hand-written HIP
kernels); ``archead`` is its thin ctypes binding, with PyTorch providing
device memory and streams only.
"""
from .archead import (  # noqa: F401
    ArcheadError,
    BuildDesc,
    Desc,
    build_head,
    PackedHead,
    logit_fidelity,
    lib,
    pack_int4,
    pack_int5,
    packed_bytes,
    unpack_int4,
    unpack_int5,
    validate_desc,
)
