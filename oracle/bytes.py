"""Persistent-byte accounting of a packed head (oracle side).

The paper measures a packed head's persistent size as the sum, over every
registered buffer, of its element count times its element size (Section 3.3,
equation for bytes(ARCHead); Appendix "Persistent storage versus working
memory").  The dense head it replaces is V * D * 2 bytes (BF16).

``packed_bytes`` applies that sum to the buffers of a head.  The defaults are
the buffers this library stores (INT4 residual bytes, fp16 scales, INT8
factors with fp16 scales); the keyword widths describe the storage variants
the paper's tables use (5-bit core-left codes, 8-bit residual scales), so the
printed storage ratios can be checked against the same formula.
"""
from __future__ import annotations

import math


def _bits_to_bytes(n_elems: int, bits: int) -> int:
    return math.ceil(n_elems * bits / 8)


def packed_bytes(V: int, d: int, g: int, rc: int, rr: int, gV: int = None,
                 gB: int = None, *, res_bits: int = 4,
                 res_scale_bits: int = 16, core_u_bits: int = 8,
                 core_v_bits: int = 8, corr_bits: int = 8,
                 factor_scale_bytes: int = 2, res_row_scale_bytes: int = 0) -> int:
    """Sum of numel x element size over the registered buffers
    (res_row_scale_bytes: per-row scale of 8-bit residual scale codes)."""
    gV = d if gV is None else gV
    gB = d if gB is None else gB
    buffers = [
        _bits_to_bytes(V * d, res_bits),            # residual codes
        _bits_to_bytes(V * (d // g), res_scale_bits),  # residual scales
        V * res_row_scale_bytes,                    # their row scales (8-bit codes)
    ]
    if rc:
        buffers += [
            _bits_to_bytes(V * rc, core_u_bits),     # core left codes
            V * factor_scale_bytes,                  # core left row scales
            _bits_to_bytes(rc * d, core_v_bits),     # core right codes
            rc * (d // gV) * factor_scale_bytes,     # core right scales
        ]
    if rr:
        buffers += [
            _bits_to_bytes(V * rr, corr_bits),       # correction left codes
            V * factor_scale_bytes,                  # correction left scales
            _bits_to_bytes(rr * d, corr_bits),       # correction right codes
            rr * (d // gB) * factor_scale_bytes,     # correction right scales
        ]
    return sum(buffers)


def dense_bf16_bytes(V: int, d: int) -> int:
    return V * d * 2


def i5_row_bytes(rc: int) -> int:
    """Bytes per row of 5-bit codes packed six per 32-bit word."""
    return 4 * ((rc + 5) // 6)


def head_bytes(h) -> int:
    """packed_bytes of a head object carrying the shape attributes and
    buffers (8-bit residual scale codes and 5-bit core-left words are
    recognised by their array types)."""
    kw = {}
    if getattr(h, "res_scales", None) is not None and h.res_scales.dtype == "uint8":
        kw.update(res_scale_bits=8, res_row_scale_bytes=2)
    b = packed_bytes(h.V, h.d, h.g, h.rc, h.rr, h.gV, h.gB, **kw)
    cu = getattr(h, "core_u", None)
    if h.rc and cu is not None and cu.dtype == "uint32":
        b += h.V * i5_row_bytes(h.rc) - h.V * h.rc   # words instead of one byte per code
    return b
