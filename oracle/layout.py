"""Packed INT4 layout and floating-point bit decoding (oracle side).

Layout ARCHEAD_INT4_V1 (the paper leaves exact tensor layouts to the
implementation, Appendix "Packed Buffers and Model-Conversion Lifecycle"):

* the residual codes of row v occupy d/2 bytes, rows back to back;
* bytes 4w..4w+3 of a row, read as a little-endian 32-bit word q, hold the
  eight elements 8w..8w+7 of that row;
* element 8w+2k (k = 0..3) is the nibble in bits [4k, 4k+4) of q and element
  8w+2k+1 the nibble in bits [16+4k, 20+4k);
* a stored nibble u encodes the signed INT4 code c = u - 8, so c spans the
  full signed range [-8, 7] (the paper's residual is signed INT4, Eq. for W_d
  in Section 3.2).

This file is written from that description alone; the HIP library has its own
reader.
"""
from __future__ import annotations

import numpy as np


def unpack_int4(packed: np.ndarray, d: int) -> np.ndarray:
    """uint8 [R, d/2] -> int8 codes [R, d] in [-8, 7]."""
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    if d % 8:
        raise ValueError("d must be a multiple of 8 (whole 32-bit words)")
    R = packed.shape[0]
    if packed.shape != (R, d // 2):
        raise ValueError(f"packed shape {packed.shape} != ({R}, {d // 2})")
    q = packed.view("<u4").astype(np.int64)            # [R, d/8] words
    out = np.empty((R, d // 8, 8), dtype=np.int8)
    for k in range(4):
        out[:, :, 2 * k] = ((q >> (4 * k)) & 0xF) - 8
        out[:, :, 2 * k + 1] = ((q >> (16 + 4 * k)) & 0xF) - 8
    return out.reshape(R, d)


def pack_int4(codes: np.ndarray) -> np.ndarray:
    """int codes [R, d] in [-8, 7] -> uint8 [R, d/2] (inverse of unpack)."""
    codes = np.asarray(codes)
    R, d = codes.shape
    if d % 8:
        raise ValueError("d must be a multiple of 8 (whole 32-bit words)")
    if codes.min(initial=0) < -8 or codes.max(initial=0) > 7:
        raise ValueError("INT4 codes must lie in [-8, 7]")
    u = (codes.astype(np.int64) + 8).reshape(R, d // 8, 8)
    q = np.zeros((R, d // 8), dtype=np.int64)
    for k in range(4):
        q |= u[:, :, 2 * k] << (4 * k)
        q |= u[:, :, 2 * k + 1] << (16 + 4 * k)
    return q.astype("<u4").view(np.uint8).reshape(R, d // 2)


def unpack_int5(words: np.ndarray, r: int) -> np.ndarray:
    """ARCHEAD_I5 words uint32 [R, ceil(r/6)] -> int8 codes [R, r].

    Layout (the library's reading of the paper's "packed 5-bit" core-left
    factor): code k of a row sits in word k // 6 at bits [5 (k % 6),
    5 (k % 6) + 5) as a 5-bit two's complement value in [-16, 15]."""
    words = np.ascontiguousarray(words, dtype=np.uint32)
    R = words.shape[0]
    if r < 1 or words.shape != (R, (r + 5) // 6):
        raise ValueError(f"words shape {words.shape} != ({R}, {(r + 5) // 6})")
    out = np.empty((R, r), dtype=np.int8)
    for k in range(r):
        f = (words[:, k // 6].astype(np.int64) >> (5 * (k % 6))) & 31
        out[:, k] = np.where(f >= 16, f - 32, f)
    return out


def pack_int5(codes: np.ndarray) -> np.ndarray:
    """int codes [R, r] in [-16, 15] -> ARCHEAD_I5 words uint32 [R, ceil(r/6)]
    (inverse of unpack_int5; unused bits zero)."""
    codes = np.asarray(codes, dtype=np.int64)
    R, r = codes.shape
    if codes.min(initial=0) < -16 or codes.max(initial=0) > 15:
        raise ValueError("5-bit codes must lie in [-16, 15]")
    w = np.zeros((R, (r + 5) // 6), dtype=np.int64)
    for k in range(r):
        w[:, k // 6] |= (codes[:, k] & 31) << (5 * (k % 6))
    return w.astype(np.uint32)


def fp16_to_f64(a) -> np.ndarray:
    """fp16 values (float16 array or uint16 bit patterns) -> float64, exact."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.float16)
    if a.dtype != np.float16:
        raise TypeError(f"expected float16 data, got {a.dtype}")
    return a.astype(np.float64)


def bf16_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exact (a bf16 is the top half of
    an IEEE single)."""
    bits = np.asarray(bits)
    if bits.dtype != np.uint16:
        raise TypeError(f"expected uint16 bf16 bit patterns, got {bits.dtype}")
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32) \
        .astype(np.float64)
