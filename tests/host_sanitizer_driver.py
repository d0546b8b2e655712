"""Runs the host-only C ABI (argument checks, byte accounting, INT4 packer)
through a library build given on the command line; used by
test_host_sanitizers.py under AddressSanitizer / UBSan.  Exits non-zero on
any wrong answer."""
from __future__ import annotations

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2608_02703_amd import archead as ab  # noqa: E402


def main(path):
    L = ab.host_lib(path)
    ok = ab.Desc.make(1000, 256, 64, 8, 4)
    assert ab.validate_desc(ok, L) == ab.OK
    bad = [ab.Desc.make(0, 256, 64, 8, 4), ab.Desc.make(1000, 256, 48, 8, 4),
           ab.Desc.make(1000, 288, 64, 8, 4), ab.Desc.make(1000, 256, 64, -1, 4),
           ab.Desc.make(1000, 256, 64, 8, 4, abi=1), ab.Desc.make(1000, 256, 64, 8, 4, enc=2),
           ab.Desc.make(2 ** 31, 256, 64, 8, 4), ab.Desc.make(1000, 32768, 64, 8, 4)]
    for d in bad:
        assert ab.validate_desc(d, L) != ab.OK
        assert L.archead_last_error()
        assert ab.packed_bytes(d, L) == 0
    assert L.archead_validate_desc(None) == ab.E_INVALID_ARG
    assert L.archead_packed_bytes(None) == 0
    assert ab.packed_bytes(ab.Desc.make(151936, 4096, 128, 64, 32), L) == 336_475_840
    assert ab.packed_bytes(ab.Desc.make(151936, 4096, 128, 64, 32, scale_dtype=ab.U8), L) == \
        331_917_760
    rng = np.random.default_rng(1)
    for rows, words in ((1, 1), (3, 7), (17, 64), (2, 513)):
        codes = rng.integers(-8, 8, size=(rows, 8 * words)).astype(np.int8)
        packed = ab.pack_int4(codes, L)
        assert np.array_equal(ab.unpack_int4(packed, 8 * words, L), codes)
    for bad_codes in (np.full((2, 8), 8, np.int8), np.zeros((1, 12), np.int8)):
        try:
            ab.pack_int4(bad_codes, L)
        except ab.ArcheadError:
            pass
        else:
            raise AssertionError("bad codes accepted")
    assert L.archead_pack_int4(None, 1, 8, None) == ab.E_INVALID_ARG
    assert L.archead_unpack_int4(None, 1, 8, None) == ab.E_INVALID_ARG
    for s in range(8):
        assert L.archead_status_str(s)
    print("host ABI under sanitizers: ok", flush=True)


if __name__ == "__main__":
    main(sys.argv[1])
