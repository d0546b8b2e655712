"""The 5-bit core-left layout ARCHEAD_I5 (the paper's "packed 5-bit" Q5(A_c),
Section 3.2 and the packed state-dictionary table; the layout is this
library's reading): hand-derived golden words, the oracle's and the C++
packer's round trips, byte accounting, and the oracle's dense head built from
5-bit words against the same codes held as int8."""
from __future__ import annotations

import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle.bytes as obytes
from oracle import head as ohead, layout
from paper_2608_02703_amd import archead as ab
from synth import make_head, make_x
from tests.fixtures import GOLDEN


def _golden():
    out = []
    with open(os.path.join(GOLDEN, "int5_layout_v1.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                r, c, w = [t.strip() for t in line.split("|")]
                out.append((int(r), np.array([[int(t) for t in c.split()]]),
                            np.array([[int(t, 16) for t in w.split()]], dtype=np.uint32)))
    return out


@pytest.fixture(scope="module")
def L():
    return ab.lib()


def test_golden_words_oracle_and_library(L):
    cases = _golden()
    assert len(cases) == 4
    for r, codes, words in cases:
        assert np.array_equal(layout.pack_int5(codes), words)
        assert np.array_equal(layout.unpack_int5(words, r), codes)
        assert np.array_equal(ab.pack_int5(codes, L), words)
        assert np.array_equal(ab.unpack_int5(words, r, L), codes)


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 7), st.integers(1, 40), st.integers(0, 2 ** 32 - 1))
def test_library_pack_matches_oracle_unpack(rows, r, seed):
    rng = np.random.default_rng(seed)
    codes = rng.integers(-16, 16, size=(rows, r)).astype(np.int8)
    words = ab.pack_int5(codes)
    assert np.array_equal(layout.unpack_int5(words, r), codes)
    assert np.array_equal(layout.pack_int5(codes), words)
    # every field of random words decodes alike on both sides
    raw = rng.integers(0, 2 ** 30, size=(rows, (r + 5) // 6), dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(ab.unpack_int5(raw, r), layout.unpack_int5(raw, r))


def test_library_pack_rejects_out_of_range(L):
    with pytest.raises(ab.ArcheadError):
        ab.pack_int5(np.full((1, 3), 16, dtype=np.int8), L)
    with pytest.raises(ab.ArcheadError):
        ab.pack_int5(np.full((1, 3), -17, dtype=np.int8), L)
    assert L.archead_pack_int5(None, 1, 6, None) == ab.E_INVALID_ARG


def test_i5_head_equals_int8_head_in_the_oracle():
    """The oracle's dense head from 5-bit words equals, bit for bit, the head
    whose core-left codes are the same values as int8."""
    h5 = make_head("tiny", V=300, d=256, g=64, rc=10, rr=6, core_u="i5")
    assert h5.core_u.dtype == np.uint32 and h5.core_u.shape == (300, 2)
    codes = layout.unpack_int5(h5.core_u, 10)
    assert codes.min() >= -15 and codes.max() <= 15
    import dataclasses
    h8 = dataclasses.replace(h5, core_u=codes.astype(np.int8))
    x = make_x("tiny", 3, d=256, basis="identity")
    assert np.array_equal(ohead.logits(h5, x), ohead.logits(h8, x))
    assert np.array_equal(ohead.logits(h5, x, vocab=[299, 3, 3]), ohead.logits(h8, x)[:, [299, 3, 3]])


@pytest.mark.parametrize("V,d,g,rc,rr", [(151936, 4096, 64, 10, 6), (1000, 256, 64, 7, 5),
                                        (151936, 4096, 128, 64, 32)])
def test_i5_packed_bytes(L, V, d, g, rc, rr):
    desc = ab.Desc.make(V, d, g, rc, rr, core_u_dtype=ab.I5)
    expect = obytes.packed_bytes(V, d, g, rc, rr) - V * rc + V * obytes.i5_row_bytes(rc)
    assert ab.packed_bytes(desc, L) == expect


def test_paper_qwen_storage_with_i5_and_8bit_scales(L):
    """The paper's Qwen3-8B setting (Section 4: r_c = 10, r_r = 6) stored with
    5-bit core-left words and 8-bit residual scale codes.  Table 1 prints
    303.96 MiB.  With one 8-bit scale code per group of 128 weights (the
    storage the table implies) this layout counts 304.35 MiB (+0.13%: the
    fp16 row scales of the scale codes and the two unused bits per word);
    with groups of 64 (the group size Section 4 names) it is 308.98 MiB."""
    Mi = 2 ** 20
    b128 = ab.packed_bytes(ab.Desc.make(151936, 4096, 128, 10, 6, scale_dtype=ab.U8,
                                        core_u_dtype=ab.I5), L)
    b64 = ab.packed_bytes(ab.Desc.make(151936, 4096, 64, 10, 6, scale_dtype=ab.U8,
                                       core_u_dtype=ab.I5), L)
    assert b128 == 319_131_168 and round(b128 / Mi, 2) == 304.35
    assert b64 == 323_993_120 and round(b64 / Mi, 2) == 308.98
    assert abs(b128 / Mi - 303.96) / 303.96 < 0.002
    # the same head with int8 core-left codes: 2 more bytes per row
    b8 = ab.packed_bytes(ab.Desc.make(151936, 4096, 128, 10, 6, scale_dtype=ab.U8), L)
    assert b8 - b128 == 151936 * (10 - 8)
