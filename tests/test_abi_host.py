"""CPU tests of the C-ABI library: exports, argument checks, byte accounting
and the host INT4 packer (checked against the oracle's own unpacker).  No
compute call is made, so no GPU is needed."""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle.bytes as obytes
from oracle import layout
from paper_2608_02703_amd import archead as ab
from synth import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "archead.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(archead_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return ab.lib()


def test_library_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(ab._SIGS), "binding and header disagree"


def test_status_strings(L):
    for s in range(6):
        assert L.archead_status_str(s)
    assert L.archead_status_str(99) == b"unknown status"


def _desc(**kw):
    base = dict(V=1000, d=256, g=64, rc=8, rr=4)
    base.update(kw)
    extra = {k: base.pop(k) for k in ("gV", "gB", "abi", "enc", "scale_dtype",
                                       "factor_dtype", "core_u_dtype") if k in base}
    return ab.Desc.make(base["V"], base["d"], base["g"], base["rc"], base["rr"],
                        **extra)


@pytest.mark.parametrize("kw,status", [
    ({}, ab.OK),
    (dict(abi=1), ab.E_INVALID_ARG),           # another ABI version
    (dict(abi=4), ab.E_INVALID_ARG),
    (dict(abi=2), ab.E_INVALID_ARG),           # before the core_u_dtype field
    (dict(core_u_dtype=ab.I5), ab.OK),
    (dict(core_u_dtype=ab.BF16), ab.E_UNSUPPORTED),
    (dict(scale_dtype=ab.U8), ab.OK),          # 8-bit group scale codes
    (dict(V=0), ab.E_INVALID_ARG),
    (dict(d=0), ab.E_INVALID_ARG),
    (dict(g=48), ab.E_INVALID_ARG),            # not a multiple of 32
    (dict(d=320, g=64, gV=64, gB=64), ab.OK),
    (dict(d=288, g=64), ab.E_INVALID_ARG),     # g does not divide d
    (dict(rc=-1), ab.E_INVALID_ARG),
    (dict(gV=96), ab.E_INVALID_ARG),           # does not divide d
    (dict(gB=16), ab.E_INVALID_ARG),           # not a multiple of 32
    (dict(rc=0, gV=0), ab.OK),                 # absent component: group ignored
    (dict(enc=2), ab.E_INVALID_ARG),
    (dict(scale_dtype=ab.BF16), ab.E_UNSUPPORTED),
    (dict(factor_dtype=ab.I32), ab.E_UNSUPPORTED),
    (dict(rc=1000, rr=100), ab.E_UNSUPPORTED),
    (dict(V=2 ** 31), ab.E_UNSUPPORTED),
    (dict(d=32768, g=64), ab.E_UNSUPPORTED),
])
def test_validate_desc(L, kw, status):
    st_ = ab.validate_desc(_desc(**kw), L)
    assert st_ == status, L.archead_last_error()
    if status != ab.OK:
        assert L.archead_last_error()
        assert ab.packed_bytes(_desc(**kw), L) == 0


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_packed_bytes_matches_oracle_on_configs(L, name):
    c = CONFIGS[name]
    d = ab.Desc.make(c["V"], c["d"], c["g"], c["rc"], c["rr"])
    assert ab.packed_bytes(d, L) == obytes.packed_bytes(c["V"], c["d"], c["g"],
                                                        c["rc"], c["rr"])


@settings(max_examples=80, deadline=None)
@given(st.integers(1, 300000), st.integers(1, 64), st.sampled_from([32, 64, 128]),
       st.integers(0, 200), st.integers(0, 200), st.integers(1, 4), st.integers(1, 4))
def test_packed_bytes_matches_oracle(V, dmul, g, rc, rr, fv, fb):
    L = ab.lib()
    d = g * dmul
    gV = d // fv if (d // fv) % 32 == 0 and d % fv == 0 else d
    gB = d // fb if (d // fb) % 32 == 0 and d % fb == 0 else d
    desc = ab.Desc.make(V, d, g, rc, rr, gV, gB)
    assert ab.packed_bytes(desc, L) == obytes.packed_bytes(V, d, g, rc, rr, gV, gB)


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 9), st.integers(1, 40), st.integers(0, 2 ** 32 - 1))
def test_cpp_pack_matches_oracle_unpack(rows, words, seed):
    L = ab.lib()
    rng = np.random.default_rng(seed)
    codes = rng.integers(-8, 8, size=(rows, 8 * words)).astype(np.int8)
    packed = ab.pack_int4(codes, L)
    assert np.array_equal(layout.unpack_int4(packed, 8 * words), codes)
    raw = rng.integers(0, 256, size=(rows, 4 * words), dtype=np.uint8)
    assert np.array_equal(ab.unpack_int4(raw, 8 * words, L),
                          layout.unpack_int4(raw, 8 * words))


def test_cpp_pack_golden_words(L):
    from tests import fixtures
    for b, c in fixtures.layout_cases():
        assert ab.pack_int4(c.reshape(1, 8), L).tolist() == [b.tolist()]
        assert ab.unpack_int4(b.reshape(1, 4), 8, L).tolist() == [c.tolist()]


def test_cpp_pack_rejects_bad_input(L):
    with pytest.raises(ab.ArcheadError) as e:
        ab.pack_int4(np.full((2, 8), 8, dtype=np.int8), L)
    assert e.value.status == ab.E_INVALID_ARG
    assert b"out of [-8, 7]" in L.archead_last_error()
    with pytest.raises(ab.ArcheadError):
        ab.pack_int4(np.zeros((1, 12), dtype=np.int8), L)   # d % 8 != 0
    assert L.archead_pack_int4(None, 1, 8, None) == ab.E_INVALID_ARG


def test_create_checks_arguments_before_touching_the_device(L):
    desc = _desc()
    h = ctypes.c_void_p(123)
    # missing residual pointers
    ptrs = ab.Ptrs()
    assert L.archead_create(ctypes.byref(desc), ctypes.byref(ptrs),
                            ctypes.byref(h)) == ab.E_INVALID_ARG
    assert h.value is None
    # r_c > 0 without core pointers
    ptrs = ab.Ptrs(res_codes=4096, res_scales=4096)
    assert L.archead_create(ctypes.byref(desc), ctypes.byref(ptrs),
                            ctypes.byref(h)) == ab.E_INVALID_ARG
    # misaligned codes
    full = ab.Ptrs(*([4096] * 10))
    full.res_codes = 4100
    assert L.archead_create(ctypes.byref(desc), ctypes.byref(full),
                            ctypes.byref(h)) == ab.E_MISALIGNED
    full = ab.Ptrs(*([4096] * 10))
    full.core_u_scale = 4097
    assert L.archead_create(ctypes.byref(desc), ctypes.byref(full),
                            ctypes.byref(h)) == ab.E_MISALIGNED
    bad = _desc(abi=7)
    assert L.archead_create(ctypes.byref(bad), ctypes.byref(full),
                            ctypes.byref(h)) == ab.E_INVALID_ARG
    assert L.archead_create(ctypes.byref(desc), ctypes.byref(full), None) == \
        ab.E_INVALID_ARG


def test_null_handle_calls(L):
    assert L.archead_workspace_bytes(None, 4, ab.OP_LOGITS) == 0
    assert L.archead_logits(None, None, 1, 8, None, ab.F32, 8, None, 0, None) == \
        ab.E_INVALID_ARG
    assert L.archead_logits_ce(None, None, 1, 8, None, ab.I32, None, None, None, 0,
                               None) == ab.E_INVALID_ARG
    assert L.archead_logits_topk(None, None, 1, 8, 5, None, None, 5, None, 0, None) == \
        ab.E_INVALID_ARG
    assert L.archead_workspace_bytes(None, 4, ab.OP_TOPK) == 0
    assert L.archead_set_gemv_max_m(None, 3) == ab.E_INVALID_ARG
    assert L.archead_get_gemv_max_m(None) == -1
    assert L.archead_prepared_bytes(None) == 0
    assert L.archead_prepare(None, None, 0, None) == ab.E_INVALID_ARG
    assert L.archead_set_mid_range(None, 2, 3) == ab.E_INVALID_ARG
    assert L.archead_get_mid_range(None, ctypes.byref(ctypes.c_int64()),
                                   ctypes.byref(ctypes.c_int64())) == ab.E_INVALID_ARG
    assert L.archead_set_dec_range(None, 2, 3) == ab.E_INVALID_ARG
    lo, hi = ctypes.c_int64(), ctypes.c_int64()
    assert L.archead_get_dec_range(None, ctypes.byref(lo), ctypes.byref(hi)) == ab.E_INVALID_ARG
    assert L.archead_set_launch(None, ab.LAUNCH_GEMV_GRID, 4) == ab.E_INVALID_ARG
    assert L.archead_get_launch(None, ab.LAUNCH_GEMV_GRID, ctypes.byref(lo)) == ab.E_INVALID_ARG
    L.archead_destroy(None)


def test_launch_knob_numbers_match_header():
    found = dict(re.findall(r"#define (ARCHEAD_LAUNCH_[A-Z0-9_]+) (\d+)", open(HEADER).read()))
    assert int(found.pop("ARCHEAD_LAUNCH_KNOBS")) == 7
    assert len(found) == 7
    for name, v in found.items():
        assert getattr(ab, name[len("ARCHEAD_"):]) == int(v), name


def test_host_only_build_agrees(tmp_path):
    """The same host translation unit built with g++ (no HIP) gives the same
    answers (it is what the sanitizer build runs)."""
    from paper_2608_02703_amd import build
    path = build.build_host()
    H = ab.host_lib(path)
    desc = _desc()
    assert ab.validate_desc(desc, H) == ab.OK
    assert ab.packed_bytes(desc, H) == ab.packed_bytes(desc, ab.lib())
    codes = np.random.default_rng(0).integers(-8, 8, size=(3, 64)).astype(np.int8)
    assert np.array_equal(ab.pack_int4(codes, H), ab.pack_int4(codes, ab.lib()))


@pytest.mark.parametrize("V,d,g,rc,rr", [(151936, 4096, 128, 64, 32), (1000, 512, 64, 0, 0),
                                        (8191, 2560, 128, 16, 0)])
def test_packed_bytes_with_8bit_scales(L, V, d, g, rc, rr):
    """8-bit residual scale codes: one byte per group plus an fp16 scale per
    row, as the oracle counts them; at the Qwen shape the head shrinks from
    336,475,840 to 331,917,760 bytes."""
    desc = ab.Desc.make(V, d, g, rc, rr, scale_dtype=ab.U8)
    got = ab.packed_bytes(desc, L)
    assert got == obytes.packed_bytes(V, d, g, rc, rr, res_scale_bits=8, res_row_scale_bytes=2)
    if (V, d, g, rc, rr) == (151936, 4096, 128, 64, 32):
        assert got == 336_475_840 - V * (d // g) * 2 + V * (d // g) + 2 * V == 331_917_760



@pytest.mark.parametrize("M,V,ld_r,ld_t,null,shift,ws,status", [
    (0, 10, 10, 10, False, 0, 1 << 20, ab.OK),                # empty: no launch
    (-1, 10, 10, 10, False, 0, 1 << 20, ab.E_INVALID_ARG),
    (65536, 10, 10, 10, False, 0, 1 << 30, ab.E_INVALID_ARG),
    (2, 0, 10, 10, False, 0, 1 << 20, ab.E_INVALID_ARG),
    (2, 2 ** 31, 2 ** 31, 2 ** 31, False, 0, 1 << 20, ab.E_INVALID_ARG),
    (2, 10, 9, 10, False, 0, 1 << 20, ab.E_INVALID_ARG),      # ld < V
    (2, 10, 10, 9, False, 0, 1 << 20, ab.E_INVALID_ARG),
    (2, 10, 10, 10, True, 0, 1 << 20, ab.E_INVALID_ARG),      # null output
    (2, 10, 10, 10, False, 2, 1 << 20, ab.E_MISALIGNED),      # fp32 buffer off by 2 bytes
    (2, 10, 10, 10, False, 0, 16, ab.E_WORKSPACE),            # short workspace
])
def test_logit_fidelity_argument_checks(L, M, V, ld_r, ld_t, null, shift, ws, status):
    """archead_logit_fidelity rejects bad shapes, pointers and workspaces
    before any HIP call (the pointers here are never dereferenced)."""
    p = 1 << 20
    args = [p + shift, ld_r, p, ld_t, M, V, p, p, 0 if null else p, p, p, ws, None]
    assert L.archead_logit_fidelity(*args) == status, L.archead_last_error()


def test_fidelity_workspace_bytes(L):
    """Per-chunk partials of 48 bytes for every 8192 logits of a row, then a
    256-aligned fp32 per position; 0 for an invalid shape."""
    assert L.archead_fidelity_workspace_bytes(0, 10) == 0
    assert L.archead_fidelity_workspace_bytes(3, 0) == 0
    assert L.archead_fidelity_workspace_bytes(1, 1) == 256 + 4
    assert L.archead_fidelity_workspace_bytes(2, 151936) == 2048 + 8   # 2 x 19 x 48 = 1824 -> 2048


def _bdesc(**kw):
    base = dict(V=1000, d=256, N=512, g=64, r_c=8, r_r=4, g_b=256, p=0.75, lam=1e-3,
                oversample=8, power_iters=2)
    base.update(kw)
    abi = base.pop("abi", ab.ABI_VERSION)
    return ab.BuildDesc(abi, base["V"], base["d"], base["N"], base["g"], base["r_c"],
                        base["r_r"], base["g_b"], base["p"], base["lam"], base["oversample"],
                        base["power_iters"])


@pytest.mark.parametrize("kw,ok", [({}, True), (dict(abi=1), False), (dict(g=48), False),
                                   (dict(d=288), False), (dict(r_c=-1), False),
                                   (dict(g_b=100), False), (dict(r_r=0, g_b=0), True),
                                   (dict(r_r=250, oversample=8), False), (dict(N=0), False),
                                   (dict(lam=-1.0), False), (dict(d=65536, g=64), False)])
def test_build_workspace_bytes(L, kw, ok):
    """archead_build_workspace_bytes: positive for a valid construction
    descriptor (at least the two fp64 V x d buffers and H), 0 otherwise."""
    n = L.archead_build_workspace_bytes(ctypes.byref(_bdesc(**kw)))
    if ok:
        b = _bdesc(**kw)
        assert n >= 2 * 8 * b.V * b.d + 8 * b.N * b.d
    else:
        assert n == 0


def test_build_head_argument_checks_before_any_device_call(L):
    """archead_build_head rejects bad arguments on the host (the pointers
    here are never dereferenced)."""
    b = _bdesc()
    need = L.archead_build_workspace_bytes(ctypes.byref(b))
    p = 1 << 20
    full = ab.Ptrs(*([p] * 10 + [0]))
    ptrs = ctypes.byref(full)

    def call(desc=b, W=p, ldw=256, H=p, ldh=256, om=p, out=ptrs, ws=p, n=need):
        return L.archead_build_head(ctypes.byref(desc) if desc is not None else None, W, ldw, H,
                                    ldh, om, out, None, None, ws, n, None)
    assert call(desc=None) == ab.E_INVALID_ARG
    assert call(desc=_bdesc(g=48)) == ab.E_INVALID_ARG
    assert call(W=None) == ab.E_INVALID_ARG
    assert call(ldw=255) == ab.E_INVALID_ARG
    assert call(ldh=100) == ab.E_INVALID_ARG
    assert call(om=None) == ab.E_INVALID_ARG                     # r_r > 0 needs a sketch
    no_core = ab.Ptrs(*([p] * 2 + [0] * 8 + [0]))
    assert call(out=ctypes.byref(no_core)) == ab.E_INVALID_ARG   # r_c > 0 needs its buffers
    assert call(ws=p + 64) == ab.E_MISALIGNED
    assert call(n=need - 1) == ab.E_WORKSPACE
    assert L.archead_last_error()
