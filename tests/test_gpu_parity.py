"""GPU parity of the HIP path against the fp64 CPU oracle (through the C ABI).

Tolerances: fp32 logits max |d| <= 2e-3 (1 + |logit|); CE max |d| <= 1e-4
nats per token; bf16 logits within one bf16 step of RNE(oracle); integer
probes and the hand-derived worked example bit-exact; argmax equal on every
token whose oracle top-2 gap exceeds twice the logit tolerance.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import head as ohead
from synth import CONFIGS, make_head, make_targets, make_x
from tests import fixtures
from tests.gpu_util import (argmax_agreement, assert_bf16_output, assert_ce_close,
                            assert_logits_close, cached_head, cached_oracle_logits, say,
                            torch_x)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


_heads = {}


def packed(cfg, **over):
    from paper_2608_02703_amd import PackedHead
    key = (cfg, tuple(sorted(over.items())))
    if key not in _heads:
        if len(_heads) > 2:
            for k in list(_heads)[:-1]:
                _heads.pop(k).close()
        h = cached_head(cfg, **over) if over else cached_head(cfg)
        _heads[key] = PackedHead.from_arrays(h)
    return _heads[key]


def gpu_logits(ph, x_bits, out_dtype=None, **kw):
    lg = ph.logits(torch_x(x_bits, **kw), out_dtype=out_dtype)
    torch.cuda.synchronize()
    if lg.dtype == torch.bfloat16:
        return lg.view(torch.int16).cpu().numpy().view(np.uint16)
    return lg.cpu().numpy()


def gpu_ce(ph, x_bits, y, dtype=None):
    t = torch.from_numpy(np.asarray(y)).to("cuda")
    if dtype is not None:
        t = t.to(dtype)
    ce, mean = ph.logits_ce(torch_x(x_bits), t)
    torch.cuda.synchronize()
    return ce.cpu().numpy(), float(mean.cpu().numpy()[0])


# ------------------------------------------------------------- exact probes

def test_worked_example_exact():
    from paper_2608_02703_amd import PackedHead
    h, x, expect, y = fixtures.worked_head()
    say("worked example V=2 d=64 g=32 rc=1 rr=1 M=3")
    ph = PackedHead.from_arrays(h)
    lg = gpu_logits(ph, x)
    assert np.array_equal(lg.astype(np.float64), expect), lg
    ce, mean = gpu_ce(ph, x, y)
    ref = ohead.cross_entropy(expect, y)
    assert_ce_close(ce, ref, 1e-6, "worked example CE")
    assert abs(mean - ref.mean()) < 1e-6
    ph.close()


def assert_scale_chain_exact(lg, ref, h):
    """One-hot x makes every logit a single product s * c.  The many-token
    kernel carries its accumulator in units of the current group's scale, so
    such a logit is c times a chain of fp32 scale ratios and one final scale:
    at most 2 * (number of scale slots) roundings of 2^-24 each, relative.
    A misplaced code or scale would be off by O(1).  Where the oracle is 0
    (a zero code, or a zero scale, which the kernel replaces by 2^-60) the
    result must vanish to below 1e-12."""
    nslot = h.d // h.g + (h.rc > 0) + (h.rr > 0)
    bound = 2 * nslot * 2.0 ** -24 * 1.01
    lg = lg.astype(np.float64)
    z = ref == 0
    assert np.abs(lg[z]).max(initial=0) < 1e-12, "nonzero where the oracle is 0"
    rel = np.where(z, 0.0, np.abs(lg - ref) / np.where(z, 1.0, np.abs(ref)))
    worst = np.unravel_index(np.argmax(rel), rel.shape)
    assert rel.max() <= bound, (f"rel err {rel.max():.3e} > {bound:.3e} at {worst}: "
                                f"gpu {lg[worst]!r} oracle {ref[worst]!r}")
    return float(rel.max())


def test_identity_probe_tiny():
    h = make_head("tiny", rc=0, rr=0)
    from paper_2608_02703_amd import PackedHead
    ph = PackedHead.from_arrays(h)
    eye = np.zeros((h.d, h.d), dtype=np.uint16)
    eye[np.arange(h.d), np.arange(h.d)] = 0x3F80
    say("identity probe tiny: M=512 V=8192 (many-token kernel)")
    lg = gpu_logits(ph, eye)
    ref = ohead.logits(h, eye)
    say(f"  max rel err {assert_scale_chain_exact(lg, ref, h):.2e}")
    ph.close()


def test_identity_probe_qwen_sampled():
    h = make_head("qwen_decode", rc=0, rr=0)
    from paper_2608_02703_amd import PackedHead
    ph = PackedHead.from_arrays(h)
    rng = np.random.default_rng(5)
    cols = np.unique(np.concatenate([[0, 1, 7, 8, 31, 32, 127, 128, 2047, 4095],
                                     rng.integers(0, h.d, 54)]))
    x = np.zeros((cols.size, h.d), dtype=np.uint16)
    x[np.arange(cols.size), cols] = 0x3F80
    say(f"identity probe qwen: M={cols.size} V={h.V} (many-token kernel)")
    lg = gpu_logits(ph, x)
    ref = ohead.logits(h, x)
    say(f"  max rel err {assert_scale_chain_exact(lg, ref, h):.2e}")
    ph.close()


# ------------------------------------------------------------- random x

LOGIT_CASES = [("tiny", 1), ("tiny", 8), ("qwen_decode", 1), ("qwen_decode", 4),
               ("qwen_decode", 16), ("gemma", 1), ("gemma", 8), ("gemma", 64)]


@pytest.mark.parametrize("cfg,M", LOGIT_CASES)
def test_logits_parity(cfg, M):
    Mmax = max(CONFIGS[cfg]["Ms"])
    say(f"logits parity {cfg} M={M}")
    ref = cached_oracle_logits(cfg, Mmax)[:M]
    ph = packed(cfg)
    x = make_x(cfg, Mmax)[:M]
    lg = gpu_logits(ph, x)
    err = assert_logits_close(lg, ref, what=f"{cfg} M={M}")
    say(f"  max rel err {err:.2e}")
    if cfg == "gemma":
        n, excl = argmax_agreement(lg, ref)
        say(f"  argmax equal on {n} tokens ({excl} near-ties excluded)")


@pytest.mark.parametrize("cfg,M", [("tiny", 8), ("qwen_decode", 4)])
def test_bf16_logits(cfg, M):
    Mmax = max(CONFIGS[cfg]["Ms"])
    ref = cached_oracle_logits(cfg, Mmax)[:M]
    x = make_x(cfg, Mmax)[:M]
    bits = gpu_logits(packed(cfg), x, out_dtype=torch.bfloat16)
    f32 = gpu_logits(packed(cfg), x)
    assert_logits_close(f32, ref, what=f"{cfg} M={M} fp32")
    assert_bf16_output(bits, f32, ref, f"{cfg} M={M} bf16")


# ------------------------------------------------------------- CE

def test_ce_parity_tiny():
    cfg = "tiny"
    ref_lg = cached_oracle_logits(cfg, 8)
    y = make_targets(cfg, 8)
    ce, mean = gpu_ce(packed(cfg), make_x(cfg, 8), y)
    ref = ohead.cross_entropy(ref_lg, y)
    err = assert_ce_close(ce, ref, what="tiny CE")
    assert abs(mean - ref.mean()) <= 1e-4
    say(f"tiny CE max err {err:.2e}")


def test_ce_parity_gemma_m64_int64_targets():
    cfg = "gemma"
    ref_lg = cached_oracle_logits(cfg, 64)
    y = make_targets(cfg, 64)
    ce, mean = gpu_ce(packed(cfg), make_x(cfg, 64), y, dtype=torch.int64)
    assert_ce_close(ce, ohead.cross_entropy(ref_lg, y), what="gemma CE")


def test_ce_target_out_of_range_is_nan():
    cfg = "tiny"
    V = CONFIGS[cfg]["V"]
    x = make_x(cfg, 8)[:4]
    ce, mean = gpu_ce(packed(cfg), x, np.array([0, -1, V, 5], dtype=np.int32))
    assert np.isnan(ce[1]) and np.isnan(ce[2])
    assert np.isfinite(ce[0]) and np.isfinite(ce[3]) and np.isnan(mean)


# ------------------------------------------------------------- special cases

@pytest.mark.parametrize("rc,rr", [(0, 0), (64, 0), (0, 32)])
def test_ablations(rc, rr):
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", rc=rc, rr=rr)
    x = make_x("tiny", 5)
    ph = PackedHead.from_arrays(h)
    assert_logits_close(gpu_logits(ph, x), ohead.logits(h, x), what=f"rc={rc} rr={rr}")
    ph.close()


def test_groupwise_factor_scales():
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", gV=128, gB=64)
    x = make_x("tiny", 3)
    ph = PackedHead.from_arrays(h)
    assert_logits_close(gpu_logits(ph, x), ohead.logits(h, x), what="gV=128 gB=64")
    ph.close()


@pytest.mark.parametrize("V,d,g,M", [(1000, 512, 64, 3), (8191, 512, 64, 7),
                                     (777, 96, 32, 5), (1500, 1024, 256, 2),
                                     (999, 3072, 128, 6), (33, 160, 32, 1)])
def test_ragged_shapes(V, d, g, M):
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=16, rr=8)
    x = make_x("tiny", M, d=d, basis="identity")
    say(f"ragged V={V} d={d} g={g} M={M}")
    ph = PackedHead.from_arrays(h)
    ref = ohead.logits(h, x)
    assert_logits_close(gpu_logits(ph, x, ld=d + 8), ref, what=f"ragged {V}x{d}")
    out = torch.full((M, V + 3), 7.0, device="cuda")
    ph.logits(torch_x(x), out=out[:, :V])
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert (o[:, V:] == 7.0).all(), "wrote past the row"
    assert_logits_close(o[:, :V], ref, what="ldo > V")
    y = np.arange(M, dtype=np.int32) * 7 % V
    ce, _ = gpu_ce(ph, x, y)
    assert_ce_close(ce, ohead.cross_entropy(ref, y), what="ragged CE")
    ph.close()


def test_determinism_bitwise():
    cfg = "qwen_decode"
    ph = packed(cfg)
    x = make_x(cfg, 16)[:4]
    a = gpu_logits(ph, x)
    b = gpu_logits(ph, x)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    y = make_targets(cfg, 4)
    c1, m1 = gpu_ce(ph, x, y)
    c2, m2 = gpu_ce(ph, x, y)
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32)) and m1 == m2


# ------------------------------------------------------------- errors

def test_error_paths_on_device():
    from paper_2608_02703_amd import archead as ab
    ph = packed("tiny")
    L = ab.lib()
    x = torch_x(make_x("tiny", 8))
    out = torch.empty((8, ph.V), device="cuda")
    ws = ph.workspace(8, ab.OP_LOGITS, x.device)
    s = ph._stream(x.device)

    def call(xp, M, ldx, outp, dt, ldo, wsp, wsn):
        return L.archead_logits(ph.handle, xp, M, ldx, outp, dt, ldo, wsp, wsn, s)
    assert call(x.data_ptr(), 0, ph.d, 0, ab.F32, ph.V, 0, 0) == ab.OK        # M = 0
    assert call(x.data_ptr() + 2, 8, ph.d, out.data_ptr(), ab.F32, ph.V,
                ws.data_ptr(), ws.numel()) == ab.E_MISALIGNED
    assert call(x.data_ptr(), 8, ph.d - 8, out.data_ptr(), ab.F32, ph.V,
                ws.data_ptr(), ws.numel()) == ab.E_INVALID_ARG
    assert call(x.data_ptr(), 8, ph.d, out.data_ptr(), ab.F32, ph.V,
                ws.data_ptr(), 16) == ab.E_WORKSPACE
    assert call(x.data_ptr(), 8, ph.d, out.data_ptr(), ab.I32, ph.V,
                ws.data_ptr(), ws.numel()) == ab.E_INVALID_ARG
    assert call(x.data_ptr(), 8, ph.d, out.data_ptr(), ab.F32, ph.V - 1,
                ws.data_ptr(), ws.numel()) == ab.E_INVALID_ARG
    assert call(x.data_ptr(), -1, ph.d, out.data_ptr(), ab.F32, ph.V,
                ws.data_ptr(), ws.numel()) == ab.E_INVALID_ARG
    assert L.archead_last_error()
    torch.cuda.synchronize()


# ------------------------------------------------------------- forced paths

@pytest.mark.parametrize("cfg,M", [("tiny", 8), ("qwen_decode", 16), ("gemma", 8),
                                   ("qwen_decode", 20)])
def test_all_paths_match_oracle(cfg, M):
    """The same tokens through the MFMA decode kernel, the decode GEMV and
    the tiled MFMA kernel (each forced for any M): all within tolerance of
    the oracle, logits and CE."""
    Mmax = max(max(CONFIGS[cfg]["Ms"]), M)
    ref = cached_oracle_logits(cfg, Mmax)[:M]
    ph = packed(cfg)
    x = make_x(cfg, Mmax)[:M]
    y = make_targets(cfg, M)
    ref_ce = ohead.cross_entropy(ref, y)
    try:
        for name in ("dec", "mid", "gemv", "tiled"):
            ph.force_path(name)
            say(f"{cfg} M={M} forced {name}")
            assert_logits_close(gpu_logits(ph, x), ref, what=f"{cfg} M={M} {name}")
            ce, mean = gpu_ce(ph, x, y)
            assert_ce_close(ce, ref_ce, what=f"{cfg} M={M} {name} CE")
    finally:
        ph.force_path("auto")


@pytest.mark.parametrize("path", ["gemv", "dec", "mid"])
def test_identity_probe_decode_kernels_bit_exact(path):
    """One-hot x, no low-rank parts: every logit is s_res * c, exact in fp32,
    and the decode kernels and the several-token kernel reach it exactly (the
    MFMA kernels' chain -136 + (136 + c) is exact too)."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", rc=0, rr=0)
    ph = PackedHead.from_arrays(h)
    ph.force_path(path)
    eye = np.zeros((h.d, h.d), dtype=np.uint16)
    eye[np.arange(h.d), np.arange(h.d)] = 0x3F80
    rows = eye[:96] if path == "gemv" else eye
    say(f"identity probe tiny, {path}: M={rows.shape[0]}")
    lg = gpu_logits(ph, rows).astype(np.float64)
    ref = ohead.logits(h, rows)
    bad = np.argwhere(lg != ref)
    assert bad.size == 0, (f"{len(bad)} logits differ, first at {bad[:3].tolist()}: "
                           f"gpu {lg[tuple(bad[0])]!r} oracle {ref[tuple(bad[0])]!r}")
    ph.close()


def test_identity_probe_dec_qwen_sampled_bit_exact():
    """The same one-hot probe on the Qwen-shaped head through the MFMA decode
    kernel (several passes of 16 tokens), bit for bit."""
    h = make_head("qwen_decode", rc=0, rr=0)
    from paper_2608_02703_amd import PackedHead
    ph = PackedHead.from_arrays(h)
    ph.force_path("dec")
    rng = np.random.default_rng(6)
    cols = np.unique(np.concatenate([[0, 1, 7, 8, 31, 32, 127, 128, 2047, 4095],
                                     rng.integers(0, h.d, 22)]))
    x = np.zeros((cols.size, h.d), dtype=np.uint16)
    x[np.arange(cols.size), cols] = 0x3F80
    say(f"identity probe qwen, dec: M={cols.size}")
    lg = gpu_logits(ph, x)
    assert np.array_equal(lg.astype(np.float64), ohead.logits(h, x))
    ph.close()


@pytest.mark.parametrize("path", ["dec", "gemv", "mid"])
def test_stage1_fallback_matches(path):
    """With the in-launch stage-1 exchange's wait bound set to zero polls,
    every consumer wave computes its t values itself; the logits and CE
    still match the oracle within tolerance (both decode kernels)."""
    from paper_2608_02703_amd import PackedHead
    h = cached_head("tiny")
    x = make_x("tiny", 8)
    y = make_targets("tiny", 8)
    ref = cached_oracle_logits("tiny", 8)
    from paper_2608_02703_amd import archead as ab
    ph = PackedHead.from_arrays(h)
    ph.set_launch(ab.LAUNCH_T_SPIN_LIMIT, 0)
    ph.force_path(path)
    say(f"{path} stage-1 fallback: tiny M=8")
    lg = gpu_logits(ph, x)
    assert_logits_close(lg, ref, what="fallback logits")
    ce, _ = gpu_ce(ph, x, y)
    assert_ce_close(ce, ohead.cross_entropy(ref, y), what="fallback CE")
    ph.close()


def test_launch_settings():
    """archead_set_launch: small persistent grids on each decode kernel still
    match the oracle; values outside the documented sets are rejected and
    leave the setting unchanged; 0 restores the built-in choice."""
    from paper_2608_02703_amd import ArcheadError, PackedHead
    from paper_2608_02703_amd import archead as ab
    h = cached_head("tiny")
    ph = PackedHead.from_arrays(h)
    try:
        for path, knob, value, M in (("gemv", ab.LAUNCH_GEMV_GRID, 3, 1),
                                     ("gemv", ab.LAUNCH_GEMV_BLOCKS_PER_CU, 1, 2),
                                     ("dec", ab.LAUNCH_DEC_BLOCKS, 2, 8),
                                     ("mid", ab.LAUNCH_MID_BLOCKS, 3, 8)):
            ph.set_launch(knob, value)
            assert ph.get_launch(knob) == value
            ph.force_path(path)
            say(f"launch setting {knob}={value} on {path}: tiny M={M}")
            x = make_x("tiny", 8)[:M]
            assert_logits_close(gpu_logits(ph, x), cached_oracle_logits("tiny", 8)[:M],
                                what=f"{path} with launch setting {knob}={value}")
            ph.set_launch(knob, 0)
            assert ph.get_launch(knob) == 0
        assert ph.get_launch(ab.LAUNCH_T_SPIN_LIMIT) == -1
        for knob, value in ((ab.LAUNCH_TILE_WAVES, 5), (ab.LAUNCH_TILE_ROWS, 256),
                            (ab.LAUNCH_TILE_ROWS, 32), (ab.LAUNCH_GEMV_GRID, -1),
                            (ab.LAUNCH_DEC_BLOCKS, 1 << 31), (ab.LAUNCH_T_SPIN_LIMIT, -2),
                            (ab.LAUNCH_T_SPIN_LIMIT + 1, 0), (-1, 0)):
            with pytest.raises(ArcheadError) as e:
                ph.set_launch(knob, value)
            assert e.value.status == ab.E_INVALID_ARG
            if 0 <= knob <= ab.LAUNCH_T_SPIN_LIMIT:
                assert ph.get_launch(knob) == (-1 if knob == ab.LAUNCH_T_SPIN_LIMIT else 0)
    finally:
        ph.close()


@pytest.mark.parametrize("V,d,g,M,rc,rr", [(1000, 512, 64, 17, 16, 8), (777, 256, 32, 5, 20, 4),
                                           (33, 128, 32, 1, 16, 8), (8191, 512, 128, 16, 64, 0),
                                           (4099, 1024, 128, 3, 0, 36), (130, 256, 64, 40, 12, 28),
                                           (777, 96, 32, 5, 20, 4), (50, 1536, 128, 2, 6, 8)])
def test_dec_ragged(V, d, g, M, rc, rr):
    """The MFMA decode kernel on partial 16-row units, several passes,
    padded rank dimensions, wide row strides, bf16 output and CE.  The last
    two shapes are outside its limits (d/g not a multiple of 4, a rank not a
    multiple of 4): forcing it there must still give correct results through
    another kernel."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=rc, rr=rr)
    x = make_x("tiny", M, d=d, basis="identity")
    ph = PackedHead.from_arrays(h)
    ph.force_path("dec")
    ref = ohead.logits(h, x)
    say(f"dec ragged V={V} d={d} g={g} M={M} rc={rc} rr={rr}")
    assert_logits_close(gpu_logits(ph, x, ld=d + 8), ref, what="dec ragged")
    out = torch.full((M, V + 3), 5.0, device="cuda")
    ph.logits(torch_x(x), out=out[:, :V])
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert (o[:, V:] == 5.0).all(), "wrote past the row"
    y = (np.arange(M) * 11 % V).astype(np.int32)
    ce, _ = gpu_ce(ph, x, y)
    assert_ce_close(ce, ohead.cross_entropy(ref, y), what="dec ragged CE")
    bits = gpu_logits(ph, x, out_dtype=torch.bfloat16)
    assert_bf16_output(bits, o[:, :V], ref, "dec ragged bf16")
    ph.close()


@pytest.mark.parametrize("V,d,g,M,rc,rr", [(1000, 512, 64, 17, 16, 8), (777, 1024, 128, 40, 20, 4),
                                           (33, 512, 64, 5, 16, 8), (8191, 512, 128, 64, 64, 0),
                                           (4099, 1024, 64, 100, 0, 36), (130, 2560, 128, 33, 12, 28),
                                           (500, 4096, 64, 20, 128, 128), (777, 96, 32, 5, 20, 4),
                                           (300, 768, 128, 20, 8, 8)])
def test_mid_ragged(V, d, g, M, rc, rr):
    """The several-token kernel on partial 16-row units, tiles of 32 and 64
    tokens with partial row blocks, several tiles, 4 to 64 scale groups,
    padded rank dimensions (up to 128 + 128), wide row strides, bf16 output
    and CE.  The last two shapes are outside its limits (g = 32; d not a
    multiple of two 256-element windows): forcing it there must still give
    correct results through another kernel."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=rc, rr=rr)
    x = make_x("tiny", M, d=d, basis="identity")
    ph = PackedHead.from_arrays(h)
    ph.force_path("mid")
    ref = ohead.logits(h, x)
    say(f"mid ragged V={V} d={d} g={g} M={M} rc={rc} rr={rr}")
    assert_logits_close(gpu_logits(ph, x, ld=d + 8), ref, what="mid ragged")
    out = torch.full((M, V + 3), 5.0, device="cuda")
    ph.logits(torch_x(x), out=out[:, :V])
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert (o[:, V:] == 5.0).all(), "wrote past the row"
    y = (np.arange(M) * 11 % V).astype(np.int32)
    ce, _ = gpu_ce(ph, x, y)
    assert_ce_close(ce, ohead.cross_entropy(ref, y), what="mid ragged CE")
    bits = gpu_logits(ph, x, out_dtype=torch.bfloat16)
    assert_bf16_output(bits, o[:, :V], ref, "mid ragged bf16")
    ph.close()


@pytest.mark.parametrize("path", ["dec", "mid"])
@pytest.mark.parametrize("V,d,g,M,rc,rr", [(1000, 512, 64, 17, 16, 8), (777, 1024, 128, 40, 20, 4),
                                           (4099, 1024, 64, 100, 0, 36), (130, 2560, 128, 33, 12, 28),
                                           (500, 8192, 128, 20, 128, 128)])
def test_8bit_scale_codes_ragged(path, V, d, g, M, rc, rr):
    """8-bit scale codes on partial 16-row units, 4 to 64 scale groups per
    row (64: one 16-byte code load per lane holds a whole row set), several
    tiles and passes, padded ranks, CE and bf16 output."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=rc, rr=rr, scales="u8")
    x = make_x("tiny", M, d=d, basis="identity")
    ph = PackedHead.from_arrays(h)
    ph.force_path(path)
    ref = ohead.logits(h, x)
    say(f"8-bit ragged {path} V={V} d={d} g={g} M={M} rc={rc} rr={rr}")
    lg = gpu_logits(ph, x, ld=d + 8)
    assert_logits_close(lg, ref, what=f"8-bit ragged {path}")
    y = (np.arange(M) * 7 % V).astype(np.int32)
    ce, _ = gpu_ce(ph, x, y)
    assert_ce_close(ce, ohead.cross_entropy(ref, y), what=f"8-bit ragged {path} CE")
    bits = gpu_logits(ph, x, out_dtype=torch.bfloat16)
    assert_bf16_output(bits, lg, ref, f"8-bit ragged {path} bf16")
    ph.close()


def test_identity_probe_mid_qwen_sampled_bit_exact():
    """The one-hot probe on the Qwen-shaped head through the several-token
    kernel (a tile of 64 tokens and a partial one), bit for bit."""
    h = make_head("qwen_decode", rc=0, rr=0)
    from paper_2608_02703_amd import PackedHead
    ph = PackedHead.from_arrays(h)
    ph.force_path("mid")
    rng = np.random.default_rng(7)
    cols = np.unique(np.concatenate([[0, 1, 7, 8, 31, 32, 127, 128, 255, 256, 2047, 4095],
                                     rng.integers(0, h.d, 90)]))
    x = np.zeros((cols.size, h.d), dtype=np.uint16)
    x[np.arange(cols.size), cols] = 0x3F80
    say(f"identity probe qwen, mid: M={cols.size}")
    lg = gpu_logits(ph, x)
    assert np.array_equal(lg.astype(np.float64), ohead.logits(h, x))
    ph.close()


def test_group_size_not_multiple_of_64_uses_decode_kernel():
    """g = 32 or 96: the many-token kernel stages 64 codes of one group, so
    such heads run the decode kernel in passes of 4 tokens at every M."""
    from paper_2608_02703_amd import PackedHead
    for V, d, g, M in ((777, 256, 32, 70), (500, 288, 96, 41)):
        h = make_head("tiny", V=V, d=d, g=g, rc=20, rr=4)
        x = make_x("tiny", M, d=d, basis="identity")
        ph = PackedHead.from_arrays(h)
        ph.force_path("tiled")
        say(f"g={g} fallback V={V} d={d} M={M}")
        assert_logits_close(gpu_logits(ph, x), ohead.logits(h, x), what=f"g={g}")
        ph.close()


def test_zero_scales_many_token_kernel():
    """Exactly-zero fp16 scales (a residual group, s_U, s_A, and one row with
    every scale zero) on the many-token kernel, whose accumulator divides by
    the current group's scale."""
    import dataclasses
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny")
    rng = np.random.default_rng(11)
    rs = h.res_scales.copy()
    rs[rng.random(rs.shape) < 0.05] = 0
    rs[7, :] = 0
    su, sa = h.core_u_scale.copy(), h.corr_a_scale.copy()
    su[rng.integers(0, h.V, 40)] = 0
    sa[rng.integers(0, h.V, 40)] = 0
    su[7] = sa[7] = 0
    h = dataclasses.replace(h, res_scales=rs, core_u_scale=su, corr_a_scale=sa)
    ph = PackedHead.from_arrays(h)
    ph.force_path("tiled")
    x = make_x("tiny", 300)
    say("zero scales: tiny head, M=300 (many-token kernel)")
    lg = gpu_logits(ph, x)
    ref = ohead.logits(h, x)
    assert np.all(lg[:, 7] == 0) or np.abs(lg[:, 7]).max() < 1e-12
    err = assert_logits_close(lg, ref, what="zero scales")
    say(f"  max rel err {err:.2e}")
    ph.close()


@pytest.mark.parametrize("V,d,g,M", [(1000, 512, 64, 130), (777, 256, 64, 33),
                                     (300, 1024, 256, 5), (513, 192, 64, 300),
                                     (1000, 2048, 64, 40), (777, 1536, 64, 17)])
def test_mfma_ragged_tiles(V, d, g, M):
    """Token and vocabulary counts that leave partial MFMA tiles; ranks that
    are not multiples of 32; row strides wider than the rows.  The last two
    shapes have few token blocks and 32 / 24 residual groups, so stage 1 is
    split along d over 4 / 2 workgroups and summed in a second kernel."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=40, rr=12)
    x = make_x("tiny", M, d=d, basis="identity")
    ph = PackedHead.from_arrays(h)
    ph.force_path("tiled")
    ref = ohead.logits(h, x)
    say(f"mfma ragged V={V} d={d} g={g} M={M}")
    assert_logits_close(gpu_logits(ph, x, ld=d + 16), ref, what="mfma ragged")
    out = torch.full((M, V + 5), 3.0, device="cuda")
    ph.logits(torch_x(x), out=out[:, :V])
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert (o[:, V:] == 3.0).all(), "wrote past the row"
    y = (np.arange(M) * 13 % V).astype(np.int64)
    ce, mean = gpu_ce(ph, x, y, dtype=torch.int64)
    assert_ce_close(ce, ohead.cross_entropy(ref, y), what="mfma ragged CE")
    bits = gpu_logits(ph, x, out_dtype=torch.bfloat16)
    assert_bf16_output(bits, o[:, :V], ref, "mfma ragged bf16")
    ph.close()


# ------------------------------------------------------------- fused argmax

def gpu_argmax(ph, x_bits):
    idx, mx = ph.logits_argmax(torch_x(x_bits))
    torch.cuda.synchronize()
    return idx.cpu().numpy(), mx.cpu().numpy()


def assert_argmax_matches_oracle(idx, ref, what):
    """idx equals the oracle's argmax on every token whose oracle top-2 gap
    exceeds twice the logit tolerance; returns the number of such tokens."""
    from tests.gpu_util import LOGIT_TOL
    top = ref.max(axis=1)
    keep = ohead.top2_gap(ref) > 2 * LOGIT_TOL * (1 + np.abs(top))
    bad = np.nonzero(keep & (np.asarray(idx) != ohead.argmax(ref)))[0]
    assert bad.size == 0, f"{what}: argmax differs from the oracle on tokens {bad[:10]}"
    return int(keep.sum())


@pytest.mark.parametrize("cfg,M", [("tiny", 8), ("qwen_decode", 16), ("gemma", 8),
                                   ("qwen_decode", 40)])
def test_argmax_equals_first_argmax_of_own_logits(cfg, M):
    """The fused argmax through each kernel (forced) is the first-index
    argmax of the same kernel's fp32 logits, bit for bit (ties included), and
    its max is their maximum; both agree with the oracle's argmax on every
    token whose top-2 gap is clear of the logit tolerance."""
    Mmax = max(max(CONFIGS[cfg]["Ms"]), M)
    ref = cached_oracle_logits(cfg, Mmax)[:M]
    ph = packed(cfg)
    x = make_x(cfg, Mmax)[:M]
    try:
        for name in ("dec", "mid", "gemv", "tiled"):
            ph.force_path(name)
            say(f"argmax {cfg} M={M} forced {name}")
            lg = gpu_logits(ph, x)
            idx, mx = gpu_argmax(ph, x)
            assert np.array_equal(idx, np.argmax(lg, axis=1)), f"{name}: argmax differs"
            assert np.array_equal(mx, lg.max(axis=1)), f"{name}: max differs"
            assert_argmax_matches_oracle(idx, ref, name)
    finally:
        ph.force_path("auto")


@pytest.mark.parametrize("path", ["dec", "mid", "gemv", "tiled"])
def test_argmax_ties_take_the_smallest_index(path):
    """x = 0 makes every logit exactly 0: the argmax is index 0.  With a
    one-hot x and no low-rank parts, two far-apart rows (in different
    workgroups and tiles, identical scales and the same code 7 at the hot
    column) share the largest logit 7 * 1.0: the argmax is the smaller of
    the two."""
    from oracle.layout import pack_int4, unpack_int4
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", rc=0, rr=0)
    i0, a, b = 5, 100, h.V - 5
    codes = unpack_int4(h.res_codes, h.d)
    codes[[a, b], i0] = 7
    h.res_codes = pack_int4(codes)
    h.res_scales = h.res_scales.copy()
    h.res_scales[a, i0 // h.g] = np.float16(1.0)
    h.res_scales[b] = h.res_scales[a]   # identical rows of scales: identical arithmetic
    ph = PackedHead.from_arrays(h)
    ph.force_path(path)
    say(f"argmax ties, {path}")
    zeros = np.zeros((3, h.d), dtype=np.uint16)
    idx, mx = gpu_argmax(ph, zeros)
    assert idx.tolist() == [0, 0, 0] and mx.tolist() == [0.0, 0.0, 0.0]
    x = np.zeros((2, h.d), dtype=np.uint16)
    x[:, i0] = 0x3F80
    ref = ohead.logits(h, x)
    assert ref[0, a] == ref[0, b] == ref[0].max() == 7.0
    idx, mx = gpu_argmax(ph, x)
    assert idx.tolist() == [a, a]
    if path == "tiled":   # its scale-ratio chain rounds in the last bits
        assert np.allclose(mx, 7.0, rtol=1e-6, atol=0)
    else:
        assert mx.tolist() == [7.0, 7.0]
    ph.close()


@pytest.mark.parametrize("cfg", ["tiny", "qwen_decode"])
def test_argmax_one_launch_gemv_any_workspace_contents(cfg):
    """1 to 4 tokens on the GEMV (one head pass, then the partials' merge):
    over a workspace holding the previous call's leftovers, all ones, or in
    every 64-bit word a foreign call stamp with a partial count, each call
    gives the first-index argmax of the same kernel's fp32 logits and their
    maximum, bit for bit."""
    from paper_2608_02703_amd.archead import OP_ARGMAX
    ph = packed(cfg)
    x = make_x(cfg, max(4, max(CONFIGS[cfg]["Ms"])))
    foreign = (0x5A5A5A5A << 32) | 7
    ph.force_path("gemv")
    try:
        for M in (1, 2, 3, 4, 1):
            lg = gpu_logits(ph, x[:M])
            xt = torch_x(x[:M])
            for fill in ("leftover", "ones", "foreign"):
                say(f"argmax on the GEMV {cfg} M={M} workspace {fill}")
                ws = ph.workspace(M, OP_ARGMAX, xt.device)
                if fill == "ones":
                    ws.fill_(0xFF)
                elif fill == "foreign":
                    ws.view(torch.int64).fill_(foreign)
                idx, mx = ph.logits_argmax(xt, ws=ws)
                torch.cuda.synchronize()
                idx, mx = idx.cpu().numpy(), mx.cpu().numpy()
                assert np.array_equal(idx, np.argmax(lg, axis=1)), f"M={M} {fill}: argmax differs"
                assert np.array_equal(mx, lg.max(axis=1)), f"M={M} {fill}: max differs"
    finally:
        ph.force_path("auto")


def test_argmax_gemma_m64_against_oracle():
    """The Gemma-shaped workload with 64 tokens (logits + argmax), through the
    library's own kernel choice: the fused argmax equals the oracle's on
    every token whose top-2 gap is clear of the logit tolerance."""
    ref = cached_oracle_logits("gemma", 64)
    ph = packed("gemma")
    idx, mx = gpu_argmax(ph, make_x("gemma", 64))
    n = assert_argmax_matches_oracle(idx, ref, "gemma M=64")
    say(f"gemma M=64 argmax: {n} clear tokens agree")
    assert n > 0
    assert_logits_close(mx[:, None], ref.max(axis=1)[:, None], what="gemma max logit")


# ------------------------------------------------------ 8-bit scale codes

@pytest.mark.parametrize("path", ["gemv", "dec", "mid", "tiled", "auto"])
def test_8bit_scale_codes_tiny(path):
    """Residual group scales stored as 8-bit codes with an fp16 row scale
    (s = rs * q): every kernel matches the oracle for logits, bf16 logits
    and CE, and the fused argmax equals the first argmax of the same
    logits."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", scales="u8")
    ph = PackedHead.from_arrays(h)
    ph.force_path(path)
    for M in (1, 8, 21):
        x = make_x("tiny", M)
        ref = ohead.logits(h, x)
        say(f"8-bit scales tiny {path} M={M}")
        lg = gpu_logits(ph, x)
        assert_logits_close(lg, ref, what=f"8-bit scales {path} M={M}")
        y = make_targets("tiny", M)
        ce, _ = gpu_ce(ph, x, y)
        assert_ce_close(ce, ohead.cross_entropy(ref, y), what=f"8-bit scales {path} M={M} CE")
        idx, mx = gpu_argmax(ph, x)
        assert np.array_equal(idx, np.argmax(lg, axis=1))
        bits = gpu_logits(ph, x, out_dtype=torch.bfloat16)
        assert_bf16_output(bits, lg, ref, f"8-bit scales {path} M={M} bf16")
    ph.close()


@pytest.mark.parametrize("path", ["gemv", "dec", "mid"])
def test_8bit_scale_codes_identity_probe_bit_exact(path):
    """One-hot x, no low-rank parts, 8-bit scale codes: every logit is
    rs * q * c, exact in fp32 (11 + 8 + 4 significant bits), bit for bit
    through the kernels that multiply a group's partial by its code and the
    row's total by the row scale."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", rc=0, rr=0, scales="u8")
    ph = PackedHead.from_arrays(h)
    ph.force_path(path)
    eye = np.zeros((64, h.d), dtype=np.uint16)
    cols = np.arange(0, h.d, h.d // 64)
    eye[np.arange(64), cols] = 0x3F80
    say(f"8-bit scales identity probe, {path}")
    lg = gpu_logits(ph, eye).astype(np.float64)
    assert np.array_equal(lg, ohead.logits(h, eye))
    ph.close()


@pytest.mark.parametrize("M", [1, 16, 40, 130])
def test_8bit_scale_codes_qwen_sampled(M):
    """The Qwen-shaped head with 8-bit scale codes through the library's own
    choice (the GEMV at M = 1, the MFMA decode kernel at M = 16, the
    several-token kernel at M = 40, the tiled kernel at M = 130): sampled
    vocabulary columns against the oracle."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode", scales="u8")
    ph = PackedHead.from_arrays(h)
    x = make_x("qwen_decode", M)
    rng = np.random.default_rng(11)
    ids = np.unique(np.concatenate([[0, 1, h.V - 1], rng.integers(0, h.V, 400)]))
    say(f"8-bit scales qwen M={M}, {ids.size} sampled columns")
    lg = gpu_logits(ph, x)[:, ids]
    assert_logits_close(lg, ohead.logits(h, x, vocab=ids), what=f"8-bit scales qwen M={M}")
    ph.close()

