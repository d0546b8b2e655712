"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: hand-derived
fixtures, closed forms, exact rational arithmetic, a theorem (Eckart-Young-
Mirsky), an independent algorithm (alternating least squares), or numbers the
paper prints.  None of them touches the HIP library.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle.bytes as obytes
from oracle import construct, head as ohead, layout, metrics
from synth import make_head, make_x, f64_to_bf16_bits
from tests import fixtures


# ---------------------------------------------------------------- P1 layout

def test_layout_golden_words():
    for b, c in fixtures.layout_cases():
        got = layout.unpack_int4(b.reshape(1, 4), 8)[0]
        assert got.tolist() == c.tolist(), (b, got, c)
        assert layout.pack_int4(c.reshape(1, 8)).tolist() == [b.tolist()]


def test_layout_every_nibble_every_position():
    rng = np.random.default_rng(7)
    base = rng.integers(-8, 8, size=(1, 8))
    for pos in range(8):
        for code in range(-8, 8):
            c = base.copy()
            c[0, pos] = code
            p = layout.pack_int4(c)
            assert layout.unpack_int4(p, 8).tolist() == c.tolist()
            # changing one element changes exactly one nibble of the word
            q0 = int(layout.pack_int4(base).view("<u4")[0, 0])
            q1 = int(p.view("<u4")[0, 0])
            diff = q0 ^ q1
            shift = 4 * (pos // 2) + (16 if pos % 2 else 0)
            assert diff & ~(0xF << shift) == 0


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 5), st.integers(1, 12), st.integers(0, 2**32 - 1))
def test_layout_round_trip_codes(rows, words, seed):
    rng = np.random.default_rng(seed)
    c = rng.integers(-8, 8, size=(rows, 8 * words))
    assert np.array_equal(layout.unpack_int4(layout.pack_int4(c), 8 * words), c)


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 5), st.integers(1, 12), st.integers(0, 2**32 - 1))
def test_layout_round_trip_bytes(rows, words, seed):
    rng = np.random.default_rng(seed)
    b = rng.integers(0, 256, size=(rows, 4 * words), dtype=np.uint8)
    assert np.array_equal(layout.pack_int4(layout.unpack_int4(b, 8 * words)), b)


def test_layout_rejects_ragged_and_out_of_range():
    with pytest.raises(ValueError):
        layout.unpack_int4(np.zeros((1, 2), np.uint8), 4)
    with pytest.raises(ValueError):
        layout.pack_int4(np.full((1, 8), 8))
    with pytest.raises(ValueError):
        layout.pack_int4(np.full((1, 8), -9))


def test_bf16_and_fp16_decoding_exact():
    # 1.0, -2.0, 0.5, smallest normal and 3.140625 as bf16 / fp16 bit patterns
    bf = np.array([0x3F80, 0xC000, 0x3F00, 0x0080, 0x4049], dtype=np.uint16)
    assert layout.bf16_to_f64(bf).tolist() == [1.0, -2.0, 0.5, 2.0 ** -126,
                                              3.140625]
    h = np.array([0x3C00, 0xC000, 0x3800, 0x0001, 0x7BFF], dtype=np.uint16)
    assert layout.fp16_to_f64(h).tolist() == [1.0, -2.0, 0.5, 2.0 ** -24,
                                             65504.0]


def test_generator_bf16_rounding_is_nearest_even():
    rng = np.random.default_rng(3)
    a = rng.standard_normal(4000) * np.exp(rng.uniform(-20, 20, 4000))
    bits = f64_to_bf16_bits(a)
    val = layout.bf16_to_f64(bits)
    up = layout.bf16_to_f64((bits.astype(np.int64) + 1).astype(np.uint16))
    dn = layout.bf16_to_f64((bits.astype(np.int64) - 1).astype(np.uint16))
    err = np.abs(val - a)
    assert np.all(err <= np.abs(up - a)) and np.all(err <= np.abs(dn - a))
    # ties go to the even pattern: 1 + 2^-8 sits halfway between 1 and 1+2^-7
    assert f64_to_bf16_bits([1 + 2 ** -8, 1 + 3 * 2 ** -8]).tolist() == \
        [0x3F80, 0x3F82]


# ------------------------------------------------------- worked example

def test_worked_example_logits_and_ce():
    h, x, expect, y = fixtures.worked_head()
    lg = ohead.logits(h, x)
    assert np.array_equal(lg, expect)
    ce = ohead.cross_entropy(lg, y)
    other = expect[np.arange(3), 1 - y]
    tgt = expect[np.arange(3), y]
    closed = [math.log1p(math.exp(o - t)) for o, t in zip(other, tgt)]
    np.testing.assert_allclose(ce, closed, rtol=1e-13, atol=1e-14)


# ------------------------------------------------------- P2 linearity

@pytest.mark.parametrize("gV,gB", [(None, None), (128, 64)])
def test_dense_equals_factorized(gV, gB):
    over = dict(V=700)
    if gV:
        over.update(gV=gV, gB=gB)
    h = make_head("tiny", **over)
    x = make_x("tiny", 5, basis="identity")
    a = ohead.logits(h, x, chunk=256)
    b = ohead.logits_factorized(h, x)
    scale = np.abs(a).max()
    assert np.max(np.abs(a - b)) <= 1e-12 * scale


# ------------------------------------------------------- P3 exact rationals

def _exact_logits(h, x_bits):
    codes = layout.unpack_int4(h.res_codes, h.d)
    F = lambda v: Fraction(float(v))                       # noqa: E731
    xs = [[F(v) for v in row] for row in layout.bf16_to_f64(x_bits)]
    sres = layout.fp16_to_f64(h.res_scales)
    out = []
    for xm in xs:
        row = []
        for v in range(h.V):
            acc = Fraction(0)
            for i in range(h.d):
                w = F(sres[v, i // h.g]) * int(codes[v, i])
                for k in range(h.rc):
                    w += F(layout.fp16_to_f64(h.core_u_scale[v:v + 1])[0]) * \
                        int(h.core_u[v, k]) * \
                        F(layout.fp16_to_f64(h.core_v_scale)[k, i // h.gV]) * \
                        int(h.core_v[k, i])
                for k in range(h.rr):
                    w += F(layout.fp16_to_f64(h.corr_a_scale[v:v + 1])[0]) * \
                        int(h.corr_a[v, k]) * \
                        F(layout.fp16_to_f64(h.corr_b_scale)[k, i // h.gB]) * \
                        int(h.corr_b[k, i])
                acc += xm[i] * w
            row.append(acc)
        out.append(row)
    return out


def test_exact_rational_brute_force():
    h = make_head("tiny", V=5, d=64, g=32, rc=2, rr=3, gV=32, gB=16)
    x = make_x("tiny", 2, d=64, basis="identity")
    exact = _exact_logits(h, x)
    lg = ohead.logits(h, x)
    for m in range(2):
        for v in range(h.V):
            e = exact[m][v]
            assert abs(lg[m, v] - float(e)) <= 1e-13 * max(1.0, abs(float(e)))


# ------------------------------------------------------- P4 identity probe

def test_identity_probe_recovers_codes_times_scales():
    h = make_head("tiny", V=300, rc=0, rr=0)
    eye = np.zeros((h.d, h.d), dtype=np.uint16)
    eye[np.arange(h.d), np.arange(h.d)] = 0x3F80            # bf16 1.0
    lg = ohead.logits(h, eye)                               # [d, V]
    codes = layout.unpack_int4(h.res_codes, h.d)
    s = layout.fp16_to_f64(h.res_scales)
    for i in (0, 1, 7, 8, h.g - 1, h.g, h.d - 1):
        assert np.array_equal(lg[i], s[:, i // h.g] * codes[:, i])


# ------------------------------------------------------- P5 special cases

def test_unit_scales_integer_matmul_exact():
    h = make_head("tiny", V=256, d=128, g=64, rc=3, rr=2)
    one = np.float16(1.0)
    for k in ("res_scales", "core_u_scale", "core_v_scale", "corr_a_scale",
              "corr_b_scale"):
        setattr(h, k, np.full_like(getattr(h, k), one))
    rng = np.random.default_rng(11)
    xi = rng.integers(-3, 4, size=(4, h.d))
    x = f64_to_bf16_bits(xi.astype(np.float64))
    Wint = layout.unpack_int4(h.res_codes, h.d).astype(np.int64) + \
        h.core_u.astype(np.int64) @ h.core_v.astype(np.int64) + \
        h.corr_a.astype(np.int64) @ h.corr_b.astype(np.int64)
    assert np.array_equal(ohead.logits(h, x), (xi @ Wint.T).astype(np.float64))


def test_group_int4_and_core_only_special_cases():
    h = make_head("tiny", V=200)
    x = make_x("tiny", 3, basis="identity")
    full = ohead.logits(h, x)
    h0 = make_head("tiny", V=200, rc=0, rr=0)
    res_only = ohead.logits(h0, x)
    hc = make_head("tiny", V=200, rr=0)
    core_only = ohead.logits(hc, x)
    X = layout.bf16_to_f64(x)
    # residual codes are drawn from the same stream whatever the ranks are
    assert np.array_equal(h0.res_codes, h.res_codes)
    np.testing.assert_allclose(core_only - res_only,
                               (X @ ohead.right_factor(h.core_v, h.core_v_scale, h.gV).T)
                               @ ohead.left_factor(h.core_u, h.core_u_scale).T,
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(full - core_only,
                               (X @ ohead.right_factor(h.corr_b, h.corr_b_scale, h.gB).T)
                               @ ohead.left_factor(h.corr_a, h.corr_a_scale).T,
                               rtol=1e-12, atol=1e-12)


def test_rowwise_scaling_g_equals_d():
    h = make_head("tiny", V=64, d=256, g=256, rc=0, rr=0)
    x = make_x("tiny", 2, d=256, basis="identity")
    X = layout.bf16_to_f64(x)
    c = layout.unpack_int4(h.res_codes, 256).astype(np.float64)
    s = layout.fp16_to_f64(h.res_scales)[:, 0]
    np.testing.assert_allclose(ohead.logits(h, x), (X @ c.T) * s[None, :],
                               rtol=1e-13, atol=1e-15)


# ------------------------------------------------------- P6 / P7 construction

def _tiny_problem(seed=0, V=48, d=24, N=300):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((V, d)) @ np.diag(np.linspace(2.0, 0.2, d))
    W += 0.3 * rng.standard_normal((V, 3)) @ rng.standard_normal((3, d))
    lam = np.arange(1, d + 1) ** -1.5
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    H = (rng.standard_normal((N, d)) * np.sqrt(lam)) @ Q.T
    return W, H


def _metric_err(E, A, B, T):
    return float(np.linalg.norm((E - A @ B) @ T) ** 2)


def _als_best(Et, r, iters=3000, seed=1):
    """Best rank-r approximation of Et by alternating least squares."""
    rng = np.random.default_rng(seed)
    B = rng.standard_normal((r, Et.shape[1]))
    for _ in range(iters):
        A = Et @ np.linalg.pinv(B)
        B = np.linalg.pinv(A) @ Et
    return float(np.linalg.norm(Et - A @ B) ** 2)


@pytest.mark.parametrize("p", [0.0, 0.5, 0.75])
def test_eym_correction_is_best_rank_r_in_metric(p):
    W, H = _tiny_problem()
    r = 4
    h, info = construct.build_head(W, H, rc=3, rr=r, g=8, p=p, lam=1e-3)
    E, T, A, B = info["E"], info["T"], info["A_w"], info["B_w"]
    best = _metric_err(E, A, B, T)
    # tail energy from the eigenvalues of the Gram matrix (E T)^T (E T)
    ev = np.sort(np.linalg.eigvalsh((E @ T).T @ (E @ T)))[::-1]
    assert best == pytest.approx(float(np.sum(ev[r:])), rel=1e-9, abs=1e-12)
    # an independent iterative solver reaches the same optimum
    assert best == pytest.approx(_als_best(E @ T, r), rel=1e-6)
    rng = np.random.default_rng(5)
    for _ in range(200):   # random rank-r products never do better
        Ar, Br = rng.standard_normal(A.shape), rng.standard_normal(B.shape)
        assert _metric_err(E, Ar, Br, T) >= best
    for eps in (1e-3, 1e-2):   # nor do small perturbations of the optimum
        for _ in range(50):
            dA = eps * rng.standard_normal(A.shape)
            dB = eps * rng.standard_normal(B.shape)
            assert _metric_err(E, A + dA, B + dB, T) >= best * (1 - 1e-12)


def test_p0_reduces_to_plain_truncated_svd():
    W, H = _tiny_problem(seed=2)
    r = 3
    _, info = construct.build_head(W, H, rc=2, rr=r, g=8, p=0.0, lam=1e-3)
    np.testing.assert_allclose(info["T"], np.eye(W.shape[1]), atol=1e-12)
    E = info["E"]
    approx = info["A_w"] @ info["B_w"]
    # best rank-r in Frobenius norm: the error equals the tail energy of E
    ev = np.sort(np.linalg.eigvalsh(E.T @ E))[::-1]
    assert np.linalg.norm(E - approx) ** 2 == pytest.approx(ev[r:].sum(),
                                                            rel=1e-9)


def test_metric_transform_inverse_and_square():
    _, H = _tiny_problem(seed=3)
    C = construct.damped_covariance(H, 1e-3)
    T, Ti = construct.metric_transform(C, 0.75)
    np.testing.assert_allclose(T @ Ti, np.eye(C.shape[0]), atol=1e-9)
    T2, _ = construct.metric_transform(C, 0.5)
    np.testing.assert_allclose(T2 @ T2, C, rtol=1e-10, atol=1e-12)
    T1, _ = construct.metric_transform(C, 1.0)
    np.testing.assert_allclose(T1, C, rtol=1e-10, atol=1e-12)
    N = H.shape[0]
    cbar = np.mean(np.sum(H * H, axis=0) / N)
    np.testing.assert_allclose(np.diag(C), np.sum(H * H, axis=0) / N +
                               1e-3 * cbar, rtol=1e-12)


def test_p_half_metric_equals_damped_logit_mse():
    W, H = _tiny_problem(seed=4)
    lam = 1e-3
    C = construct.damped_covariance(H, lam)
    T, _ = construct.metric_transform(C, 0.5)
    N = H.shape[0]
    cbar = np.mean(np.sum(H * H, axis=0) / N)
    rng = np.random.default_rng(9)
    for _ in range(5):
        D = rng.standard_normal(W.shape)
        lhs = np.linalg.norm(D @ T) ** 2
        rhs = np.linalg.norm(H @ D.T) ** 2 / N + lam * cbar * np.linalg.norm(D) ** 2
        assert lhs == pytest.approx(rhs, rel=1e-10)


def test_construction_packs_valid_head():
    W, H = _tiny_problem(seed=6, V=40, d=32)
    h, info = construct.build_head(W, H, rc=3, rr=2, g=16, p=0.75, lam=1e-3)
    lg = ohead.logits(h, np.eye(32))
    np.testing.assert_allclose(lg.T, info["W_d"] +
                               ohead.left_factor(h.corr_a, h.corr_a_scale) @
                               ohead.right_factor(h.corr_b, h.corr_b_scale, h.gB),
                               rtol=1e-12, atol=1e-12)
    assert np.abs(layout.unpack_int4(h.res_codes, 32)).max() <= 7
    assert np.abs(h.core_u).max() <= 15 and np.abs(h.corr_a).max() <= 127


# ------------------------------------------------------- P8 CE closed forms

@pytest.mark.parametrize("V,printed", [(8192, 9.010913), (151936, 11.931215),
                                       (262144, 12.476649), (128256, 11.761784)])
def test_ce_equal_logits_is_ln_v(V, printed):
    ce = ohead.cross_entropy(np.zeros((2, V)), [0, V - 1])
    assert ce[0] == pytest.approx(math.log(V), rel=1e-14)
    assert round(ce[1], 6) == printed


def test_ce_zero_head_gives_ln_v():
    h = make_head("tiny", V=1000)
    h.res_codes[:] = 0x88                                  # every code 0
    for k in ("core_u", "corr_a"):
        getattr(h, k)[:] = 0
    ce = ohead.cross_entropy(ohead.logits(h, make_x("tiny", 3, basis="identity")),
                             [0, 5, 999])
    np.testing.assert_allclose(ce, math.log(1000), rtol=1e-14)


def test_ce_single_logit_and_shift_invariance():
    V = 5000
    for a in (-3.0, 0.0, 2.5, 40.0):
        lg = np.zeros((1, V))
        lg[0, 17] = a
        ce = ohead.cross_entropy(lg, [17])[0]
        assert ce == pytest.approx(math.log1p((V - 1) * math.exp(-a)), rel=1e-12)
    rng = np.random.default_rng(1)
    lg = rng.standard_normal((3, 777)) * 5
    y = [0, 400, 776]
    np.testing.assert_allclose(ohead.cross_entropy(lg + 123.0, y),
                               ohead.cross_entropy(lg, y), rtol=1e-12)
    assert np.isnan(ohead.cross_entropy(lg, [0, -1, 777])[1:]).all()


def test_argmax_smallest_index_on_ties():
    lg = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0]])
    assert ohead.argmax(lg).tolist() == [1, 0]
    assert ohead.top2_gap(lg).tolist() == [0.0, 0.0]


# ------------------------------------------------------- P9 printed metrics

def test_paper_rows_obey_ppl_identities():
    rows = fixtures.paper_metric_rows()
    dense = rows["dense_bf16"]
    for name, r in rows.items():
        # CE printed to 3 decimals: its rounding moves exp(CE) by <= 0.05 %
        assert abs(metrics.ppl(r["ce"]) - r["ppl"]) <= r["ppl"] * 5.01e-4 + 5e-4, name
        lo = metrics.rel_ppl(r["dce"] - 5e-4, 0.0)
        hi = metrics.rel_ppl(r["dce"] + 5e-4, 0.0)
        assert lo - 5e-4 <= r["rel"] <= hi + 5e-4, name
        assert abs(r["ppl"] / dense["ppl"] - r["rel"]) <= 6e-4, name
        assert metrics.delta_ce(r["ce"], dense["ce"]) == pytest.approx(r["dce"],
                                                                       abs=1e-9)


# ------------------------------------------------------- P10 / P11 storage

def test_group_int4_storage_ratio_matches_paper():
    rows = fixtures.paper_metric_rows()
    V, d = 151936, 4096
    ratio = obytes.packed_bytes(V, d, 64, 0, 0) / obytes.dense_bf16_bytes(V, d)
    assert ratio == 0.265625
    assert round(ratio, 4) == rows["group_int4"]["ratio"]


def test_paper_storage_table_reproduced():
    Mi = 2 ** 20
    for name, r in fixtures.paper_storage_rows().items():
        dense = obytes.dense_bf16_bytes(r["V"], r["D"]) / Mi
        assert round(dense, 1) == r["dense"], name
        assert round(r["dense"] / r["packed"], 3) == pytest.approx(r["ratio"],
                                                                   abs=1.5e-3)
        # INT4 residual, one byte of scale per 128 weights, r_c = 10 5-bit
        # left codes, INT8 right codes, r_r = 6 INT8 correction, fp16 row scales
        packed = obytes.packed_bytes(r["V"], r["D"], 64, 10, 6, res_scale_bits=4,
                                     core_u_bits=5) / Mi
        if name == "gemma4_e4b":   # matches fp16 scales per 64 weights instead
            packed = obytes.packed_bytes(r["V"], r["D"], 64, 10, 6,
                                         core_u_bits=5) / Mi
            assert abs(packed - r["packed"]) < 1.4, (name, packed)
        else:
            assert abs(packed - r["packed"]) < 0.2, (name, packed)


@pytest.mark.parametrize("cfg,expect", [
    ("tiny", 3_096_768), ("qwen_decode", 336_475_840), ("gemma", 372_490_432),
    ("sweep128k", 568_464_768)])
def test_config_packed_bytes(cfg, expect):
    from synth import CONFIGS
    c = CONFIGS[cfg]
    V, d, g, rc, rr = c["V"], c["d"], c["g"], c["rc"], c["rr"]
    per_buffer = [V * d // 2, V * (d // g) * 2, V * rc, V * 2, rc * d, rc * 2,
                  V * rr, V * 2, rr * d, rr * 2]
    assert sum(per_buffer) == expect
    assert obytes.packed_bytes(V, d, g, rc, rr) == expect


def test_8bit_scale_codes_decode_exactly():
    """8-bit residual scale codes (the "quantized group scales" of the
    paper's packed-buffer table, read as q * rs with an fp16 row scale):
    the oracle's scales are exactly rs * q, the generator's codes stay within
    half a step of the fp16 draws, and a one-hot x gives logits equal to the
    exact rational rs * q * c."""
    from fractions import Fraction
    h16 = make_head("tiny", V=64, d=128, g=64, rc=0, rr=0)
    h8 = make_head("tiny", V=64, d=128, g=64, rc=0, rr=0, scales="u8")
    assert h8.res_scales.dtype == np.uint8 and h8.res_row_scales.dtype == np.float16
    rs = h8.res_row_scales.astype(np.float64)
    s8 = ohead.residual_scales(h8, 0, h8.V)
    assert np.array_equal(s8, rs[:, None] * h8.res_scales.astype(np.float64))
    s16 = h16.res_scales.astype(np.float64)
    assert np.all(np.abs(s8 - s16) <= rs[:, None] / 2 + 1e-3 * s16)
    codes = layout.unpack_int4(h8.res_codes, h8.d)
    for col in (0, 63, 64, 127):
        x = np.zeros((1, h8.d), dtype=np.uint16)
        x[0, col] = 0x3F80
        lg = ohead.logits(h8, x)[0]
        for v in (0, 7, 63):
            exact = (Fraction(float(h8.res_row_scales[v])) * int(h8.res_scales[v, col // h8.g])
                     * int(codes[v, col]))
            assert Fraction(lg[v]) == exact



# ------------------------------------------------ P12 logit fidelity metrics

def _softmax64(z):
    from scipy.special import softmax
    return softmax(np.asarray(z, dtype=np.float64), axis=-1)


def test_fidelity_kl_matches_library_relative_entropy():
    """KL(p_ref || p_test) against scipy's relative entropy of the two
    softmax distributions; the reverse direction differs (asymmetric
    case), so swapped operands fail."""
    from scipy.stats import entropy
    rng = np.random.default_rng(21)
    a = 3.0 * rng.standard_normal((6, 37))
    b = a + rng.standard_normal((6, 37))
    kl, _, _, _ = metrics.logit_fidelity(a, b)
    for m in range(6):
        want = entropy(_softmax64(a[m]), _softmax64(b[m]))
        rev = entropy(_softmax64(b[m]), _softmax64(a[m]))
        assert kl[m] == pytest.approx(want, rel=1e-12, abs=1e-15)
        assert abs(want - rev) > 1e-3 * want


def test_fidelity_kl_two_token_closed_form():
    """V = 2: the softmax of [0, s] is Bernoulli(sigmoid(s)), whose KL has a
    closed form."""
    for s, t in [(0.3, -1.2), (4.0, 2.5), (-7.0, 1.0)]:
        p, q = 1 / (1 + math.exp(-s)), 1 / (1 + math.exp(-t))
        want = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
        kl, _, _, _ = metrics.logit_fidelity(np.array([[0.0, s]]), np.array([[0.0, t]]))
        assert kl[0] == pytest.approx(want, rel=1e-12)


def test_fidelity_kl_zero_on_equal_and_shift_invariant():
    """KL is 0 for equal logits and does not change when a constant is added
    to one position's logits on either side (softmax is shift invariant); a
    dropped log-sum-exp term fails this."""
    rng = np.random.default_rng(22)
    a = 5.0 * rng.standard_normal((4, 100))
    b = a + 0.5 * rng.standard_normal((4, 100))
    kl0, sq0, _, _ = metrics.logit_fidelity(a, a)
    assert np.all(np.abs(kl0) < 1e-13) and np.all(sq0 == 0)
    kl, _, _, _ = metrics.logit_fidelity(a, b)
    assert np.all(kl > 0)
    shift = np.array([[3.0], [-40.0], [0.25], [900.0]])
    kl_a, _, _, _ = metrics.logit_fidelity(a + shift, b)
    kl_b, _, _, _ = metrics.logit_fidelity(a, b - shift)
    np.testing.assert_allclose(kl_a, kl, rtol=1e-9)
    np.testing.assert_allclose(kl_b, kl, rtol=1e-9)


def test_fidelity_squared_error_closed_form():
    """A constant offset c on every logit gives V c^2 per position."""
    a = np.random.default_rng(23).standard_normal((3, 50))
    _, sq, _, _ = metrics.logit_fidelity(a, a + 0.5)
    np.testing.assert_allclose(sq, 50 * 0.25, rtol=1e-12)


def test_fidelity_mse_is_the_activation_objective():
    """Mean over positions of the summed squared logit error equals
    Tr(Delta C Delta^T) with C = H^T H / N and Delta = W - W_hat, the
    objective of Eq. (1), computed here in its trace form."""
    rng = np.random.default_rng(24)
    N, V, D = 40, 30, 12
    H = rng.standard_normal((N, D))
    W = rng.standard_normal((V, D))
    Wh = W + 0.05 * rng.standard_normal((V, D))
    _, sq, _, _ = metrics.logit_fidelity(H @ W.T, H @ Wh.T)
    Dl = W - Wh
    C = H.T @ H / N
    assert metrics.fidelity_summary(np.zeros(N), sq, np.zeros(N))["mse"] == \
        pytest.approx(float(np.trace(Dl @ C @ Dl.T)), rel=1e-10)


def test_fidelity_rank_hand_fixture_with_ties():
    """ref's first maximum is index 1; in test, index 2 is larger and index 0
    ties with index 1 but comes first, so index 1 sits at rank 2."""
    ref = np.array([[0.0, 5.0, 5.0, 1.0], [1.0, 0.0, 0.0, 0.0], [2.0, 2.0, 2.0, 2.0]])
    test = np.array([[2.0, 2.0, 7.0, 2.0], [9.0, 9.0, 9.0, 9.0], [1.0, 3.0, 0.0, 3.0]])
    _, _, idx, rank = metrics.logit_fidelity(ref, test)
    assert idx.tolist() == [1, 0, 0]
    assert rank.tolist() == [2, 0, 2]


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 12), st.integers(0, 2 ** 31 - 1))
def test_fidelity_rank_brute_force_stable_sort(V, seed):
    """rank = position of the reference's first argmax in a stable
    descending sort of the test logits (a library sort), with values drawn
    from a small set so that ties are frequent; top-1 agreement equals
    equality of the two first-index argmaxes."""
    rng = np.random.default_rng(seed)
    a = rng.integers(-2, 3, size=(5, V)).astype(np.float64)
    b = rng.integers(-2, 3, size=(5, V)).astype(np.float64)
    _, _, idx, rank = metrics.logit_fidelity(a, b)
    for m in range(5):
        order = np.argsort(-b[m], kind="stable")
        assert idx[m] == ohead.argmax(a[m:m + 1])[0]
        assert rank[m] == int(np.nonzero(order == idx[m])[0][0])
    top1 = metrics.fidelity_summary(np.zeros(5), np.zeros(5), rank, ks=(1,))["top1"]
    assert top1 == pytest.approx(100.0 * np.mean(ohead.argmax(a) == ohead.argmax(b)))
