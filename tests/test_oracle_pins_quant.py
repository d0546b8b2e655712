"""Value pins of the oracle's quantizers and of its vocabulary-subset logits.

* ``construct.quantize_symmetric`` / ``dequantize`` against hand-worked
  groups (tests/golden/quantize_symmetric_v1.txt): 4, 5 and 8 bits, half-way
  values, a zero group, a negative absmax, and cases where rounding the scale
  to fp16 before the codes changes a code (paper Algorithm 2, QuantizeCore /
  QuantizeINT8).
* ``construct.quantize_core`` on a rank-1 head whose SVD, codes and scales
  are derived by hand (tests/golden/quantize_core_rank1_v1.txt), including
  the residual taken against the unquantized core (Section 3.2).
* ``head.logits(h, x, vocab=ids)`` equals the matching columns of the full
  logits bit for bit (fp16 and 8-bit scale heads, unsorted and repeated ids
  across chunk boundaries), and exact rationals on a few ids (Section 3.2,
  the inference equation evaluated per vocabulary row).
"""
from __future__ import annotations

import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import construct, head as ohead, layout
from synth import make_head, make_x
from tests.fixtures import GOLDEN


def _quant_cases():
    out = []
    with open(os.path.join(GOLDEN, "quantize_symmetric_v1.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            bits, vals, scale, codes = [p.strip() for p in line.split("|")]
            out.append((int(bits), np.array([float(v) for v in vals.split()]),
                        float(scale), np.array([int(c) for c in codes.split()])))
    return out


QUANT_CASES = _quant_cases()


def test_quant_fixture_is_complete():
    bits = {b for b, *_ in QUANT_CASES}
    assert bits == {4, 5, 8}
    assert any(s == 0.0 for _, _, s, _ in QUANT_CASES), "zero group"
    assert len(QUANT_CASES) >= 10


@pytest.mark.parametrize("case", range(len(QUANT_CASES)))
def test_quantize_symmetric_hand_worked(case):
    bits, vals, scale, codes = QUANT_CASES[case]
    c, s = construct.quantize_symmetric(vals[None, :], bits, vals.size)
    assert s.dtype == np.float16 and s.shape == (1, 1)
    assert float(s[0, 0]) == scale
    assert c.dtype == np.int8 and c[0].tolist() == codes.tolist()
    # dequantize: code times scale, exactly
    deq = construct.dequantize(c, s)
    assert deq[0].tolist() == [float(Fraction(int(k)) * Fraction(scale)) for k in codes]


def test_quantize_symmetric_groups_along_the_last_axis():
    """Several groups per row and several rows: each (row, group) is the
    hand-worked case placed there, so a grouping along the wrong axis or a
    shared scale fails."""
    picks = [QUANT_CASES[i] for i in range(len(QUANT_CASES))
             if QUANT_CASES[i][0] == 4 and QUANT_CASES[i][1].size == 4]
    assert len(picks) >= 3
    a, b, c = picks[:3]
    X = np.array([np.concatenate([a[1], b[1]]), np.concatenate([c[1], a[1]])])
    codes, scales = construct.quantize_symmetric(X, 4, 4)
    assert scales.shape == (2, 2)
    assert [float(v) for v in scales.ravel()] == [a[2], b[2], c[2], a[2]]
    assert codes.tolist() == [list(a[3]) + list(b[3]), list(c[3]) + list(a[3])]


def test_quantize_rounding_alternatives_fail_the_fixture():
    """The fixture discriminates: flooring, rounding half away from zero, or
    an unrounded scale each change at least one expected code."""
    def alt(vals, bits, mode):
        qmax = 2 ** (bits - 1) - 1
        amax = np.abs(vals).max()
        s = amax / qmax if mode == "unrounded" else float(np.float16(amax / qmax))
        if s == 0:
            return np.zeros(vals.size, dtype=int)
        r = vals / s
        if mode == "floor":
            q = np.floor(r + 0.5)
        elif mode == "half_away":
            q = np.sign(r) * np.floor(np.abs(r) + 0.5)
        else:
            q = np.rint(r)
        return np.clip(q, -qmax, qmax).astype(int)
    for mode in ("floor", "half_away", "unrounded"):
        assert any(alt(v, b, mode).tolist() != c.tolist() for b, v, _, c in QUANT_CASES), mode


def _core_fixture():
    vals = {}
    with open(os.path.join(GOLDEN, "quantize_core_rank1_v1.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = line.split(":")
                vals[k.strip()] = [float(t) for t in v.split()]
    return vals


def test_quantize_core_rank1_hand_worked():
    f = _core_fixture()
    W = np.array([f[f"W_row{i}"] for i in range(4)])
    W_d, out = construct.quantize_core(W, rc=1, g=4)
    cu = out["core_u"][:, 0].astype(int)
    cv = out["core_v"][0].astype(int)
    sign = 1 if cv[0] > 0 else -1          # the SVD's common sign
    assert (sign * cu).tolist() == [int(v) for v in f["core_u_codes_s"]]
    assert [float(v) for v in out["core_u_scale"][:, 0]] == f["core_u_scales"]
    assert (sign * cv).tolist() == [int(v) for v in f["core_v_codes_s"]]
    assert [float(v) for v in out["core_v_scale"][:, 0]] == f["core_v_scale"]
    res = out["res_int4"].astype(int)
    for i in range(4):
        assert res[i].tolist() == [int(v) for v in f[f"res_codes_row{i}"]], i
        assert [float(v) for v in out["res_scales"][i]] == f[f"res_scales_row{i}"], i
    # W_d from the hand values: every entry is exact in fp64
    Au = np.array(f["core_u_codes_s"]) * np.array(f["core_u_scales"])
    Bv = np.array(f["core_v_codes_s"]) * f["core_v_scale"][0]
    R = np.array([np.array(f[f"res_codes_row{i}"]) *
                  np.repeat(f[f"res_scales_row{i}"], 4) for i in range(4)])
    assert np.array_equal(W_d, np.outer(Au, Bv) + R)


# ------------------------------------------------ logits on a vocabulary subset

@pytest.mark.parametrize("scales", ["f16", "u8"])
def test_logits_vocab_subset_equals_full_columns(scales):
    h = make_head("tiny", V=300, d=128, g=64, rc=8, rr=4, scales=scales)
    x = make_x("tiny", 3, d=128, basis="identity")
    full = ohead.logits(h, x, chunk=64)
    rng = np.random.default_rng(31)
    ids = np.concatenate([[299, 0, 63, 64, 65, 127, 128, 5, 5, 299],
                          rng.integers(0, h.V, 40)])       # unsorted, repeated
    for chunk in (7, 64, 4096):
        sub = ohead.logits(h, x, vocab=ids, chunk=chunk)
        assert sub.shape == (3, ids.size)
        assert np.array_equal(sub, full[:, ids]), chunk
    # the gathered rows carry their own row scales (8-bit codes) and factors
    if scales == "u8":
        assert h.res_row_scales is not None
        assert np.unique(h.res_row_scales[ids]).size > 1


def test_logits_vocab_subset_exact_rationals():
    """A few ids against exact rational arithmetic from the buffers."""
    h = make_head("tiny", V=50, d=64, g=32, rc=2, rr=1, scales="u8")
    x = make_x("tiny", 2, d=64, basis="identity")
    ids = np.array([49, 3, 3, 17])
    sub = ohead.logits(h, x, vocab=ids)
    codes = layout.unpack_int4(h.res_codes, h.d)
    xf = layout.bf16_to_f64(x)
    F = Fraction
    for m in range(2):
        for j, v in enumerate(ids):
            acc = F(0)
            for i in range(h.d):
                w = F(float(h.res_row_scales[v])) * int(h.res_scales[v, i // h.g]) * int(codes[v, i])
                for k in range(h.rc):
                    w += (F(float(h.core_u_scale[v])) * int(h.core_u[v, k]) *
                          F(float(h.core_v_scale[k, 0])) * int(h.core_v[k, i]))
                for k in range(h.rr):
                    w += (F(float(h.corr_a_scale[v])) * int(h.corr_a[v, k]) *
                          F(float(h.corr_b_scale[k, 0])) * int(h.corr_b[k, i]))
                acc += w * F(float(xf[m, i]))
            assert abs(float(acc) - sub[m, j]) <= 1e-13 * max(1.0, abs(float(acc)))
