"""Pins of the oracle's top-k selection (oracle.metrics.topk), the reference
for archead_logits_topk: the candidate set of top-k decoding and of the
top-k agreement metric (Section 4, "Logit Fidelity", Table 8); and of the
oracle's dense bf16 head logits (oracle.head.dense_bf16_logits), the
reference side of the fidelity pass.

* hand-worked rows (tests/golden/topk_v1.txt): ties, NaN, -inf, signed
  zero, k = V and k = 1;
* brute force on tiny integer-valued rows with many ties: k rounds of
  "take the first index of the largest remaining value";
* k = 1 is the first-index argmax; the selected values are the k largest of
  the row as a multiset;
* agreement with the rank the fidelity metric reports: the reference's
  argmax token is in the test head's top k exactly when its rank is < k.
"""
from __future__ import annotations

import os

import numpy as np

from oracle import metrics

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "topk_v1.txt")


def _golden():
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, row, idx, vals = (p.split() for p in line.split(";"))
        yield (int(k[0]), np.array([float(v) for v in row]), np.array([int(i) for i in idx]),
               np.array([float(v) for v in vals]))


def test_topk_hand_worked():
    n = 0
    for k, row, idx, vals in _golden():
        v, i = metrics.topk(row[None, :], k)
        assert np.array_equal(i[0], idx), (row, k, i[0], idx)
        assert np.array_equal(v[0], vals), (row, k, v[0], vals)
        # signed zero: the value kept is the entry itself
        assert np.array_equal(np.signbit(v[0]), np.signbit(vals))
        n += 1
    assert n == 6


def _brute(row, k):
    left = [(float(v), j) for j, v in enumerate(row) if not np.isnan(v)]
    out = []
    for _ in range(k):
        if not left:
            out.append((-np.inf, -1))
            continue
        best = 0
        for t in range(1, len(left)):
            if left[t][0] > left[best][0]:     # strictly larger: the first index stays
                best = t
        out.append(left.pop(best))
    return out


def test_topk_brute_force_ties():
    rng = np.random.default_rng(3)
    for _ in range(200):
        V = int(rng.integers(1, 12))
        row = rng.integers(-3, 4, V).astype(np.float64)
        if rng.random() < 0.3:
            row[rng.integers(0, V)] = np.nan
        for k in range(1, V + 2):
            v, i = metrics.topk(row[None, :], k)
            want = _brute(row, k)
            assert [(float(a), int(b)) for a, b in zip(v[0], i[0])] == want, (row, k)


def test_topk_argmax_and_multiset():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((7, 500)).astype(np.float32)
    x[:, 100] = x[:, 7]            # exact ties across the row
    v, i = metrics.topk(x, 10)
    assert np.array_equal(i[:, 0], np.argmax(x, axis=1))
    assert np.array_equal(v, np.take_along_axis(x, i, axis=1))
    assert np.array_equal(np.sort(v, axis=1), np.sort(np.sort(x, axis=1)[:, -10:], axis=1))
    assert np.all(np.diff(v, axis=1) <= 0)
    assert v.dtype == np.float32


def test_topk_matches_fidelity_rank():
    rng = np.random.default_rng(5)
    ref = rng.standard_normal((40, 60))
    test = ref + 0.3 * rng.standard_normal((40, 60))
    test[::5, :] = np.round(test[::5, :])   # ties in some rows
    _, _, ref_idx, rank = metrics.logit_fidelity(ref, test)
    for k in (1, 2, 5, 10):
        _, i = metrics.topk(test, k)
        member = np.array([ref_idx[m] in i[m] for m in range(ref.shape[0])])
        assert np.array_equal(member, rank < k)


def test_dense_bf16_logits_exact_on_tiny():
    """oracle.head.dense_bf16_logits against exact rational dot products:
    bf16 values are dyadic rationals, so every logit has an exact value, which
    the fp64 result must match to its rounding."""
    from fractions import Fraction
    from oracle import head as ohead
    from oracle import layout
    rng = np.random.default_rng(6)
    V, d, M = 5, 9, 3
    def bits(shape):   # finite bf16 patterns of both signs, magnitudes ~2^-8 .. 2
        r = rng.integers(0, 2 ** 16, size=shape)
        return ((r & 0x3FFF) | 0x3C00 | (r & 0x8000)).astype(np.uint16)
    w_bits, x_bits = bits((V, d)), bits((M, d))
    got = ohead.dense_bf16_logits(w_bits, x_bits)
    w = layout.bf16_to_f64(w_bits)
    x = layout.bf16_to_f64(x_bits)
    for m in range(M):
        for v in range(V):
            exact = sum(Fraction(float(x[m, i])) * Fraction(float(w[v, i])) for i in range(d))
            assert abs(got[m, v] - float(exact)) <= 1e-14 * max(1.0, abs(float(exact)))
