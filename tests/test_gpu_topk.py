"""GPU parity of archead_logits_topk (top-k selection; the candidate set of
top-k decoding and of the top-k agreement metric, Section 4 "Logit
Fidelity", Table 8) against the oracle's selection, through the C ABI.

The selection is an integer decision taken on the kernel's fp32 logits, so
the oracle selects over those same logits (archead_logits for the same M and
path): indices and values must match bit for bit, ties included.  Against
the oracle's fp64 logits the indices must agree wherever the order is
decided by more than the logit tolerance; where they differ, the two
entries' fp64 logits must lie within that tolerance of each other.

Cases: every kernel (forced) and the library's choice, M = 1 (the fused
single-token GEMV), small M on the decode kernels, several token tiles, and
M = 300 (two chunks of the unfused path, the second ragged); k = 1, 10, 64;
8-bit scale codes, 5-bit core-left codes with ranks 10 / 6, a ragged V;
vocabulary rows duplicated so that exact ties land in the top k; and the
Qwen3-8B-shaped head at M = 1 against the full fp64 oracle logits.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest

from oracle import head as ohead
from oracle import metrics
from synth import make_head, make_x
from tests.gpu_util import LOGIT_TOL, say, torch_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _duplicate_rows(h, src, dst):
    """The head with vocabulary rows dst replaced by copies of row src
    (bit-identical logits for every token)."""
    rep = {}
    for name in ("res_codes", "res_scales", "core_u", "core_u_scale", "corr_a",
                 "corr_a_scale", "res_row_scales"):
        a = getattr(h, name)
        if a is None or a.shape[0] != h.V:
            continue
        a = a.copy()
        a[dst] = a[src]
        rep[name] = a
    return dataclasses.replace(h, **rep)


def _check(ph, x_bits, k, ref=None, what=""):
    xt = torch_x(x_bits)
    lg = ph.logits(xt)
    vals, idx = ph.logits_topk(xt, k)
    torch.cuda.synchronize()
    lg, vals, idx = lg.cpu().numpy(), vals.cpu().numpy(), idx.cpu().numpy()
    ov, oi = metrics.topk(lg, k)
    bad = np.argwhere(idx != oi)
    assert bad.size == 0, (f"{what} k={k}: {len(bad)} indices differ, first {bad[0]}: "
                           f"{idx[tuple(bad[0])]} vs {oi[tuple(bad[0])]}")
    assert np.array_equal(vals.view(np.uint32), ov.view(np.uint32)), f"{what} k={k}: values"
    if ref is not None:
        _, ri = metrics.topk(ref, k)
        for m, j in np.argwhere(idx != ri):
            a, b = ref[m, idx[m, j]], ref[m, ri[m, j]]
            assert abs(a - b) <= 2 * LOGIT_TOL * (1 + max(abs(a), abs(b))), \
                f"{what} k={k}: token {m} slot {j}: {idx[m, j]} vs oracle {ri[m, j]} ({a} vs {b})"


HEADS = [  # (label, make_head overrides)
    ("tiny", {}),
    ("u8 scales", dict(scales="u8")),
    ("i5 rc10 rr6 g64", dict(rc=10, rr=6, core_u="i5", scales="u8")),
    ("ragged V", dict(V=1000)),
]


@pytest.mark.parametrize("label,kw", HEADS)
def test_topk_every_kernel(label, kw):
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", **kw)
    ph = PackedHead.from_arrays(h)
    try:
        x_all = make_x("tiny", 300, d=h.d)
        ref_all = ohead.logits(h, x_all[:40])
        for path, Ms in (("auto", (1, 2, 40, 300)), ("gemv", (1, 3)), ("dec", (5,)),
                         ("mid", (21,)), ("tiled", (1, 70))):
            ph.force_path(path)
            for M in Ms:
                for k in (1, 10, 64):
                    say(f"top-k {label}: {path} M={M} k={k}")
                    ref = ref_all[:M] if M <= 40 else None
                    _check(ph, x_all[:M], k, ref, f"{label} {path} M={M}")
    finally:
        ph.close()


def test_topk_exact_ties():
    from paper_2608_02703_amd import PackedHead
    h0 = make_head("tiny")
    x = make_x("tiny", 8)
    top = int(np.argmax(ohead.logits(h0, x[:1])[0]))
    V = h0.V
    dst = np.array(sorted({0, 1, top + 1 if top + 1 < V else top - 1, 4097, V - 1} - {top}))
    h = _duplicate_rows(h0, top, dst)
    ph = PackedHead.from_arrays(h)
    try:
        for path, M in (("gemv", 1), ("auto", 1), ("dec", 8), ("mid", 8), ("tiled", 8)):
            ph.force_path(path)
            say(f"top-k ties: {path} M={M}")
            xt = torch_x(x[:M])
            vals, idx = ph.logits_topk(xt, 10)
            torch.cuda.synchronize()
            idx = idx.cpu().numpy()
            # token 0: the tied copies lead, in index order
            want = np.array(sorted(list(dst) + [top]))
            assert np.array_equal(idx[0, :want.size], want), (path, idx[0], want)
            _check(ph, x[:M], 10, what=f"ties {path}")
    finally:
        ph.close()


@pytest.mark.timeout(900)
def test_topk_qwen_single_token_fused():
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode")
    ph = PackedHead.from_arrays(h)
    try:
        x = make_x("qwen_decode", 1)
        say("top-k qwen M=1 (fused GEMV): oracle logits")
        ref = ohead.logits(h, x)
        for k in (1, 10, 64):
            say(f"top-k qwen M=1 k={k}")
            _check(ph, x, k, ref, "qwen M=1")
    finally:
        ph.close()


def test_topk_argument_checks():
    from paper_2608_02703_amd import PackedHead
    from paper_2608_02703_amd import archead as ab
    h = make_head("tiny", V=50)
    ph = PackedHead.from_arrays(h)
    try:
        xt = torch_x(make_x("tiny", 2, d=h.d))
        for k in (0, 51, 65):
            with pytest.raises(RuntimeError):
                ph.logits_topk(xt, k)
        vals, idx = ph.logits_topk(xt, 50)   # k = V: the whole row, sorted
        torch.cuda.synchronize()
        lg = ph.logits(xt).cpu().numpy()
        _, oi = metrics.topk(lg, 50)
        assert np.array_equal(idx.cpu().numpy(), oi)
        assert ab.TOPK_MAX == 64
    finally:
        ph.close()
