"""GPU parity of archead_logit_fidelity_head: KL, squared logit error, the
dense head's top-1 and its rank among the packed logits, computed inside the
packed head's tile pass against a dense bf16 head (Section 4, "Logit
Fidelity", Table 8), through the C ABI.

Against the oracle (oracle.metrics.logit_fidelity on the fp64 logits of the
dense head, oracle.head.dense_bf16_logits, and of the packed head):
KL within 1e-4 + 1e-3 KL, the squared error within 1e-3 relative, the
top-1 index equal wherever the dense head's top two logits are further apart
than the logit tolerance.  The rank is an integer decision on the packed
head's fp32 logits, so it is checked exactly against those logits
(archead_logits, the same per-element arithmetic) and the GPU's own top-1.
Dense heads near the packed one (small KL, top-1 mostly kept) and unrelated
to it (large KL); ragged vocabulary and token tiles; 8-bit scales and 5-bit
U_c; a dense head with a row stride wider than d; the Qwen3-8B shape.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import head as ohead
from oracle import metrics
from synth import f64_to_bf16_bits, make_head, make_x
from tests.gpu_util import LOGIT_TOL, say, torch_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _dense_near(h, eps, seed=0):
    """bf16 rows of the packed head's dense weights plus relative noise eps
    (eps = None: an unrelated random head of the same scale)."""
    w = ohead.dense_rows(h, 0, h.V)
    rng = np.random.default_rng(seed)
    n = rng.standard_normal(w.shape) * w.std()
    return f64_to_bf16_bits(n if eps is None else w + eps * n)


def _dense_torch(bits, ld=None):
    V, d = bits.shape
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()
    if ld is None or ld == d:
        return t
    buf = torch.zeros((V, ld), dtype=torch.bfloat16, device="cuda")
    buf[:, :d] = t
    return buf[:, :d]


def _check(ph, h, w_bits, x, what, ld=None):
    xt = torch_x(x)
    kl, sq, idx, rank = ph.logit_fidelity_head(xt, _dense_torch(w_bits, ld))
    lg = ph.logits(xt)
    torch.cuda.synchronize()
    kl, sq, idx, rank = (t.cpu().numpy() for t in (kl, sq, idx, rank))
    lg = lg.cpu().numpy()
    ref = ohead.dense_bf16_logits(w_bits, x)
    test = ohead.logits(h, x)
    okl, osq, oidx, _ = metrics.logit_fidelity(ref, test)
    assert np.all(np.abs(kl - okl) <= 1e-4 + 1e-3 * np.abs(okl)), \
        f"{what}: KL {kl[:4]} vs oracle {okl[:4]}"
    assert np.all(np.abs(sq - osq) <= 1e-3 * np.abs(osq) + 1e-3), f"{what}: sq {sq[:4]} vs {osq[:4]}"
    top = ref.max(axis=1)
    clear = ohead.top2_gap(ref) > 2 * LOGIT_TOL * (1 + np.abs(top))
    bad = np.nonzero(clear & (idx != oidx))[0]
    assert bad.size == 0, f"{what}: top-1 differs at tokens {bad[:5]}"
    # rank: exactly the count over the packed head's own fp32 logits
    for m in range(x.shape[0]):
        b = lg[m, idx[m]]
        want = int(np.count_nonzero(lg[m] > b) + np.count_nonzero(lg[m, :idx[m]] == b))
        assert rank[m] == want, f"{what}: token {m} rank {rank[m]} vs {want}"
    return okl, idx, rank


@pytest.mark.parametrize("label,kw,eps", [
    ("near", {}, 0.02),
    ("unrelated", {}, None),
    ("u8 scales", dict(scales="u8"), 0.05),
    ("i5 rc10 rr6 g64", dict(rc=10, rr=6, core_u="i5", scales="u8"), 0.02),
    ("ragged V", dict(V=1000), 0.02),
])
def test_fidelity_head_matches_oracle(label, kw, eps):
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", **kw)
    w_bits = _dense_near(h, eps)
    ph = PackedHead.from_arrays(h)
    try:
        x_all = make_x("tiny", 130, d=h.d)
        for M in (1, 37, 64, 130):
            say(f"fidelity head {label}: M={M}")
            okl, idx, rank = _check(ph, h, w_bits, x_all[:M], f"{label} M={M}")
        if eps is not None:
            assert okl.max() < 0.5 and np.mean(rank == 0) > 0.5, "near head: small KL, top-1 kept"
        else:
            assert okl.mean() > 0.5
        say(f"fidelity head {label}: strided dense rows")
        _check(ph, h, w_bits, x_all[:37], f"{label} strided", ld=h.d + 24)
    finally:
        ph.close()


def test_fidelity_head_argument_checks():
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=300)
    ph = PackedHead.from_arrays(h)
    try:
        xt = torch_x(make_x("tiny", 2, d=h.d))
        w = _dense_torch(_dense_near(h, 0.02))
        with pytest.raises(RuntimeError):      # ldw % 8 != 0
            ph.logit_fidelity_head(xt, torch.zeros((h.V, h.d + 4), dtype=torch.bfloat16,
                                                   device="cuda")[:, :h.d])
        kl, sq, idx, rank = ph.logit_fidelity_head(xt[:0], w)   # M = 0
        assert kl.numel() == 0
    finally:
        ph.close()
    hg = make_head("tiny", V=300, g=32)                           # no tiled kernel
    pg = PackedHead.from_arrays(hg)
    try:
        with pytest.raises(RuntimeError):
            pg.logit_fidelity_head(torch_x(make_x("tiny", 2, d=hg.d)), _dense_torch(_dense_near(hg, 0.02)))
    finally:
        pg.close()


@pytest.mark.timeout(900)
def test_fidelity_head_qwen_shape():
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode")
    say("fidelity head qwen: dense head")
    w_bits = _dense_near(h, 0.02)
    ph = PackedHead.from_arrays(h)
    try:
        x = make_x("qwen_decode", 8)
        say("fidelity head qwen: M=8")
        _check(ph, h, w_bits, x, "qwen M=8")
    finally:
        ph.close()
