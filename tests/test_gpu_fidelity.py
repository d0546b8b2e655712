"""GPU parity of the logit fidelity pass (archead_logit_fidelity) against the
oracle's definitions, on the same fp32 logit arrays.

Tolerances: ref_idx and rank bit-exact (both sides compare the same fp32
values); sq within 1e-6 relative (fp64 sums of exact fp64 differences, one
rounding to fp32); KL within 1e-5 (1 + max_v |ref - test|): the kernel's
fp32 exponentials carry ~1e-7 relative error into the two softmax sums and
the p-weighted difference sum, whose size is bounded by max |ref - test|.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import head as ohead, metrics
from synth import make_head, make_x
from tests.gpu_util import say, torch_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def run(ref, test, ld_pad=0, ld_pad_test=None):
    from paper_2608_02703_amd import logit_fidelity
    M, V = ref.shape
    if ld_pad:
        r = torch.zeros(M, V + ld_pad, dtype=torch.float32, device="cuda")
        pt = ld_pad + 3 if ld_pad_test is None else ld_pad_test
        t = torch.zeros(M, V + pt, dtype=torch.float32, device="cuda")
        r[:, :V] = torch.from_numpy(ref)
        t[:, :V] = torch.from_numpy(test)
        r, t = r[:, :V], t[:, :V]
    else:
        r = torch.from_numpy(ref).cuda()
        t = torch.from_numpy(test).cuda()
    kl, sq, idx, rank = logit_fidelity(r, t)
    torch.cuda.synchronize()
    return kl.cpu().numpy(), sq.cpu().numpy(), idx.cpu().numpy(), rank.cpu().numpy()


def check(ref, test, **kw):
    kl, sq, idx, rank = run(ref, test, **kw)
    okl, osq, oidx, orank = metrics.logit_fidelity(ref, test)
    assert np.array_equal(idx, oidx), "ref_idx"
    assert np.array_equal(rank, orank), "rank"
    np.testing.assert_allclose(sq, osq, rtol=1e-6, atol=0)
    dmax = np.abs(ref.astype(np.float64) - test.astype(np.float64)).max(axis=1)
    err = np.abs(kl.astype(np.float64) - okl)
    tol = 1e-5 * (1.0 + dmax)
    assert np.all(err <= tol), f"KL max err {err.max():.3e} (tol {tol.min():.3e})"
    return okl, orank


@pytest.mark.parametrize("V", [1, 63, 1000, 4097, 151936])
def test_fidelity_random_logits(V):
    """Gaussian logits of LM-head scale with a perturbation of a few percent
    (KL near the paper's 1e-2 range), several tiles of 512 lanes and a
    ragged tail."""
    rng = np.random.default_rng(V)
    M = 7
    ref = (4.0 * rng.standard_normal((M, V))).astype(np.float32)
    test = (ref + 0.3 * rng.standard_normal((M, V))).astype(np.float32)
    say(f"fidelity random V={V}")
    okl, _ = check(ref, test)
    if V > 1:
        assert np.all(okl > 0)


def test_fidelity_ties_and_equal_rows():
    """Integer-valued logits from a small set (frequent ties in both rows),
    one row equal to its reference (KL 0, rank 0) and one constant row."""
    rng = np.random.default_rng(5)
    M, V = 9, 3000
    ref = rng.integers(-3, 4, size=(M, V)).astype(np.float32)
    test = rng.integers(-3, 4, size=(M, V)).astype(np.float32)
    test[2] = ref[2]
    ref[4] = 1.0
    say("fidelity ties")
    check(ref, test)
    kl, sq, _, rank = run(ref, test)
    assert rank[2] == 0 and sq[2] == 0 and abs(kl[2]) < 1e-6


def test_fidelity_ties_across_chunks():
    """Equal maxima of the reference in different 8192-logit chunks (the
    first one wins), and test logits equal to the one at the reference's
    argmax before it in its own chunk, before it in an earlier chunk, and
    after it in a later chunk (only the first two count toward the rank);
    a maximum in the ragged tail of the last chunk."""
    rng = np.random.default_rng(8)
    M, V = 4, 3 * 8192 + 5
    ref = rng.standard_normal((M, V)).astype(np.float32)
    test = rng.standard_normal((M, V)).astype(np.float32)
    ref[0, [9000, 20000]] = 50.0
    test[0, [9000, 50, 8500, 24000]] = 30.0
    ref[1, [100, 8192 + 100, V - 1]] = 40.0
    test[1, 100] = 30.0
    ref[2, V - 2] = 60.0
    test[2, [0, V - 1]] = test[2, V - 2] = 30.0
    test[3] = ref[3]
    say("fidelity ties across chunks")
    _, rank = check(ref, test)
    kl, sq, idx, _ = run(ref, test)
    assert idx.tolist() == [9000, 100, V - 2, int(np.argmax(ref[3]))]
    assert rank[0] == 2 and rank[1] == 0 and rank[2] == 1 and rank[3] == 0


@pytest.mark.parametrize("pads", [(45, 48), (3, 7)])
def test_fidelity_strided_rows(pads):
    """Leading dimensions larger than V and different on the two sides: rows
    that start off 16-byte boundaries (element-wise walk), and rows that all
    start on them with a ragged tail of one element (16-byte walk)."""
    rng = np.random.default_rng(6)
    ref = (3.0 * rng.standard_normal((5, 2053))).astype(np.float32)
    test = (ref + 0.2 * rng.standard_normal(ref.shape)).astype(np.float32)
    say(f"fidelity strided {pads}")
    check(ref, test, ld_pad=pads[0], ld_pad_test=pads[1])


def test_fidelity_empty_is_noop():
    from paper_2608_02703_amd import logit_fidelity
    e = torch.empty(0, 10, dtype=torch.float32, device="cuda")
    kl, sq, idx, rank = logit_fidelity(e, e)
    torch.cuda.synchronize()
    assert kl.numel() == 0 and rank.numel() == 0


def test_fidelity_packed_head_against_its_oracle():
    """The packed head's own logits (HIP path, fp32) scored against the
    oracle's fp64 logits of the same head: agreement is near perfect (top-1
    differs only where the oracle's top-2 gap is within rounding), and the
    kernel's figures match the oracle's on the same arrays."""
    from oracle.metrics import fidelity_summary
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny")
    ph = PackedHead.from_arrays(h)
    x = make_x("tiny", 24)
    test = ph.logits(torch_x(x))
    torch.cuda.synchronize()
    ref = ohead.logits(h, x).astype(np.float32)
    say("fidelity packed head vs oracle logits")
    okl, orank = check(ref, test.cpu().numpy())
    assert np.all(okl < 1e-6)
    gap = ohead.top2_gap(ohead.logits(h, x))
    assert np.all(orank[gap > 1e-2] == 0)
    kl, sq, idx, rank = run(ref, test.cpu().numpy())
    s = fidelity_summary(kl, sq, rank)
    assert s["top10"] == 100.0
    ph.close()
