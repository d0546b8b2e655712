"""GPU tests of archead_prepare: the many-token kernel reading its
head-derived tables (scale ratios, final scales, bf16 V_c / B_w codes,
paired U_c / A_w codes) from a prepared buffer gives the same bits as the
same kernel rebuilding them in the workspace per call, and matches the
oracle.

Tolerances: prepared against per-call tables bit-exact (logits, CE, argmax:
the same kernels read the same values); against the oracle the logit and CE
bounds of the other parity tests.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import head as ohead
from synth import make_head, make_targets, make_x
from tests.gpu_util import assert_ce_close, assert_logits_close, say, torch_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _run(ph, x, y):
    lg = ph.logits(torch_x(x)).cpu().numpy()
    ce, mean = ph.logits_ce(torch_x(x), torch.from_numpy(y).cuda())
    idx, mx = ph.logits_argmax(torch_x(x))
    torch.cuda.synchronize()
    return lg, ce.cpu().numpy(), float(mean.cpu()[0]), idx.cpu().numpy()


@pytest.mark.parametrize("V,d,g,M,rc,rr,scales", [
    (1000, 512, 64, 130, 40, 12, "f16"),     # ragged token and vocabulary tiles
    (513, 192, 64, 300, 40, 12, "f16"),      # two token tiles
    (1000, 512, 64, 260, 16, 8, "u8"),       # 8-bit group scale codes
    (777, 256, 128, 40, 0, 32, "f16"),       # no core
    (777, 256, 64, 40, 20, 0, "f16"),        # no correction
])
def test_prepared_tables_bit_identical(V, d, g, M, rc, rr, scales):
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=rc, rr=rr, scales=scales)
    x = make_x("tiny", M, d=d)
    y = (np.arange(M) * 37 % V).astype(np.int64)
    ph = PackedHead.from_arrays(h)
    ph.force_path("tiled")
    say(f"prepared tables V={V} d={d} g={g} M={M} rc={rc} rr={rr} {scales}")
    base = _run(ph, x, y)
    ph.prepare()
    prep = _run(ph, x, y)
    again = _run(ph, x, y)            # the tables are read, never rewritten
    ph.prepare(False)
    detached = _run(ph, x, y)
    for name, r in (("prepared", prep), ("prepared, second call", again),
                    ("detached", detached)):
        assert np.array_equal(r[0].view(np.uint32), base[0].view(np.uint32)), f"{name} logits"
        assert np.array_equal(r[1].view(np.uint32), base[1].view(np.uint32)), f"{name} CE"
        assert r[2] == base[2], f"{name} mean CE"
        assert np.array_equal(r[3], base[3]), f"{name} argmax"
    ref = ohead.logits(h, x)
    assert_logits_close(prep[0], ref, what="prepared logits")
    assert_ce_close(prep[1], ohead.cross_entropy(ref, y), what="prepared CE")
    ph.close()


def test_prepared_qwen_prefill_ce_sampled():
    """The Qwen3-8B-shaped head with prepared tables: CE of 512 prefill
    tokens (Zipf targets) bit-identical to per-call tables, and the CE of a
    sample of tokens against the oracle."""
    from paper_2608_02703_amd import PackedHead
    from tests.gpu_util import cached_head
    h = cached_head("qwen_decode")
    M = 512
    x = make_x("qwen_prefill", M)
    y = make_targets("qwen_prefill", M)
    ph = PackedHead.from_arrays(h)
    say("prepared tables, Qwen-shaped prefill CE, M=512")
    t = torch.from_numpy(y).cuda()
    ce0, m0 = ph.logits_ce(torch_x(x), t)
    ph.prepare()
    ce1, m1 = ph.logits_ce(torch_x(x), t)
    torch.cuda.synchronize()
    a, b = ce0.cpu().numpy(), ce1.cpu().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert float(m0.cpu()[0]) == float(m1.cpu()[0])
    rows = np.array([0, 1, 255, 256, 511])
    ref = ohead.logits(h, x[rows])
    assert_ce_close(b[rows], ohead.cross_entropy(ref, y[rows]), what="prepared Qwen CE")
    ph.close()


def test_prepare_argument_errors():
    """Short and misaligned buffers are rejected before any launch and leave
    the head unprepared; a head with no many-token kernel (g % 64 != 0)
    reports 0 bytes and refuses a buffer."""
    from paper_2608_02703_amd import PackedHead, archead as ab
    h = make_head("tiny", V=300, d=256, g=64, rc=8, rr=4)
    ph = PackedHead.from_arrays(h)
    L = ab.lib()
    n = int(L.archead_prepared_bytes(ph.handle))
    assert n > 0 and n % 256 == 0
    buf = torch.empty(n + 512, dtype=torch.uint8, device="cuda")
    p = buf.data_ptr()
    assert L.archead_prepare(ph.handle, p, n - 1, None) == ab.E_WORKSPACE
    assert L.archead_prepare(ph.handle, p + 16, n, None) == ab.E_MISALIGNED
    assert L.archead_prepare(ph.handle, None, 4, None) == ab.E_INVALID_ARG
    assert L.archead_prepare(ph.handle, None, 0, None) == ab.OK
    ph.close()
    h32 = make_head("tiny", V=300, d=256, g=32, rc=8, rr=4)
    ph = PackedHead.from_arrays(h32)
    assert int(L.archead_prepared_bytes(ph.handle)) == 0
    assert L.archead_prepare(ph.handle, p, n, None) == ab.E_UNSUPPORTED
    ph.close()
