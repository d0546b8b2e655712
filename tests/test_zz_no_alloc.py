"""archead_logits_noalloc (the entry point for callers that cannot allocate)
against archead_logits through the C ABI: bit-identical logits on two calls
in a row (the second with fewer tokens, and on another kernel), fp32 and
bf16 output, and the size limit of its static workspace."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

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


def _same_bits(a, b):
    a, b = a.cpu().numpy(), b.cpu().numpy()
    return a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("cfg,Ms", [("tiny", (8, 3)), ("qwen_decode", (16, 1)),
                                    ("qwen_decode", (32, 4))])
def test_noalloc_matches_workspace_call(cfg, Ms):
    from paper_2608_02703_amd import PackedHead
    h = make_head(cfg)
    ph = PackedHead.from_arrays(h)
    xall = make_x(cfg, max(Ms))
    for M in Ms:                                    # second call: smaller input
        x = torch_x(xall[:M])
        say(f"noalloc {cfg} M={M}")
        ref = ph.logits(x)
        got = ph.logits_noalloc(x)
        torch.cuda.synchronize()
        assert _same_bits(got, ref), f"{cfg} M={M}: noalloc differs from archead_logits"
        ref16 = ph.logits(x, out_dtype=torch.bfloat16)
        got16 = ph.logits_noalloc(x, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        assert _same_bits(got16.view(torch.int16), ref16.view(torch.int16))
    ph.close()


def test_noalloc_rejects_a_workspace_beyond_its_array():
    from paper_2608_02703_amd import PackedHead, archead as ab
    h = make_head("qwen_decode")
    ph = PackedHead.from_arrays(h)
    M = 4096                                        # the many-token path's tables
    assert ph.workspace_bytes(M) > ab.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((M, h.d), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((1, 1), device="cuda")
    L = ab.lib()
    st = L.archead_logits_noalloc(ph.handle, x.data_ptr(), M, h.d, out.data_ptr(), ab.F32,
                                  h.V, ctypes.c_void_p(0))
    assert st == ab.E_WORKSPACE
    assert b"static workspace" in L.archead_last_error()
    assert L.archead_logits_noalloc(ph.handle, x.data_ptr(), 0, h.d, 0, ab.F32, h.V,
                                    ctypes.c_void_p(0)) == ab.OK
    torch.cuda.synchronize()
    ph.close()
