"""GPU parity for the storage variants of the rank-r factors: ranks that are
not multiples of 4 and 5-bit core-left codes in ARCHEAD_I5 (the paper's
Q5(A_c), Section 3.2; its Qwen3-8B setting r_c = 10, r_r = 6, Section 4),
on every kernel, through the C ABI.

* Random heads and tokens through each kernel (forced) and the library's own
  choice: logits, CE, bf16 logits and the fused argmax against the oracle.
* An exact probe of the factor-code reads: residual codes all zero, V_c and
  B_w identity rows with unit scales, one-hot tokens at the rank dimensions,
  so every logit is the single product s_U[v] cU[v, j] (or s_A[v] cA[v, j]),
  exact in fp32: bit for bit on the decode GEMV, the MFMA decode and the
  several-token kernels; within the fp32 scale-chain bound on the tiled one.
* The Qwen3-8B-shaped head in the paper's storage (V = 151936, d = 4096,
  g = 64, 5-bit U_c, r_c = 10, r_r = 6, 8-bit residual scale codes) on
  sampled columns at M = 1, 16, 40 and 130, and its CE at M = 4096.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest

from oracle import head as ohead
from synth import make_head, make_targets, make_x
from tests.gpu_util import (assert_bf16_output, assert_ce_close, assert_logits_close, say,
                            torch_x)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def gpu_logits(ph, x_bits, out_dtype=None):
    lg = ph.logits(torch_x(x_bits), out_dtype=out_dtype)
    torch.cuda.synchronize()
    if lg.dtype == torch.bfloat16:
        return lg.view(torch.int16).cpu().numpy().view(np.uint16)
    return lg.cpu().numpy()


HEADS = [  # (V, d, g, rc, rr, core_u, scales)
    (1000, 512, 64, 10, 6, "i5", "f16"),
    (777, 1024, 128, 10, 6, "i8", "u8"),
    (1000, 512, 128, 64, 32, "i5", "f16"),
    (513, 512, 64, 7, 5, "i8", "f16"),
    (1500, 1024, 64, 13, 3, "i5", "u8"),
    (300, 512, 64, 10, 0, "i5", "f16"),
    (300, 512, 64, 0, 6, "i8", "f16"),
]


@pytest.mark.parametrize("V,d,g,rc,rr,cu,scales", HEADS)
def test_general_factor_codes_every_kernel(V, d, g, rc, rr, cu, scales):
    from paper_2608_02703_amd import PackedHead
    h = make_head("tiny", V=V, d=d, g=g, rc=rc, rr=rr, core_u=cu, scales=scales)
    ph = PackedHead.from_arrays(h)
    try:
        for path, Ms in (("gemv", (1, 3)), ("dec", (5, 16)), ("mid", (21, 40)),
                         ("tiled", (70,)), ("auto", (2, 33))):
            ph.force_path(path)
            for M in Ms:
                x = make_x("tiny", M, d=d, basis="identity")
                ref = ohead.logits(h, x)
                say(f"factor codes V={V} d={d} g={g} rc={rc} rr={rr} {cu} {scales}: {path} M={M}")
                lg = gpu_logits(ph, x)
                assert_logits_close(lg, ref, what=f"{path} M={M}")
                y = (np.arange(M) * 7 % V).astype(np.int32)
                ce, _ = ph.logits_ce(torch_x(x), torch.from_numpy(y).cuda())
                torch.cuda.synchronize()
                assert_ce_close(ce.cpu().numpy(), ohead.cross_entropy(ref, y), what=f"{path} CE")
                idx, mx = ph.logits_argmax(torch_x(x))
                torch.cuda.synchronize()
                assert np.array_equal(idx.cpu().numpy(), np.argmax(lg, axis=1))
                bits = gpu_logits(ph, x, out_dtype=torch.bfloat16)
                assert_bf16_output(bits, lg, ref, f"{path} M={M} bf16")
    finally:
        ph.close()


def _probe_head(V, d, g, rc, rr, cu, seed=0):
    """Residual codes all zero (nibble 8), V_c = [I_rc | 0] and B_w = identity
    on columns rc .. rc + rr - 1, unit V_c / B_w scales; random U_c / A_w codes
    and row scales."""
    h = make_head("tiny", V=V, d=d, g=g, rc=rc, rr=rr, core_u=cu, draw=seed)
    cv = np.zeros((rc, d), np.int8)
    cv[np.arange(rc), np.arange(rc)] = 1
    cb = np.zeros((rr, d), np.int8)
    cb[np.arange(rr), rc + np.arange(rr)] = 1
    return dataclasses.replace(
        h, res_codes=np.full_like(h.res_codes, 0x88), core_v=cv,
        core_v_scale=np.ones((rc, 1), np.float16), corr_b=cb,
        corr_b_scale=np.ones((rr, 1), np.float16))


@pytest.mark.parametrize("rc,rr,cu", [(10, 6, "i5"), (13, 3, "i5"), (7, 5, "i8"),
                                      (64, 32, "i5")])
def test_factor_code_probe_exact(rc, rr, cu):
    from paper_2608_02703_amd import PackedHead
    V, d, g = 1000, 512, 64
    h = _probe_head(V, d, g, rc, rr, cu)
    cols = np.arange(rc + rr)
    x = np.zeros((cols.size, d), dtype=np.uint16)
    x[np.arange(cols.size), cols] = 0x3F80
    ref = ohead.logits(h, x)
    # every logit is one product of a factor code and its row scale
    from oracle import layout
    cuv = layout.unpack_int5(h.core_u, rc) if cu == "i5" else h.core_u
    expect = np.concatenate([(h.core_u_scale.astype(np.float64)[:, None] * cuv).T,
                             (h.corr_a_scale.astype(np.float64)[:, None] * h.corr_a).T])
    assert np.array_equal(ref, expect)
    ph = PackedHead.from_arrays(h)
    try:
        for path in ("gemv", "dec", "mid", "tiled"):
            ph.force_path(path)
            say(f"factor-code probe rc={rc} rr={rr} {cu}: {path}")
            rows = x if path != "gemv" else x[:8]
            lg = gpu_logits(ph, rows).astype(np.float64)
            want = ref[:rows.shape[0]]
            if path == "tiled":
                # the accumulator is carried in units of the current slot's
                # scale: a few fp32 ratio roundings per logit
                rel = np.abs(lg - want) / np.maximum(np.abs(want), 1e-30)
                assert np.all((want == 0) <= (np.abs(lg) < 1e-12))
                assert rel[want != 0].max() <= 8 * 2.0 ** -24
            else:
                bad = np.argwhere(lg != want)
                assert bad.size == 0, (f"{path}: {len(bad)} logits differ, first {bad[0]}: "
                                       f"{lg[tuple(bad[0])]!r} vs {want[tuple(bad[0])]!r}")
    finally:
        ph.close()


@pytest.mark.timeout(900)
def test_paper_qwen_storage_head():
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode", g=64, rc=10, rr=6, core_u="i5", scales="u8")
    ph = PackedHead.from_arrays(h)
    rng = np.random.default_rng(14)
    ids = np.unique(np.concatenate([[0, 1, h.V - 1], rng.integers(0, h.V, 600)]))
    x_all = make_x("qwen_decode", 130)
    ref_all = ohead.logits(h, x_all, vocab=ids)
    for M in (1, 16, 40, 130):
        say(f"paper-storage qwen head (g=64, I5 r_c=10, r_r=6, 8-bit scales): M={M}")
        lg = gpu_logits(ph, x_all[:M])[:, ids]
        assert_logits_close(lg, ref_all[:M], what=f"paper storage M={M}")
    M = 4096
    x = make_x("qwen_prefill", M)
    y = make_targets("qwen_prefill", M)
    ce, mean = ph.logits_ce(torch_x(x), torch.from_numpy(y).cuda())
    torch.cuda.synchronize()
    ce = ce.cpu().numpy()
    rows = np.unique(np.concatenate([[0, M - 1], rng.integers(0, M, 14)]))
    ref = ohead.cross_entropy(ohead.logits(h, x[rows]), y[rows])
    err = assert_ce_close(ce[rows], ref, what="paper storage CE M=4096")
    say(f"  CE at M=4096 on {rows.size} sampled tokens: max |dCE| {err:.2e}")
    ph.close()


@pytest.mark.timeout(900)
def test_qwen_g64_fp16_scales_gemv():
    """A Qwen-shaped head with groups of 64 and fp16 scales (the reading of
    the paper's Gemma storage figure): 64 group scales per row take 32-lane
    segments on the decode GEMV, and the MFMA decode kernels read the groups
    in pairs.  Sampled columns at M = 1 (GEMV), 2, 8, 16 (k_dec) and 32."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode", g=64)
    ph = PackedHead.from_arrays(h)
    try:
        rng = np.random.default_rng(15)
        ids = np.unique(np.concatenate([[0, 1, 127, 128, h.V - 1], rng.integers(0, h.V, 600)]))
        x = make_x("qwen_decode", 32)
        ref = ohead.logits(h, x, vocab=ids)
        for M in (1, 2, 8, 16, 32):
            say(f"qwen g=64 fp16 scales: M={M}")
            lg = gpu_logits(ph, x[:M])
            assert_logits_close(lg[:, ids], ref[:M], what=f"g64 fp16 M={M}")
    finally:
        ph.close()
