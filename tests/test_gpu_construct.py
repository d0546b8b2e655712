"""GPU construction of a packed head (archead_build_head) against the fp64
oracle's construction (paper Algorithm 2; Sections 3.1-3.2), through the C
ABI.

* Small shapes with well-separated spectra (so the truncated SVDs are well
  conditioned and the randomized SVD converges to the exact one): scales
  equal, codes equal except at quantizer near-ties, core and correction
  factors equal up to the sign of each rank component.
* V = 8192, d = 512 with the workload's power-law hidden-state spectrum: the
  unquantized correction's metric error ||(E - A_w B_w) T_p||_F^2 against
  the Eckart-Young-Mirsky tail of the exact SVD of E T_p (never below it, and
  within a small factor above it).
* The built head through archead_logits, against the oracle's logits of the
  same buffers.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import construct, head as ohead
from tests.gpu_util import assert_logits_close, say, torch_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _hidden(d, N, rng, gap_dims=0, alpha=1.5):
    """H ~ N(0, Sigma), Sigma with eigenvalues i^-alpha (the first gap_dims
    multiplied by 100) under a random orthogonal basis; fp32 values."""
    lam = np.arange(1, d + 1, dtype=np.float64) ** -alpha
    lam[:gap_dims] *= 100.0
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    return ((rng.standard_normal((N, d)) * np.sqrt(lam)) @ Q.T).astype(np.float32).astype(np.float64)


def _problem(V, d, N, seed, sigma_decay=1.0, gap_dims=0, alpha=1.5):
    """W with singular values 10 * i^-sigma_decay under random orthogonal
    bases (V >= d), and H from _hidden."""
    rng = np.random.default_rng(seed)
    Uw, _ = np.linalg.qr(rng.standard_normal((V, d)))
    Vw, _ = np.linalg.qr(rng.standard_normal((d, d)))
    sv = 10.0 * np.arange(1, d + 1, dtype=np.float64) ** -sigma_decay
    W = ((Uw * sv) @ Vw.T).astype(np.float32).astype(np.float64)
    return W, _hidden(d, N, rng, gap_dims, alpha)


def _gpu_build(W, H, **kw):
    from paper_2608_02703_amd import build_head
    Wt = torch.from_numpy(W.astype(np.float32)).cuda()
    Ht = torch.from_numpy(H.astype(np.float32)).cuda()
    ph, a_w, b_w = build_head(Wt, Ht, return_factors=True, **kw)
    torch.cuda.synchronize()
    host = {k: (None if v is None else v.cpu().numpy()) for k, v in ph.buffers.items()}
    return ph, host, (None if a_w is None else a_w.cpu().numpy()), \
        (None if b_w is None else b_w.cpu().numpy())


def _near_tie(vals, scales, group, qmax, tol=1e-7):
    """Positions whose value / scale lies within tol of a rounding boundary
    (a half-integer) or of the clip range: the quantizer may round either
    way there under fp64 rounding differences."""
    v = np.asarray(vals, dtype=np.float64)
    s = np.repeat(np.asarray(scales, dtype=np.float64).reshape(v.shape[0], -1), group, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(s > 0, v / s, 0.0)
    frac = np.abs(np.abs(r - np.trunc(r)) - 0.5)
    return (frac < tol * np.maximum(1.0, np.abs(r)))


def _rel_signs(got_rows, ref_rows):
    """Per rank component, the sign relating the GPU's factor row to the
    oracle's (an SVD fixes each singular pair only up to a common sign): the
    product of their signs at the oracle row's largest-magnitude entry."""
    ref_rows = np.asarray(ref_rows, dtype=np.float64)
    idx = np.argmax(np.abs(ref_rows), axis=1)
    r = np.arange(ref_rows.shape[0])
    s = np.sign(np.asarray(got_rows, dtype=np.float64)[r, idx]) * np.sign(ref_rows[r, idx])
    assert np.all(s != 0)
    return s


@pytest.mark.timeout(600)
@pytest.mark.parametrize("rc,rr,g,gB", [(8, 4, 64, 256), (0, 6, 32, 64), (5, 0, 64, 256)])
def test_build_matches_oracle_construction(rc, rr, g, gB):
    V, d, N = 2048, 256, 4096
    W, H = _problem(V, d, N, seed=3, gap_dims=max(rr, 1))
    kw = dict(rc=rc, rr=rr, g=g, p=0.75, lam=1e-3, gB=gB)
    say(f"construction V={V} d={d} N={N} rc={rc} rr={rr} g={g} gB={gB}")
    ph, got, a_w, b_w = _gpu_build(W, H, oversample=8, power_iters=6, **kw)
    ref, info = construct.build_head(W, H, rc=rc, rr=rr, g=g, p=0.75, lam=1e-3, gB=gB)
    # QuantizeCore: residual scales exact, codes exact away from near-ties
    from oracle import layout
    R = W - (info["A_c"] @ info["B_c"] if rc else 0.0)
    tie = _near_tie(R, ref.res_scales, g, 7)
    assert np.array_equal(got["res_scales"].view(np.uint16), ref.res_scales.view(np.uint16))
    gc = layout.unpack_int4(got["res_codes"], d)
    rc_ = layout.unpack_int4(ref.res_codes, d)
    bad = (gc != rc_) & ~tie
    assert not bad.any(), f"{bad.sum()} residual codes differ away from ties"
    say(f"  residual: {tie.sum()} near-tie positions of {tie.size}")
    if rc:
        sgn = _rel_signs(got["core_v"], info["B_c"])
        assert np.array_equal(got["core_u_scale"].view(np.uint16), ref.core_u_scale.view(np.uint16))
        assert np.array_equal(got["core_v_scale"].ravel().view(np.uint16),
                              ref.core_v_scale.ravel().view(np.uint16))
        tie_u = _near_tie(info["A_c"], ref.core_u_scale, rc, 15)
        bad_u = (got["core_u"] * sgn[None, :] != ref.core_u) & ~tie_u
        assert not bad_u.any(), f"{bad_u.sum()} core_u codes differ"
        tie_v = _near_tie(info["B_c"], ref.core_v_scale, d, 127)
        bad_v = (got["core_v"] * sgn[:, None] != ref.core_v) & ~tie_v
        assert not bad_v.any(), f"{bad_v.sum()} core_v codes differ"
    if rr:
        sgn = _rel_signs(b_w, info["B_w"])
        Aw = a_w * sgn[None, :]
        Bw = b_w * sgn[:, None]
        ea = np.abs(Aw - info["A_w"]).max() / np.abs(info["A_w"]).max()
        eb = np.abs(Bw - info["B_w"]).max() / np.abs(info["B_w"]).max()
        say(f"  correction factors vs exact SVD: rel err A_w {ea:.2e}, B_w {eb:.2e}")
        assert ea < 1e-8 and eb < 1e-8
        assert np.array_equal(got["corr_a_scale"].view(np.uint16), ref.corr_a_scale.view(np.uint16))
        assert np.array_equal(got["corr_b_scale"].view(np.uint16), ref.corr_b_scale.view(np.uint16))
        tie_a = _near_tie(info["A_w"], ref.corr_a_scale, rr, 127, tol=1e-6)
        bad_a = (got["corr_a"] * sgn[None, :] != ref.corr_a) & ~tie_a
        assert not bad_a.any(), f"{bad_a.sum()} corr_a codes differ"
        tie_b = _near_tie(info["B_w"], ref.corr_b_scale, gB, 127, tol=1e-6)
        bad_b = (got["corr_b"] * sgn[:, None] != ref.corr_b) & ~tie_b
        assert not bad_b.any(), f"{bad_b.sum()} corr_b codes differ"
    ph.close()


def _host_head(ph, got):
    import types
    h = types.SimpleNamespace(V=ph.V, d=ph.d, g=ph.g, rc=ph.rc, rr=ph.rr, gV=ph.gV, gB=ph.gB)
    empty = {"core_u": np.zeros((ph.V, 0), np.int8), "core_u_scale": np.zeros(ph.V, np.float16),
             "core_v": np.zeros((0, ph.d), np.int8), "core_v_scale": np.zeros((0, 1), np.float16),
             "corr_a": np.zeros((ph.V, 0), np.int8), "corr_a_scale": np.zeros(ph.V, np.float16),
             "corr_b": np.zeros((0, ph.d), np.int8), "corr_b_scale": np.zeros((0, 1), np.float16)}
    for k, v in got.items():
        if k == "res_row_scales":
            continue
        setattr(h, k, empty.get(k) if v is None else v)
    h.core_u_scale = np.asarray(h.core_u_scale).reshape(-1)
    h.corr_a_scale = np.asarray(h.corr_a_scale).reshape(-1)
    return h


@pytest.mark.timeout(900)
def test_build_eym_tail_and_forward_8192x512():
    V, d, N, rc, rr = 8192, 512, 4096, 16, 32
    rng = np.random.default_rng(11)
    W = (0.02 * rng.standard_normal((V, d))).astype(np.float32).astype(np.float64)
    H = _hidden(d, N, np.random.default_rng(12))
    say(f"construction V={V} d={d} N={N} rc={rc} rr={rr}: EYM tail")
    ph, got, a_w, b_w = _gpu_build(W, H, rc=rc, rr=rr, g=64, p=0.75, lam=1e-3, oversample=10,
                                   power_iters=4)
    h = _host_head(ph, got)
    W_d = np.concatenate([ohead.residual_rows(h, v0, min(V, v0 + 4096)) +
                          ohead.core_rows(h, v0, min(V, v0 + 4096))
                          for v0 in range(0, V, 4096)])
    E = W - W_d
    T, _ = construct.metric_transform(construct.damped_covariance(H, 1e-3), 0.75)
    ET = E @ T
    err = float(np.linalg.norm(ET - a_w @ (b_w @ T)) ** 2)
    ev = np.sort(np.linalg.eigvalsh(ET.T @ ET))[::-1]
    tail = float(ev[rr:].sum())
    say(f"  metric error {err:.6e}, exact tail {tail:.6e}, ratio {err / tail:.6f}, "
        f"captured {1 - err / float(ev.sum()):.4f} of ||E T_p||^2")
    assert err >= tail * (1 - 1e-9)
    assert err <= tail * 1.02
    # the built head through the forward kernels
    x = (rng.standard_normal((8, d)) * 0.05)
    from synth import f64_to_bf16_bits
    xb = f64_to_bf16_bits(x)
    lg = ph.logits(torch_x(xb))
    torch.cuda.synchronize()
    ref = ohead.logits(h, xb)
    e = assert_logits_close(lg.cpu().numpy(), ref, what="built head logits")
    say(f"  built head forward: max rel err {e:.2e}")
    ph.close()
