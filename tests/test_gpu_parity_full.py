"""Full-size GPU parity against the fp64 oracle, through the C ABI.

* Qwen3-8B-shaped prefill / perplexity workload: all 4096 per-token CE values
  and their mean against the oracle's (tests/golden/qwen_prefill_ce_v1.txt,
  written by the committed oracle-only script beside it), |dCE| <= 1e-4.
* The 128k-vocabulary head: every vocabulary column at every M of its sweep.
* The decode GEMV at one token (the kernel the M = 1 decode step runs) on the
  Qwen-shaped head, bit for bit: one-hot tokens (no low-rank parts) make every
  logit the exact product s_res * c, with fp16 and with 8-bit scale codes.
* The residual stream alone (r_c = r_r = 0) at one token on random x, against
  an fp32 rounding bound derived from the head and x (far tighter than the
  2e-3 (1 + |l|) logit tolerance, which the residual's small share of the
  logits would otherwise leave loose).
"""
from __future__ import annotations

import hashlib
import os

import numpy as np
import pytest

from oracle import head as ohead
from oracle import layout
from synth import CONFIGS, make_head, make_targets, make_x
from tests.fixtures import GOLDEN
from tests.gpu_util import (CE_TOL, assert_ce_close, assert_logits_close, cached_head, say,
                            torch_x)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _golden_prefill_ce():
    vals, meta = [], {}
    with open(os.path.join(GOLDEN, "qwen_prefill_ce_v1.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            if ":" in line:
                k, v = line.split(":", 1)
                meta[k.strip()] = v.strip()
            else:
                vals.append(float(line))
    return np.array(vals), meta


@pytest.mark.timeout(900)
@pytest.mark.parametrize("prepared", [False, True])
def test_ce_parity_qwen_prefill_full(prepared):
    from paper_2608_02703_amd import PackedHead
    ref, meta = _golden_prefill_ce()
    cfg = "qwen_prefill"
    M = CONFIGS[cfg]["Ms"][0]
    x = make_x(cfg, M)
    y = make_targets(cfg, M)
    assert int(meta["tokens"]) == M == ref.size
    assert hashlib.sha256(np.ascontiguousarray(x).tobytes()).hexdigest() == meta["x_sha256"], \
        "the generator drew different hidden states than the golden file's"
    assert hashlib.sha256(y.astype(np.int32).tobytes()).hexdigest() == meta["targets_sha256"]
    ph = PackedHead.from_arrays(cached_head("qwen_decode"))
    if prepared:
        ph.prepare()
    say(f"prefill CE M={M}, all tokens (prepared tables: {prepared})")
    ce, mean = ph.logits_ce(torch_x(x), torch.from_numpy(y).cuda())
    torch.cuda.synchronize()
    ce = ce.cpu().numpy()
    mean = float(mean.cpu().numpy()[0])
    err = assert_ce_close(ce, ref, what="prefill CE, all 4096 tokens")
    ref_mean = float(meta["mean_ce"])
    assert abs(mean - ref_mean) <= CE_TOL, (mean, ref_mean)
    say(f"  max |dCE| {err:.2e}; mean CE {mean:.6f} vs oracle {ref_mean:.6f}")
    ph.close()


@pytest.mark.timeout(1200)
def test_logits_parity_sweep128k_all_columns():
    cfg = "sweep128k"
    from paper_2608_02703_amd import PackedHead
    h = cached_head(cfg)
    Ms = CONFIGS[cfg]["Ms"]
    x_all = make_x(cfg, max(Ms))
    say(f"sweep128k: oracle logits for M={max(Ms)} over all {h.V} columns")
    ref_all = ohead.logits(h, x_all)
    ph = PackedHead.from_arrays(h)
    for M in Ms:
        say(f"sweep128k M={M}, all columns")
        lg = ph.logits(torch_x(x_all[:M]))
        torch.cuda.synchronize()
        err = assert_logits_close(lg.cpu().numpy(), ref_all[:M], what=f"sweep128k M={M}")
        say(f"  max rel err {err:.2e}")
    ph.close()


QWEN_PROBE_COLS = (0, 1, 7, 8, 31, 32, 127, 128, 255, 256, 2047, 2048, 4064, 4095)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("scales", ["f16", "u8"])
def test_identity_probe_gemv_one_token_qwen_bit_exact(scales):
    """M = 1 calls through the decode GEMV (the one-token kernel the headline
    decode step runs) with a one-hot token at sampled columns: every logit of
    the Qwen-shaped head (no low-rank parts) is exactly s_res * c."""
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode", rc=0, rr=0, scales=scales)
    ph = PackedHead.from_arrays(h)
    ph.force_path("gemv")
    rng = np.random.default_rng(12)
    cols = np.unique(np.concatenate([QWEN_PROBE_COLS, rng.integers(0, h.d, 10)]))
    x = np.zeros((cols.size, h.d), dtype=np.uint16)
    x[np.arange(cols.size), cols] = 0x3F80
    say(f"identity probe qwen ({scales} scales), GEMV at M=1: {cols.size} columns")
    ref = ohead.logits(h, x)
    for j in range(cols.size):
        lg = ph.logits(torch_x(x[j:j + 1]))
        torch.cuda.synchronize()
        lg = lg.cpu().numpy()[0].astype(np.float64)
        bad = np.nonzero(lg != ref[j])[0]
        assert bad.size == 0, (f"column {cols[j]}: {bad.size} logits differ, first row "
                               f"{bad[0]}: gpu {lg[bad[0]]!r} oracle {ref[j, bad[0]]!r}")
    ph.close()


def _residual_rounding_bound(h, x_bits, lam=8.0):
    """Per-logit bound on the fp32 rounding error of the residual stream at
    one token, under the probabilistic rounding model (each rounding an
    independent error of at most u = 2^-24 relative to the rounded value;
    Higham and Mary, SIAM J. Sci. Comput. 41(5), 2019): |error| <= lam * u *
    sqrt(sum_k B_k^2) over bounds B_k of every rounded intermediate.  Taken
    per 32-code chunk: the chunk bias -136 * sum x and the 16 two-product
    dot steps (66 roundings of values at most 279 * sum_chunk |x|); per group
    the chunk and group partials and their scaled value (5 roundings of at
    most s * sum_group |c x|); the sum over groups (d/g roundings of at most
    sum_j s_j sum_group |c x|); |c| <= 8 throughout.  x_bits: one token."""
    u = 2.0 ** -24
    ax = np.abs(layout.bf16_to_f64(x_bits))
    chunk_x = ax.reshape(-1, 32).sum(axis=1)                  # [d/32]
    cx = 8.0 * ax.reshape(-1, h.g).sum(axis=1)                # |c| <= 8: [d/g]
    s = ohead.residual_scales(h, 0, h.V)                      # [V, d/g]
    inner = 66.0 * ((s * 279.0) ** 2 * (chunk_x.reshape(-1, h.g // 32) ** 2).sum(axis=1)).sum(axis=1)
    grp = 5.0 * ((s * cx) ** 2).sum(axis=1)
    total = (s * cx).sum(axis=1)
    return lam * u * np.sqrt(inner + grp + (h.d // h.g) * total ** 2)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("scales", ["f16", "u8"])
def test_residual_only_qwen_one_token_tight_bound(scales):
    from paper_2608_02703_amd import PackedHead
    h = make_head("qwen_decode", rc=0, rr=0, scales=scales)
    ph = PackedHead.from_arrays(h)
    say(f"residual-only qwen ({scales} scales), M=1 random x, rounding bound")
    xs = make_x("qwen_decode", 2)
    refs = ohead.logits(h, xs)
    for j in range(2):
        x = xs[j:j + 1]
        ref = refs[j]
        lg = ph.logits(torch_x(x))
        torch.cuda.synchronize()
        lg = lg.cpu().numpy()[0].astype(np.float64)
        bound = _residual_rounding_bound(h, x[0])
        ratio = np.abs(lg - ref) / bound
        worst = int(np.argmax(ratio))
        say(f"  token {j}: max |d| {np.abs(lg - ref).max():.2e}, max |d|/bound "
            f"{ratio.max():.3f}, median bound {np.median(bound):.2e}, "
            f"residual logit std {ref.std():.3f}")
        assert ratio.max() <= 1.0, (f"row {worst}: gpu {lg[worst]!r} oracle {ref[worst]!r} "
                                    f"bound {bound[worst]:.3e}")
        # the bound is far inside the 2e-3 (1 + |l|) logit tolerance
        assert np.median(bound / (2e-3 * (1 + np.abs(ref)))) < 0.1
    ph.close()
