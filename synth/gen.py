"""Seeded generators for packed heads, hidden states and targets.

Every stream is drawn from ``default_rng(SeedSequence([2608, 2703, cfg_id,
stream_id, draw]))`` so a buffer never depends on the order in which others
were drawn.  Values follow the synthetic recipe of the five head shapes used
throughout the tests and the benchmark:

* residual codes: the packed INT4 bytes themselves, uniform over 0..255, so
  every stored nibble is uniform over 0..15 and every signed code (nibble - 8)
  uniform over [-8, 7], whatever nibble order a reader uses;
* residual group scales: |N(0, 0.02)| rounded once to fp16;
* factor codes: integers uniform in [-127, 127] (int8);
* factor scales: |N(0, 0.01)| rounded once to fp16;
* hidden states: x = (z * sqrt(lambda)) Q^T with z ~ N(0, 1), lambda_i
  proportional to i^-alpha normalised to sum 1, Q a Haar-random orthogonal
  basis (QR of a Gaussian matrix with the sign fix); for the Gemma-shaped head
  four seeded channels are then multiplied by 20; finally one round-to-nearest
  -even step to bf16 (the bits are returned as uint16);
* targets: uniform over [0, V), or Zipf(s) over ranks 1..V (finite support,
  inverse CDF) mapped to ids through a seeded permutation.
"""
from __future__ import annotations

import dataclasses
import functools
from typing import Optional

import numpy as np

# name -> shape and distribution parameters of the five workloads
CONFIGS = {
    "tiny": dict(cfg_id=1, V=8192, d=512, g=64, rc=64, rr=32, Ms=(1, 8),
                 alpha=1.5, outliers=0, targets="uniform"),
    "qwen_decode": dict(cfg_id=2, V=151936, d=4096, g=128, rc=64, rr=32,
                        Ms=(1, 4, 16), alpha=1.5, outliers=0, targets="uniform"),
    # the prefill workload evaluates the same packed head as the decode one
    "qwen_prefill": dict(cfg_id=3, head_cfg_id=2, V=151936, d=4096, g=128, rc=64, rr=32,
                         Ms=(4096,), alpha=1.5, outliers=0, targets="zipf",
                         zipf_s=1.1),
    "gemma": dict(cfg_id=4, V=262144, d=2560, g=128, rc=64, rr=32,
                  Ms=(1, 8, 64), alpha=2.0, outliers=4, targets="uniform"),
    "sweep128k": dict(cfg_id=5, V=128256, d=8192, g=128, rc=128, rr=64,
                      Ms=(1, 2, 4, 8, 16, 32, 64, 128, 256, 512), alpha=1.5,
                      outliers=0, targets="uniform"),
}

_STREAMS = {name: i for i, name in enumerate([
    "basis", "x", "res_codes", "res_scales", "core_u", "core_u_scale",
    "core_v", "core_v_scale", "corr_a", "corr_a_scale", "corr_b",
    "corr_b_scale", "targets", "outlier_idx", "zipf_perm", "spare"])}

RES_SCALE_SIGMA = 0.02
FACTOR_SCALE_SIGMA = 0.01
OUTLIER_FACTOR = 20.0


def _rng(cfg_id: int, stream: str, draw: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([2608, 2703, int(cfg_id), _STREAMS[stream],
                                 int(draw)])
    return np.random.default_rng(ss)


def f64_to_bf16_bits(a) -> np.ndarray:
    """Round float64 values to bf16 (8 significant bits, ties to even) once,
    returning the 16-bit patterns as uint16.  Inputs must lie in the normal
    bf16 range (or be zero); the generators never leave it."""
    a = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(a)                      # a = m * 2**e, 0.5 <= |m| < 1
    r = np.ldexp(np.round(np.ldexp(m, 8)), e - 8)
    bits = r.astype(np.float32).view(np.uint32) >> np.uint32(16)
    return bits.astype(np.uint16)


@dataclasses.dataclass
class HeadArrays:
    """Host copies of every buffer of a packed head (row-major numpy arrays).

    res_codes    uint8   [V, d/2]      INT4 code bytes (nibble order: see
                                       the layout notes in include/archead.h)
    res_scales   float16 [V, d/g]
    core_u       int8    [V, rc]       core_u_scale float16 [V]
                 (or uint32 [V, ceil(rc/6)]: 5-bit codes, six per word)
    core_v       int8    [rc, d]       core_v_scale float16 [rc, d/gV]
    corr_a       int8    [V, rr]       corr_a_scale float16 [V]
    corr_b       int8    [rr, d]       corr_b_scale float16 [rr, d/gB]
    """
    V: int
    d: int
    g: int
    rc: int
    rr: int
    gV: int
    gB: int
    res_codes: np.ndarray
    res_scales: np.ndarray
    core_u: np.ndarray
    core_u_scale: np.ndarray
    core_v: np.ndarray
    core_v_scale: np.ndarray
    corr_a: np.ndarray
    corr_a_scale: np.ndarray
    corr_b: np.ndarray
    corr_b_scale: np.ndarray
    res_row_scales: Optional[np.ndarray] = None   # fp16 [V] with uint8 res_scales

    BUFFERS = ("res_codes", "res_scales", "core_u", "core_u_scale", "core_v",
               "core_v_scale", "corr_a", "corr_a_scale", "corr_b",
               "corr_b_scale")


def _cfg(cfg) -> dict:
    if isinstance(cfg, str):
        return dict(CONFIGS[cfg])
    return dict(cfg)


def _fp16_abs_normal(rng, sigma, shape) -> np.ndarray:
    return np.abs(rng.normal(0.0, sigma, size=shape)).astype(np.float16)


def _int8_uniform(rng, shape) -> np.ndarray:
    return rng.integers(-127, 128, size=shape, dtype=np.int16).astype(np.int8)


def make_head(cfg="tiny", draw: int = 0, **over) -> HeadArrays:
    """Draw a packed head.  ``over`` may replace V, d, g, rc, rr, gV, gB (for
    ragged and degenerate shapes); gV/gB default to d (one scale per row).
    ``scales="u8"`` stores the residual group scales as 8-bit codes with an
    fp16 scale per row (the same draws rounded to rs * q, rs = max / 255).
    ``core_u="i5"`` draws 5-bit core-left codes uniform in [-15, 15] and
    stores them six per 32-bit word (uint32 [V, ceil(rc/6)]: field k of a
    row at bits 5 (k % 6) of word k // 6, two's complement, unused bits
    zero)."""
    c = _cfg(cfg)
    scales = over.pop("scales", "f16")
    core_u_fmt = over.pop("core_u", "i8")
    unknown = set(over) - {"V", "d", "g", "rc", "rr", "gV", "gB", "cfg_id"}
    if unknown:
        raise TypeError(f"unknown head overrides {sorted(unknown)}")
    c.update(over)
    if "cfg_id" in over:
        c.pop("head_cfg_id", None)
    V, d, g, rc, rr = c["V"], c["d"], c["g"], c["rc"], c["rr"]
    gV = c.get("gV", d)
    gB = c.get("gB", d)
    cid = c.get("head_cfg_id", c["cfg_id"])
    assert d % 2 == 0 and d % g == 0 and d % gV == 0 and d % gB == 0
    r = functools.partial(_rng, cid, draw=draw)
    res_codes = r("res_codes").integers(0, 256, size=(V, d // 2), dtype=np.uint8)
    res_scales = _fp16_abs_normal(r("res_scales"), RES_SCALE_SIGMA, (V, d // g))
    if core_u_fmt == "i5":
        f = r("core_u").integers(-15, 16, size=(V, rc)).astype(np.int64) & 31
        w = np.zeros((V, (rc + 5) // 6), dtype=np.int64)
        for k in range(rc):
            w[:, k // 6] |= f[:, k] << (5 * (k % 6))
        core_u = w.astype(np.uint32)
    elif core_u_fmt == "i8":
        core_u = _int8_uniform(r("core_u"), (V, rc))
    else:
        raise ValueError(f"core_u must be 'i8' or 'i5', not {core_u_fmt!r}")
    core_u_scale = _fp16_abs_normal(r("core_u_scale"), FACTOR_SCALE_SIGMA, (V,))
    core_v = _int8_uniform(r("core_v"), (rc, d))
    core_v_scale = _fp16_abs_normal(r("core_v_scale"), FACTOR_SCALE_SIGMA,
                                    (rc, d // gV))
    corr_a = _int8_uniform(r("corr_a"), (V, rr))
    corr_a_scale = _fp16_abs_normal(r("corr_a_scale"), FACTOR_SCALE_SIGMA, (V,))
    corr_b = _int8_uniform(r("corr_b"), (rr, d))
    corr_b_scale = _fp16_abs_normal(r("corr_b_scale"), FACTOR_SCALE_SIGMA,
                                    (rr, d // gB))
    res_row_scales = None
    if scales == "u8":
        top = res_scales.astype(np.float64).max(axis=1)
        res_row_scales = (top / 255.0).astype(np.float16)
        rs = res_row_scales.astype(np.float64)
        rs_safe = np.where(rs > 0, rs, 1.0)
        q = np.rint(res_scales.astype(np.float64) / rs_safe[:, None])
        res_scales = np.clip(q, 0, 255).astype(np.uint8)
    elif scales != "f16":
        raise ValueError(f"scales must be 'f16' or 'u8', not {scales!r}")
    return HeadArrays(V, d, g, rc, rr, gV, gB, res_codes, res_scales, core_u,
                      core_u_scale, core_v, core_v_scale, corr_a, corr_a_scale,
                      corr_b, corr_b_scale, res_row_scales)


@functools.lru_cache(maxsize=2)
def _haar_basis(d: int, cfg_id: int) -> np.ndarray:
    rng = _rng(cfg_id, "basis")
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    q *= np.sign(np.diag(r))[None, :]
    return q


def spectrum(d: int, alpha: float) -> np.ndarray:
    lam = np.arange(1, d + 1, dtype=np.float64) ** (-float(alpha))
    return lam / lam.sum()


def make_x(cfg="tiny", M: int = 1, draw: int = 0, d: Optional[int] = None,
           basis: str = "haar") -> np.ndarray:
    """bf16 hidden states [M, d] as uint16 bit patterns.

    ``basis="haar"`` uses the seeded Haar basis (the workload recipe);
    ``basis="identity"`` skips the rotation (cheap, for shapes where only the
    value distribution matters, e.g. ragged-shape tests)."""
    c = _cfg(cfg)
    d = c["d"] if d is None else d
    cid = c["cfg_id"]
    lam = spectrum(d, c["alpha"])
    z = _rng(cid, "x", draw).standard_normal((M, d)) * np.sqrt(lam)[None, :]
    if basis == "haar":
        x = z @ _haar_basis(d, cid).T
    elif basis == "identity":
        x = z[:, _rng(cid, "spare", draw).permutation(d)]
    else:
        raise ValueError(basis)
    if c.get("outliers", 0):
        idx = _rng(cid, "outlier_idx").choice(d, size=c["outliers"],
                                              replace=False)
        x[:, idx] *= OUTLIER_FACTOR
    return f64_to_bf16_bits(x)


def make_targets(cfg="tiny", M: int = 1, draw: int = 0,
                 V: Optional[int] = None) -> np.ndarray:
    """int32 target ids [M]."""
    c = _cfg(cfg)
    V = c["V"] if V is None else V
    cid = c["cfg_id"]
    rng = _rng(cid, "targets", draw)
    if c.get("targets", "uniform") == "uniform":
        return rng.integers(0, V, size=M).astype(np.int32)
    s = float(c.get("zipf_s", 1.1))
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    rank = np.searchsorted(cdf, rng.random(M), side="right")
    rank = np.minimum(rank, V - 1)
    perm = _rng(cid, "zipf_perm").permutation(V)
    return perm[rank].astype(np.int32)


def make_workload(cfg="tiny", M: Optional[int] = None, draw: int = 0):
    c = _cfg(cfg)
    M = c["Ms"][-1] if M is None else M
    return make_head(c, draw=draw), make_x(c, M, draw=draw), \
        make_targets(c, M, draw=draw)
