"""Helpers for the GPU parity tests: upload, tolerance checks, oracle caches."""
from __future__ import annotations

import functools
import sys

import numpy as np

from oracle import head as ohead
from oracle import layout
from synth import make_head, make_targets, make_x, f64_to_bf16_bits

LOGIT_TOL = 2e-3      # max |d logit| <= 2e-3 * (1 + |logit|) for fp32 logits
CE_TOL = 1e-4         # max |d CE| in nats per token


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_x(bits: np.ndarray, device="cuda", ld=None):
    """uint16 bf16 bit patterns [M, d] -> torch.bfloat16 on the device,
    optionally inside a wider buffer of row stride ``ld``."""
    import torch
    M, d = bits.shape
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    if ld is None or ld == d:
        return t.to(device)
    buf = torch.zeros((M, ld), dtype=torch.bfloat16, device=device)
    buf[:, :d] = t.to(device)
    return buf[:, :d]


def assert_logits_close(gpu: np.ndarray, ref: np.ndarray, tol=LOGIT_TOL, what=""):
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - ref) / (1.0 + np.abs(ref))
    worst = np.unravel_index(np.argmax(err), err.shape)
    assert np.isfinite(gpu).all(), f"{what}: non-finite GPU logits"
    assert err.max() <= tol, (f"{what}: max rel err {err.max():.3e} at {worst}: "
                              f"gpu {gpu[worst]!r} oracle {ref[worst]!r}")
    return float(err.max())


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return layout.bf16_to_f64(np.asarray(bits).view(np.uint16))


BF16_CHECK_MIN_ABS = 1.0 / 16


def _ordered(b):  # bf16 bit patterns -> a monotone integer line
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def assert_bf16_output(gpu_bits: np.ndarray, gpu_f32: np.ndarray, ref: np.ndarray,
                       what=""):
    """bf16 logits: (1) bit-exactly the round-to-nearest-even of the kernel's
    own fp32 result (itself checked against the oracle), and (2) equal to
    RNE(oracle) or one of its two bf16 neighbours wherever |logit| >= 1/16.
    Below that a bf16 step (< 2^-11) approaches the fp32 accumulation error,
    so only (1) and the fp32 tolerance apply."""
    g = np.asarray(gpu_bits).view(np.uint16).astype(np.int64)
    own = f64_to_bf16_bits(np.asarray(gpu_f32, dtype=np.float64)).astype(np.int64)
    mism = np.argwhere(g != own)
    assert mism.size == 0, f"{what}: bf16 != RNE(fp32) at {mism[:5].tolist()}"
    rne = f64_to_bf16_bits(ref).astype(np.int64)
    big = np.abs(ref) >= BF16_CHECK_MIN_ABS
    diff = np.abs(_ordered(g) - _ordered(rne))[big]
    assert diff.max(initial=0) <= 1, \
        f"{what}: bf16 output {diff.max()} steps from RNE(oracle)"


def assert_ce_close(gpu, ref, tol=CE_TOL, what=""):
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - ref)
    assert np.isfinite(gpu).all(), f"{what}: non-finite CE"
    assert err.max() <= tol, f"{what}: max |dCE| {err.max():.3e} (gpu {gpu[err.argmax()]}, oracle {ref[err.argmax()]})"
    return float(err.max())


def argmax_agreement(gpu_logits: np.ndarray, ref: np.ndarray, tol=LOGIT_TOL):
    """(n_checked, n_excluded): the argmax must agree on every token whose
    oracle top-2 gap exceeds twice the logit tolerance."""
    gap = ohead.top2_gap(ref)
    top = ref.max(axis=1)
    keep = gap > 2 * tol * (1 + np.abs(top))
    g = np.asarray(gpu_logits).argmax(axis=1)
    o = ohead.argmax(ref)
    bad = np.nonzero(keep & (g != o))[0]
    assert bad.size == 0, f"argmax differs on tokens {bad[:10]}"
    return int(keep.sum()), int((~keep).sum())


@functools.lru_cache(maxsize=3)
def cached_head(cfg: str, **over):
    return make_head(cfg, **over)


@functools.lru_cache(maxsize=4)
def cached_oracle_logits(cfg: str, M: int, draw: int = 0):
    """Oracle logits [M, V] of the config's head on its first M tokens."""
    h = cached_head(cfg)
    x = make_x(cfg, M, draw=draw)
    return ohead.logits(h, x)
