"""Dense fp64 evaluation of the packed ARCHead head (oracle side).

What the packed head represents (ARCHead, Section 3.2, equations for W_d,
W_hat and Y_hat; Appendix table "Logical contents of the packed ARCHead state
dictionary"):

  W_d    = Q5(A_c) Q8(B_c) + Q_SC4(W - A_c B_c)     quantized core
  W_hat  = W_d + A_w B_w                            core plus correction
  Y_hat  = H W_hat^T = H W_d^T + (H B_w^T) A_w^T    logits

In buffer terms (names of the packed buffers, shapes as in the layout notes):

  W_res [v, i] = s_res[v, i // g] * c[v, i]                    (residual)
  W_core[v, i] = sum_k (s_U[v] cU[v, k]) (s_V[k, i // gV] cV[k, i])
  W_corr[v, i] = sum_k (s_A[v] cA[v, k]) (s_B[k, i // gB] cB[k, i])
  W_hat = W_res + W_core + W_corr,    logits[m, v] = sum_i x[m, i] W_hat[v, i]

The residual group scales s_res are stored either as fp16 or, the paper's
"quantized group scales" (packed-buffer table), as 8-bit codes q with one
fp16 scale rs per vocabulary row: s_res[v, j] = rs[v] * q[v, j] (a uint8
res_scales array plus res_row_scales [V]; the format is this library's
reading, the paper leaves it open).

The core left factor's codes are int8, or 5-bit codes bit-packed six per
32-bit word (uint32 [V, ceil(r_c/6)], the paper's "packed 5-bit" Q5(A_c);
layout in oracle.layout.unpack_int5).

A rank of zero means the component is absent (the paper's "core only" and
"Group INT4" ablations).  The head object is any object with the attributes
V, d, g, rc, rr, gV, gB and the ten buffers (res_codes, res_scales, core_u,
core_u_scale, core_v, core_v_scale, corr_a, corr_a_scale, corr_b,
corr_b_scale) as numpy arrays.

Every value is converted to float64 exactly (integer codes, fp16 scales, bf16
activations), so the only rounding is fp64 accumulation.
"""
from __future__ import annotations

import numpy as np

from .layout import bf16_to_f64, fp16_to_f64, unpack_int4, unpack_int5

ROW_CHUNK = 4096


def residual_rows(h, v0: int, v1: int) -> np.ndarray:
    """W_res for vocabulary rows [v0, v1): s_res[v, i // g] * c[v, i]."""
    c = unpack_int4(h.res_codes[v0:v1], h.d).astype(np.float64)
    return c * np.repeat(residual_scales(h, v0, v1), h.g, axis=1)


def residual_scales(h, v0: int, v1: int) -> np.ndarray:
    """s_res for rows [v0, v1) as float64 [n, d/g]: the fp16 values, or
    rs[v] * q[v, j] for 8-bit codes."""
    sc = np.asarray(h.res_scales[v0:v1])
    if sc.dtype == np.uint8:
        rs = fp16_to_f64(np.asarray(h.res_row_scales)[v0:v1])
        return rs[:, None] * sc.astype(np.float64)
    return fp16_to_f64(sc)


def left_factor(codes, scales, rank: int = None) -> np.ndarray:
    """Row-scaled left factor: s[v] * codes[v, k] (U_c or A_w).  codes are
    int8 [n, rank], or uint32 ARCHEAD_I5 words [n, ceil(rank/6)] of 5-bit
    codes (then rank is required)."""
    codes = np.asarray(codes)
    if codes.dtype == np.uint32:
        codes = unpack_int5(codes, rank)
    return fp16_to_f64(scales)[:, None] * codes.astype(np.float64)


def right_factor(codes, scales, group: int) -> np.ndarray:
    """Group-scaled right factor: s[k, i // group] * codes[k, i] (V_c or B_w)."""
    s = fp16_to_f64(scales)
    s = s.reshape(s.shape[0], -1)
    return np.repeat(s, group, axis=1) * np.asarray(codes).astype(np.float64)


def core_rows(h, v0: int, v1: int) -> np.ndarray:
    if h.rc == 0:
        return np.zeros((v1 - v0, h.d))
    return left_factor(h.core_u[v0:v1], h.core_u_scale[v0:v1], h.rc) @ \
        right_factor(h.core_v, h.core_v_scale, h.gV)


def correction_rows(h, v0: int, v1: int) -> np.ndarray:
    if h.rr == 0:
        return np.zeros((v1 - v0, h.d))
    return left_factor(h.corr_a[v0:v1], h.corr_a_scale[v0:v1]) @ \
        right_factor(h.corr_b, h.corr_b_scale, h.gB)


def dense_rows(h, v0: int, v1: int) -> np.ndarray:
    """Rows [v0, v1) of W_hat = W_res + W_core + W_corr, in float64."""
    return residual_rows(h, v0, v1) + core_rows(h, v0, v1) + \
        correction_rows(h, v0, v1)


def _as_f64_x(x) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_to_f64(x)
    return x.astype(np.float64)


def logits(h, x, vocab=None, chunk: int = ROW_CHUNK) -> np.ndarray:
    """logits [M, n] = x W_hat^T in float64.

    x: bf16 bit patterns (uint16) [M, d] or real values.  vocab: optional
    array of vocabulary ids (then only those columns are returned, in that
    order).  Rows of W_hat are formed ``chunk`` at a time to bound memory;
    each logit is still exactly sum_i x[m, i] W_hat[v, i]."""
    X = _as_f64_x(x)
    if vocab is None:
        out = np.empty((X.shape[0], h.V))
        for v0 in range(0, h.V, chunk):
            v1 = min(h.V, v0 + chunk)
            out[:, v0:v1] = X @ dense_rows(h, v0, v1).T
        return out
    vocab = np.asarray(vocab, dtype=np.int64)
    out = np.empty((X.shape[0], vocab.size))
    for j in range(0, vocab.size, chunk):
        ids = vocab[j:j + chunk]
        out[:, j:j + ids.size] = X @ _gather_rows(h, ids).T
    return out


def _gather_rows(h, ids) -> np.ndarray:
    class _Sub:  # the selected rows viewed as a smaller head
        pass
    s = _Sub()
    for k in ("d", "g", "rc", "rr", "gV", "gB", "core_v", "core_v_scale",
              "corr_b", "corr_b_scale"):
        setattr(s, k, getattr(h, k))
    s.V = ids.size
    for k in ("res_codes", "res_scales", "core_u", "core_u_scale", "corr_a",
              "corr_a_scale"):
        setattr(s, k, np.asarray(getattr(h, k))[ids])
    if getattr(h, "res_row_scales", None) is not None:
        s.res_row_scales = np.asarray(h.res_row_scales)[ids]
    return dense_rows(s, 0, ids.size)


def logits_factorized(h, x) -> np.ndarray:
    """Y_hat = x W_res^T + (x V_c^T) U_c^T + (x B_w^T) A_w^T, the bracketing
    of the paper's inference equation, in float64 (used to check linearity
    against the dense path)."""
    X = _as_f64_x(x)
    out = np.empty((X.shape[0], h.V))
    for v0 in range(0, h.V, ROW_CHUNK):
        v1 = min(h.V, v0 + ROW_CHUNK)
        out[:, v0:v1] = X @ residual_rows(h, v0, v1).T
    if h.rc:
        t_c = X @ right_factor(h.core_v, h.core_v_scale, h.gV).T
        out += t_c @ left_factor(h.core_u, h.core_u_scale, h.rc).T
    if h.rr:
        t_w = X @ right_factor(h.corr_b, h.corr_b_scale, h.gB).T
        out += t_w @ left_factor(h.corr_a, h.corr_a_scale).T
    return out


def dense_bf16_logits(w_bits: np.ndarray, x) -> np.ndarray:
    """Logits of a dense bf16 head (the reference the paper's fidelity
    metrics compare a compressed head against, Section 4 "Logit Fidelity"):
    x [M, d] times W^T, W the bf16 bit patterns [V, d], every value converted
    to fp64 exactly, one fp64 matrix product."""
    w = bf16_to_f64(np.asarray(w_bits).view(np.uint16))
    return _as_f64_x(x) @ w.T


def cross_entropy(lg: np.ndarray, targets) -> np.ndarray:
    """Per-token CE [M] = logsumexp_v(lg[m, :]) - lg[m, y_m], natural log.

    The log-sum-exp is taken with the row maximum factored out, which is the
    same quantity.  A target outside [0, V) gives NaN for that token."""
    lg = np.asarray(lg, dtype=np.float64)
    y = np.asarray(targets, dtype=np.int64)
    mx = lg.max(axis=1)
    lse = mx + np.log(np.exp(lg - mx[:, None]).sum(axis=1))
    ok = (y >= 0) & (y < lg.shape[1])
    tgt = np.where(ok, lg[np.arange(lg.shape[0]), np.clip(y, 0, lg.shape[1] - 1)],
                   np.nan)
    return lse - tgt


def argmax(lg: np.ndarray) -> np.ndarray:
    """Smallest index attaining the row maximum."""
    return np.asarray(lg).argmax(axis=1)


def top2_gap(lg: np.ndarray) -> np.ndarray:
    """Difference between the largest and second-largest logit of each row."""
    part = np.partition(np.asarray(lg), -2, axis=1)
    return part[:, -1] - part[:, -2]
