"""Offline construction of a packed ARCHead head (oracle side, small shapes).

Follows the paper's construction (Section 3.1 for the metric, Section 3.2 for
the core and correction, Algorithm 2 "Expanded packed-head construction" for
the order of steps), with an exact SVD where the paper uses a randomized one:

  C_lambda = H^T H / N + lambda * cbar * I,  cbar = mean diagonal of H^T H / N
  C_lambda = Q Lambda Q^T                    (symmetric eigendecomposition)
  T_p = Q Lambda^p Q^T,  T_p^-1 = Q Lambda^-p Q^T
  W_d = Q5(A_c) Q8(B_c) + Q_SC4(W - A_c B_c)   (QuantizeCore)
  E = W - W_d                                  (realized core error)
  E T_p ~ U_r Sigma_r V_r^T                    (rank-r_r truncated SVD)
  A_w = U_r Sigma_r,  B_w = V_r^T T_p^-1
  A_w row-wise INT8, B_w group-wise INT8       (QuantizeINT8)

Readings where the paper leaves details open:
  * damping uses lambda * cbar * I (the appendix form) rather than lambda * I;
  * the rank-r_c core split is A_c = U Sigma, B_c = V^T of W's truncated SVD,
    mirroring how the paper splits the correction;
  * every quantizer is symmetric round-to-nearest with scale = absmax / qmax
    (qmax = 2^(b-1) - 1: 7 for SC4, 15 for 5-bit, 127 for INT8), the scale
    rounded to fp16 first and the codes computed against the rounded scale;
    an all-zero group gets scale 0 and codes 0;
  * the SC4 residual is quantized against the unquantized core A_c B_c, and
    E is measured against the dequantized core, as the paper states both.
"""
from __future__ import annotations

import types

import numpy as np

from .layout import fp16_to_f64, pack_int4


def damped_covariance(H: np.ndarray, lam: float) -> np.ndarray:
    """C_lambda = H^T H / N + lambda * cbar * I."""
    H = np.asarray(H, dtype=np.float64)
    C = H.T @ H / H.shape[0]
    cbar = float(np.mean(np.diag(C)))
    return C + lam * cbar * np.eye(C.shape[0])


def metric_transform(C_lam: np.ndarray, p: float):
    """(T_p, T_p^-1) from the eigendecomposition of the damped covariance."""
    evals, Q = np.linalg.eigh(C_lam)
    if evals.min() <= 0:
        raise ValueError("damped covariance is not positive definite")
    T = (Q * evals ** p) @ Q.T
    Tinv = (Q * evals ** (-p)) @ Q.T
    return T, Tinv


def fit_correction(E: np.ndarray, T: np.ndarray, Tinv: np.ndarray, r: int):
    """A_w = U_r Sigma_r, B_w = V_r^T T_p^-1 from the SVD of E T_p."""
    U, S, Vt = np.linalg.svd(np.asarray(E, dtype=np.float64) @ T,
                             full_matrices=False)
    return U[:, :r] * S[:r], Vt[:r] @ Tinv


def quantize_symmetric(X: np.ndarray, bits: int, group: int):
    """Round-to-nearest symmetric quantization along the last axis in groups
    of ``group``.  Returns (codes int8 [..., n], scales fp16 [..., n/group])."""
    X = np.asarray(X, dtype=np.float64)
    qmax = 2 ** (bits - 1) - 1
    rows, n = X.shape
    Xg = X.reshape(rows, n // group, group)
    scale = (np.abs(Xg).max(axis=2) / qmax).astype(np.float16)
    s64 = fp16_to_f64(scale)
    safe = np.where(s64 > 0, s64, 1.0)
    codes = np.clip(np.rint(Xg / safe[:, :, None]), -qmax, qmax)
    codes = np.where(s64[:, :, None] > 0, codes, 0).astype(np.int8)
    return codes.reshape(rows, n), scale


def dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    rows, n = codes.shape
    s = fp16_to_f64(scales).reshape(rows, -1)
    return codes.astype(np.float64) * np.repeat(s, n // s.shape[1], axis=1)


def quantize_core(W: np.ndarray, rc: int, g: int):
    """QuantizeCore: 5-bit A_c (per row), INT8 B_c (per row), SC4 residual."""
    W = np.asarray(W, dtype=np.float64)
    V, d = W.shape
    out = {}
    if rc:
        U, S, Vt = np.linalg.svd(W, full_matrices=False)
        Ac, Bc = U[:, :rc] * S[:rc], Vt[:rc]
        out["core_u"], out["core_u_scale"] = quantize_symmetric(Ac, 5, rc)
        out["core_v"], out["core_v_scale"] = quantize_symmetric(Bc, 8, d)
        core_q = dequantize(out["core_u"], out["core_u_scale"]) @ \
            dequantize(out["core_v"], out["core_v_scale"])
        R = W - Ac @ Bc
        out["A_c"], out["B_c"] = Ac, Bc          # the unquantized core factors
    else:
        core_q = np.zeros_like(W)
        R = W
    res_codes, res_scales = quantize_symmetric(R, 4, g)
    out["res_int4"], out["res_scales"] = res_codes, res_scales
    W_d = core_q + dequantize(res_codes, res_scales)
    return W_d, out


def build_head(W: np.ndarray, H: np.ndarray, rc: int, rr: int, g: int,
               p: float, lam: float, gB: int = None):
    """Run the construction and return (head, info).

    ``head`` carries the attributes the oracle and the packed library read
    (V, d, g, rc, rr, gV, gB and the ten buffers); ``info`` holds the
    intermediate matrices (T_p, T_p^-1, W_d, E, unquantized A_w and B_w)."""
    W = np.asarray(W, dtype=np.float64)
    V, d = W.shape
    gB = d if gB is None else gB
    C_lam = damped_covariance(H, lam)
    T, Tinv = metric_transform(C_lam, p)
    W_d, core = quantize_core(W, rc, g)
    E = W - W_d
    h = types.SimpleNamespace(V=V, d=d, g=g, rc=rc, rr=rr, gV=d, gB=gB)
    h.res_codes = pack_int4(core["res_int4"])
    h.res_scales = core["res_scales"]
    h.core_u = core.get("core_u", np.zeros((V, 0), np.int8))
    h.core_u_scale = core.get("core_u_scale", np.zeros((V, 1), np.float16))[:, 0]
    h.core_v = core.get("core_v", np.zeros((0, d), np.int8))
    h.core_v_scale = core.get("core_v_scale", np.zeros((0, 1), np.float16))
    info = dict(T=T, Tinv=Tinv, W_d=W_d, E=E, C_lam=C_lam, A_c=core.get("A_c"),
                B_c=core.get("B_c"))
    if rr:
        A_w, B_w = fit_correction(E, T, Tinv, rr)
        h.corr_a, sa = quantize_symmetric(A_w, 8, rr)
        h.corr_a_scale = sa[:, 0]
        h.corr_b, h.corr_b_scale = quantize_symmetric(B_w, 8, gB)
        info.update(A_w=A_w, B_w=B_w)
    else:
        h.corr_a = np.zeros((V, 0), np.int8)
        h.corr_a_scale = np.zeros((V,), np.float16)
        h.corr_b = np.zeros((0, d), np.int8)
        h.corr_b_scale = np.zeros((0, 1), np.float16)
    return h, info
