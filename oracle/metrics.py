"""Evaluation metrics used by the paper (Section 4, "Data and metrics").

Perplexity is exp of the mean token cross-entropy (natural log); relative
perplexity is the compressed PPL divided by the dense PPL, i.e. exp of the
cross-entropy difference.
"""
from __future__ import annotations

import numpy as np


def ppl(mean_ce: float) -> float:
    return float(np.exp(mean_ce))


def rel_ppl(mean_ce: float, mean_ce_ref: float) -> float:
    return float(np.exp(mean_ce) / np.exp(mean_ce_ref))


def delta_ce(mean_ce: float, mean_ce_ref: float) -> float:
    return float(mean_ce - mean_ce_ref)


# ------------------------------------------------------------ logit fidelity
# Section 4, "Logit Fidelity" (Table 8): how closely the packed head's logits
# follow the dense head's on the same positions.  Readings taken here (the
# text names the metrics without formulas):
#   * KL is KL(p_dense || p_packed), p = softmax of one position's logits;
#   * top-k agreement at a position: the dense head's top-1 token lies in the
#     packed head's top k (k = 1 is the printed top-1 agreement); ranks
#     follow a stable descending order, so among equal logits the smaller
#     vocabulary index ranks first, as for the first-index argmax;
#   * MSE is the squared logit error summed over the vocabulary and averaged
#     over positions, i.e. (1/N) ||H W^T - H What^T||_F^2, the activation
#     objective of Eq. (1) evaluated on the positions measured.

def logit_fidelity(ref: np.ndarray, test: np.ndarray):
    """Per-position fidelity of `test` logits to `ref` logits, both [M, V].

    Returns (kl, sq, ref_idx, rank), each of length M, in fp64 / int64:
      kl[m]      = sum_v p[v] (log p[v] - log q[v]), p = softmax(ref[m]),
                   q = softmax(test[m]);
      sq[m]      = sum_v (ref[m, v] - test[m, v])^2;
      ref_idx[m] = the first v attaining max ref[m];
      rank[m]    = the position of ref_idx[m] when test[m] is sorted in
                   decreasing order, equal values by increasing v (0 = the
                   packed head's first argmax).
    Plain per-row definitions; only the log-sum-exp is shifted by the row
    maximum so that exp does not overflow.
    """
    a = np.asarray(ref, dtype=np.float64)
    b = np.asarray(test, dtype=np.float64)
    assert a.shape == b.shape and a.ndim == 2
    M, V = a.shape
    kl = np.zeros(M)
    sq = np.zeros(M)
    ref_idx = np.zeros(M, dtype=np.int64)
    rank = np.zeros(M, dtype=np.int64)
    for m in range(M):
        la = a[m] - a[m].max()
        la = la - np.log(np.exp(la).sum())          # log p
        lb = b[m] - b[m].max()
        lb = lb - np.log(np.exp(lb).sum())          # log q
        kl[m] = float(np.sum(np.exp(la) * (la - lb)))
        sq[m] = float(np.sum((a[m] - b[m]) ** 2))
        i = int(np.argmax(a[m]))                    # first index of the maximum
        ref_idx[m] = i
        bi = b[m, i]
        rank[m] = int(np.count_nonzero(b[m] > bi) + np.count_nonzero(b[m, :i] == bi))
    return kl, sq, ref_idx, rank


def topk(logits: np.ndarray, k: int):
    """Top-k selection per row of `logits` [M, V]: the k entries that come
    first when a row is sorted by decreasing value, equal values by
    increasing index (the order behind the top-k agreement above and the
    first-index argmax; the candidate set of top-k decoding).  NaN entries
    are never selected; slots left empty (fewer than k non-NaN entries) are
    (-inf, -1).  Returns (vals [M, k] in the input's precision, idx [M, k]
    int64).  One library sort per row on the key (-value, index).
    """
    a = np.asarray(logits)
    assert a.ndim == 2 and k >= 1
    M, V = a.shape
    vals = np.full((M, k), -np.inf, dtype=a.dtype)
    idx = np.full((M, k), -1, dtype=np.int64)
    for m in range(M):
        ok = np.flatnonzero(~np.isnan(a[m]))
        order = ok[np.lexsort((ok, -a[m, ok]))][:k]   # last key is the primary one
        vals[m, :order.size] = a[m, order]
        idx[m, :order.size] = order
    return vals, idx


def fidelity_summary(kl, sq, rank, ks=(1, 5, 10)) -> dict:
    """Table 8's aggregates over positions: mean KL, MSE (mean squared
    logit error summed over the vocabulary) and top-k agreement in percent."""
    rank = np.asarray(rank)
    out = {"kl": float(np.mean(kl)), "mse": float(np.mean(sq))}
    for k in ks:
        out[f"top{k}"] = 100.0 * float(np.mean(rank < k))
    return out
