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
