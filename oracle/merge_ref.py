"""fp64 log-sum-exp merge of partial attention results.

TEST INFRASTRUCTURE ONLY. Softmax attention over a union of disjoint token
sets A_1..A_n can be rebuilt from each set's normalised output o_c and
log-normaliser lse_c:  M = max_c lse_c,  w_c = exp(lse_c - M),
out = sum_c w_c o_c / sum_c w_c,  lse = M + ln sum_c w_c.
Sets with lse_c = -inf (no tokens) carry no weight.
"""
from __future__ import annotations

import numpy as np


def merge(outs, lses):
    """outs: [n, ..., D], lses: [n, ...]; merges along axis 0."""
    outs = np.asarray(outs, dtype=np.float64)
    lses = np.asarray(lses, dtype=np.float64)
    m = lses.max(axis=0)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    w = np.where(np.isfinite(lses), np.exp(lses - m_safe[None]), 0.0)
    den = w.sum(axis=0)
    num = (w[..., None] * outs).sum(axis=0)
    with np.errstate(invalid="ignore", divide="ignore"):
        out = np.where(finite[..., None], num / np.where(den > 0, den, 1.0)[..., None], 0.0)
        lse = np.where(finite, m_safe + np.log(np.where(den > 0, den, 1.0)), -np.inf)
    return out, lse
