"""Dense numpy float64 softmax attention on explicitly gathered K and V.

TEST INFRASTRUCTURE ONLY. A second, independent code path for tiny inputs:
it gathers the cache with per-token Python indexing, then evaluates
softmax(scale * q K^T) V as whole-matrix numpy float64 operations
(the decode step of App. B.1: one query row per sequence and head).
"""
from __future__ import annotations

import numpy as np


def widen(bits) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def gather_dense(k_pool, v_pool, block_table, seq, kvh, length):
    """[L, D] float64 keys and values of one (sequence, KV head)."""
    k_pool = np.asarray(k_pool)          # [N, Hkv, D/8, P, 8]
    v_pool = np.asarray(v_pool)          # [N, Hkv, D, P]
    page = k_pool.shape[3]
    rows_k, rows_v = [], []
    for t in range(length):
        pg = int(block_table[seq][t // page])
        slot = t % page
        rows_k.append(widen(k_pool[pg, kvh, :, slot, :].reshape(-1)))
        rows_v.append(widen(v_pool[pg, kvh, :, slot]))
    d = v_pool.shape[2]
    if not rows_k:
        return np.zeros((0, d)), np.zeros((0, d))
    return np.stack(rows_k), np.stack(rows_v)


def decode_attn(q, k_pool, v_pool, block_table, seq_lens, scale):
    """Returns (out [B,Hq,D], lse [B,Hq]) in float64."""
    q = np.asarray(q)
    b, hq, d = q.shape
    hkv = np.asarray(k_pool).shape[1]
    g = hq // hkv
    out = np.zeros((b, hq, d))
    lse = np.full((b, hq), -np.inf)
    for s in range(b):
        n = int(seq_lens[s])
        if n == 0:
            continue
        for kvh in range(hkv):
            kd, vd = gather_dense(k_pool, v_pool, block_table, s, kvh, n)
            qs = widen(q[s, kvh * g:(kvh + 1) * g, :])          # [g, D]
            z = scale * (qs @ kd.T)                              # [g, L]
            zmax = z.max(axis=1, keepdims=True)
            w = np.exp(z - zmax)
            den = w.sum(axis=1, keepdims=True)
            out[s, kvh * g:(kvh + 1) * g, :] = (w @ vd) / den
            lse[s, kvh * g:(kvh + 1) * g] = (zmax + np.log(den))[:, 0]
    return out, lse
