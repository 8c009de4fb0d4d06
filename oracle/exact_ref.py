"""High-precision decimal attention for a handful of tokens.

TEST INFRASTRUCTURE ONLY. Brute force at 60 significant digits with the
standard-library decimal module (correctly rounded exp and ln), so its
results are the exact attention values to far below fp64 resolution.
It pins the fp64 oracle on tiny inputs: out = sum_t e^{z_t} v_t / sum_t e^{z_t},
lse = ln sum_t e^{z_t}, with z_t = scale * q.k_t (App. B.1 decode step).
"""
from __future__ import annotations

import struct
from decimal import Decimal, localcontext

import numpy as np

PREC = 60


def bf16_to_decimal(bits: int) -> Decimal:
    """Exact decimal value of a bf16 bit pattern (finite values only)."""
    f = struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]
    return Decimal(f)  # float -> Decimal is exact


def attention_one(q_bits, k_rows_bits, v_rows_bits, scale: Decimal):
    """q_bits [D], k/v_rows_bits [L][D] -> (out [D] Decimal, lse Decimal)."""
    with localcontext() as ctx:
        ctx.prec = PREC
        qd = [bf16_to_decimal(x) for x in q_bits]
        z = []
        for row in k_rows_bits:
            acc = Decimal(0)
            for a, b in zip(qd, row):
                acc += a * bf16_to_decimal(b)
            z.append(scale * acc)
        w = [zz.exp() for zz in z]
        den = sum(w, Decimal(0))
        d = len(qd)
        out = []
        for j in range(d):
            num = Decimal(0)
            for wt, row in zip(w, v_rows_bits):
                num += wt * bf16_to_decimal(row[j])
            out.append(num / den)
        return out, den.ln()


def decode_attn(q, k_pool, v_pool, block_table, seq_lens, scale):
    """Decimal brute force over the paged layout; returns float64 arrays of
    the correctly rounded results plus the Decimal values."""
    q = np.asarray(q)
    k_pool = np.asarray(k_pool)
    v_pool = np.asarray(v_pool)
    b, hq, d = q.shape
    hkv = k_pool.shape[1]                 # k_pool [N, Hkv, D/8, P, 8]
    page = k_pool.shape[3]
    g = hq // hkv
    with localcontext() as ctx:
        ctx.prec = PREC
        sc = Decimal(scale)
    out = np.zeros((b, hq, d))
    lse = np.full((b, hq), -np.inf)
    dec = {}
    for s in range(b):
        n = int(seq_lens[s])
        if n == 0:
            continue
        for h in range(hq):
            kvh = h // g
            krows, vrows = [], []
            for t in range(n):
                pg = int(block_table[s][t // page])
                krows.append([int(x) for x in k_pool[pg, kvh, :, t % page, :].reshape(-1)])
                vrows.append([int(x) for x in v_pool[pg, kvh, :, t % page]])
            o, l = attention_one([int(x) for x in q[s, h, :]], krows, vrows, sc)
            dec[(s, h)] = (o, l)
            out[s, h, :] = [float(x) for x in o]
            lse[s, h] = float(l)
    return out, lse, dec
