"""Re-derivation of the split-K work plan from its written rule.

TEST INFRASTRUCTURE ONLY. The paper balances skewed trajectory lengths across
rollout instances (routing and migration, Sec. 5.2); inside one GPU the same
skew is balanced by cutting long (sequence, KV head) ranges into page-aligned
chunks. This module restates that rule in plain Python so the C planner can be
checked against it bit for bit:

  pages_s = ceil(L_s / 16)
  T       = sum_s pages_s * Hkv                       (page-heads in the batch)
  C       = chunk_pages if given (> 0), else
            clamp(ceil(T / (units_per_cu * num_cus)), min_chunk, max_chunk)
  n_s     = ceil(pages_s / C)                         (0 pages -> one empty item)
  chunk c of (s, kvh) covers pages [floor(c*pages_s/n_s), floor((c+1)*pages_s/n_s))
  items   sorted by page count descending, ties by (s, kvh, c) ascending
  partial slots: pairs with n_s > 1, in (s, kvh) order, chunk c -> base + c
  combine items: one per such pair, in (s, kvh) order

Item rows (int32 x 8):
  attention: seq, kv_head, page_begin, page_end, seq_len, slot (-1 = direct),
             combine index (-1 if n_s = 1), n_s
  combine:   seq, kv_head, slot_base, n_s, 0, 0, 0, 0
"""
from __future__ import annotations

import numpy as np

PAGE = 16
DEFAULTS = dict(units_per_cu=8, min_chunk=16, max_chunk=4096)


def _ceil(a, b):
    return -(-a // b)


def _align(x, a=256):
    return _ceil(x, a) * a


def plan(seq_lens, num_kv_heads, num_q_heads, head_dim, num_cus, chunk_pages=0,
         units_per_cu=None, min_chunk=None, max_chunk=None):
    upc = DEFAULTS["units_per_cu"] if not units_per_cu else units_per_cu
    mn = DEFAULTS["min_chunk"] if not min_chunk else min_chunk
    mx = DEFAULTS["max_chunk"] if not max_chunk else max_chunk
    lens = [int(x) for x in seq_lens]
    pages = [_ceil(L, PAGE) for L in lens]
    total = sum(pages) * num_kv_heads
    if chunk_pages > 0:
        c_pages = chunk_pages
    else:
        c_pages = min(max(_ceil(total, upc * num_cus), mn), mx)

    rows = []      # (size, s, kvh, c, row)
    combine = []
    slot = 0
    for s, (L, npg) in enumerate(zip(lens, pages)):
        for kvh in range(num_kv_heads):
            if npg == 0:
                rows.append((0, s, kvh, 0, [s, kvh, 0, 0, L, -1, -1, 1]))
                continue
            n = _ceil(npg, c_pages)
            for c in range(n):
                b = c * npg // n
                e = (c + 1) * npg // n
                if n > 1:
                    row = [s, kvh, b, e, L, slot + c, len(combine), n]
                else:
                    row = [s, kvh, b, e, L, -1, -1, 1]
                rows.append((e - b, s, kvh, c, row))
            if n > 1:
                combine.append([s, kvh, slot, n, 0, 0, 0, 0])
                slot += n
    rows.sort(key=lambda r: (-r[0], r[1], r[2], r[3]))
    items = np.array([r[4] for r in rows], dtype=np.int32).reshape(-1, 8)
    comb = np.array(combine, dtype=np.int32).reshape(-1, 8)
    g = num_q_heads // num_kv_heads
    if slot:
        ws = _align(slot * g * head_dim * 4) + _align(slot * g * 4)
    else:
        ws = 0
    return dict(items=items, combine=comb, chunk_pages=c_pages, num_partials=slot,
                workspace_bytes=ws, work_bytes=(items.shape[0] + comb.shape[0]) * 8 * 4)
