"""Re-derivation of the work plan (length-balanced worker slices) from its written rule.

TEST INFRASTRUCTURE ONLY. The paper balances skewed trajectory lengths across
rollout instances (routing and migration, Sec. 5.3); inside one GPU the same
skew is balanced by giving every resident wave the same number of KV pages.
This module restates that rule in plain Python, independently of the C
planner, so the two can be compared bit for bit:

  pairs p = (s, kvh), s-major; pages_p = ceil(L_s / 16); T = sum_p pages_p
  W = ceil(T / chunk_pages) if chunk_pages > 0
      else min(workers_per_cu * num_cus, ceil(T / min_chunk))   (1 if T = 0 < #pairs)
  G = the largest of 8, 4, 2 with W a positive multiple of G*num_cus, else 1 (workers per launch group)
  worker w owns global pages [floor(T*C(w)/C(W)), floor(T*C(w+1)/C(W))) with
  C(v) = 1000*v + p*D(v), D(v) = v % G if (v // G) is even else G - v % G:
  workers of even groups weigh 1000 + p, of odd groups 1000 - p
  (p = xcd_parity_skew per mille, -250 .. 250, default 0; 0 when chunk_pages
  is forced, when these slices would leave a worker no page, or when they cut
  more than W // 8 pairs more than the equal ones, p = 0, would); cut at pair
  boundaries into segments (items); empty
  pairs go to worker e mod W after its segments; n_p = segments of pair p
  partial slots for pairs with n_p > 1 in pair order, segment c -> base + c

Work list rows (int32 x 8): W worker-table rows (first item, count, then the
first six ints of that item's row), then the items worker by worker
  (seq, kv_head, page_begin, page_end, seq_len, slot or -1, combine index or -1, n_p),
then one combine row per cut pair (seq, kv_head, slot_base, n_p, seq_len, 0, 0, 0).
"""
from __future__ import annotations

import numpy as np

PAGE = 16
DEFAULTS = dict(workers_per_cu=4, min_chunk=8)


def _ceil(a, b):
    return -(-a // b)


def _align(x, a=256):
    return _ceil(x, a) * a


def plan(seq_lens, num_kv_heads, num_q_heads, head_dim, num_cus, chunk_pages=0,
         workers_per_cu=None, min_chunk=None, xcd_parity_skew=0):
    wpc = workers_per_cu or DEFAULTS["workers_per_cu"]
    mn = min_chunk or DEFAULTS["min_chunk"]
    skew = 0 if chunk_pages > 0 else int(xcd_parity_skew)
    lens = [int(x) for x in seq_lens]
    pairs = [(s, kvh) for s in range(len(lens)) for kvh in range(num_kv_heads)]
    pages = [_ceil(lens[s], PAGE) for s, _ in pairs]
    total = sum(pages)
    if not pairs:
        workers = 0
    elif total == 0:
        workers = 1
    elif chunk_pages > 0:
        workers = _ceil(total, chunk_pages)
    else:
        workers = min(wpc * num_cus, _ceil(total, mn))

    group = next((g for g in (8, 4, 2) if workers >= g * num_cus and workers % (g * num_cus) == 0), 1)

    # every (worker, pair) overlap is a segment
    starts = np.cumsum([0] + pages)

    def cuts_for(p):
        def weight_upto(v):      # C(v): the weights of workers 0 .. v - 1
            r = v % group
            return 1000 * v + p * (r if (v // group) % 2 == 0 else group - r)
        return [total * weight_upto(w) // weight_upto(workers) for w in range(workers + 1)] if workers else [0]

    def pairs_cut(bounds):       # pairs with a worker boundary strictly inside them
        inner = np.asarray(bounds[1:-1], dtype=np.int64)
        lo, hi = np.asarray(starts[:-1], np.int64), np.asarray(starts[1:], np.int64)
        first_after = np.searchsorted(inner, lo, side="right")   # boundaries > start
        first_at_end = np.searchsorted(inner, hi, side="left")   # boundaries >= end
        return int(np.count_nonzero(first_at_end > first_after))

    bounds = cuts_for(skew)
    if skew and workers > 1:
        equal = cuts_for(0)
        leaves_one_empty = any(bounds[w + 1] == bounds[w] for w in range(workers))
        if leaves_one_empty or pairs_cut(bounds) - pairs_cut(equal) > workers // 8:
            bounds = equal
    per_worker = [[] for _ in range(workers)]
    seg_of_pair = {p: [] for p in range(len(pairs))}
    for w in range(workers):
        lo, hi = bounds[w], bounds[w + 1]
        for p, npg in enumerate(pages):
            if npg == 0:
                continue
            a, b = max(lo, starts[p]), min(hi, starts[p] + npg)
            if a < b:
                seg = [p, int(a - starts[p]), int(b - starts[p])]
                per_worker[w].append(seg)
                seg_of_pair[p].append(seg)
    empties = [p for p, npg in enumerate(pages) if npg == 0]
    for e, p in enumerate(empties):
        seg = [p, 0, 0]
        per_worker[e % workers].append(seg)
        seg_of_pair[p].append(seg)

    slot, combine, meta = 0, [], {}
    for p in range(len(pairs)):
        n = len(seg_of_pair[p])
        if n > 1:
            meta[p] = (slot, len(combine), n)
            s, kvh = pairs[p]
            combine.append([s, kvh, slot, n, lens[s], 0, 0, 0])
            slot += n

    table = np.zeros((workers, 8), dtype=np.int32)
    rows = []
    for w in range(workers):
        table[w, 0] = len(rows)
        table[w, 1] = len(per_worker[w])
        for p, b, e in per_worker[w]:
            s, kvh = pairs[p]
            if p in meta:
                base, ci, n = meta[p]
                c = [tuple(x) for x in seg_of_pair[p]].index((p, b, e))
                rows.append([s, kvh, b, e, lens[s], base + c, ci, n])
            else:
                rows.append([s, kvh, b, e, lens[s] if e > b else 0, -1, -1, 1])
    items = np.array(rows, dtype=np.int32).reshape(-1, 8)
    for w in range(workers):
        if table[w, 1]:
            table[w, 2:] = items[table[w, 0], :6]
    comb = np.array(combine, dtype=np.int32).reshape(-1, 8)
    g = num_q_heads // num_kv_heads
    ws = _align(slot * g * head_dim * 4) + _align(slot * g * 4) if slot else 0
    return dict(table=table, items=items, combine=comb, num_workers=workers, workers_per_group=group,
                chunk_pages=max(b - a for a, b in zip(bounds, bounds[1:])) if workers and total else 0,
                num_partials=slot, workspace_bytes=ws,
                work_bytes=(table.shape[0] + items.shape[0] + comb.shape[0]) * 8 * 4)


def extend_plan(seq_lens, q_lens, num_kv_heads, num_q_heads, rows_per_item=384):
    """The extend work list, re-derived from its rule: new tokens cut into
    blocks of floor(384 / g) per (sequence, KV head); an item starting at new
    token t0 with nt tokens reads ceil((P_s + t0 + nt) / 32) blocks of 32
    keys; items by that count, largest first, ties in (s, kvh, t0) order.
    Rows: (seq, kv_head, t0, nt, P_s, cu_s, steps, 0)."""
    g = num_q_heads // num_kv_heads
    n = rows_per_item // g
    items = []
    cu = 0
    for s, (L, e) in enumerate(zip(seq_lens, q_lens)):
        L, e = int(L), int(e)
        prefix = L - e
        for kvh in range(num_kv_heads):
            for t0 in range(0, e, n):
                nt = min(n, e - t0)
                steps = _ceil(prefix + t0 + nt, 2 * PAGE)
                items.append((-steps, s, kvh, t0, (s, kvh, t0, nt, prefix, cu, steps, 0)))
        cu += e
    items.sort(key=lambda x: x[:4])
    return np.array([it[4] for it in items], dtype=np.int32).reshape(-1, 8), n
