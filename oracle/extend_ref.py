"""Extend (re-prefill) attention over a paged KV cache, and the store of the
new tokens' keys and values, written plainly.

TEST INFRASTRUCTURE ONLY. When a trajectory is interrupted and resumed on an
instance (partial rollout and migration, Sec. 2.3, coordination techniques
1 and 4), that instance recomputes its KV cache, a re-prefill, before decoding
goes on; prefill and re-prefill take the second largest share of rollout time
(Table "time_breakdown", Sec. 6.5). Such a pass appends E_s new tokens to
sequence s, whose cache then holds L_s tokens: a prefix of P_s = L_s - E_s
tokens that were already cached (0 for a full re-prefill) and the new ones at
positions P_s .. L_s - 1. Every new token's query attends causally:

  new token j of sequence s (position p = P_s + j, query row r = cu_s + j,
  cu_s = E_0 + .. + E_{s-1}), query head h, kvh = h / g:
    z_t      = scale * q[r,h] . K_s[t]            t = 0 .. p
    out[r,h] = sum_t exp(z_t) V_s[t] / sum_t exp(z_t)
    lse[r,h] = ln sum_t exp(z_t)

That is, row r is exactly a decode step over the same block-table row with
length p + 1, and extend_attn evaluates it that way, with the decode oracle
(sf_oracle.c) over one virtual sequence per query row.

Store of the new tokens (before the attention reads them): token j of
sequence s, whose key and value for KV head kvh are k_new[r][kvh] and
v_new[r][kvh] (uint16 bf16 bits [T][Hkv][D]), goes to page
block_table[s][p // 16], slot p % 16, with the layouts of the decode oracle.
"""
from __future__ import annotations

import numpy as np

import oracle
from oracle.append_ref import write_token

PAGE = 16


def cu_lens(q_lens) -> np.ndarray:
    """Query-row offsets cu_s (length B + 1)."""
    e = np.asarray(q_lens, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(e)])


def row_map(seq_lens, q_lens):
    """(sequence, position) of every query row, in row order."""
    seqs, pos = [], []
    for s, (L, e) in enumerate(zip(np.asarray(seq_lens, np.int64), np.asarray(q_lens, np.int64))):
        if not 0 <= e <= L:
            raise ValueError("need 0 <= q_lens[s] <= seq_lens[s]")
        for j in range(int(e)):
            seqs.append(s)
            pos.append(int(L - e + j))
    return np.array(seqs, np.int64), np.array(pos, np.int64)


def extend_attn(q, k_pool, v_pool, block_table, seq_lens, q_lens, scale, rows=None, nthreads: int = 0):
    """fp64 extend attention. q: uint16 [T, Hq, D]; returns (out [n, Hq, D],
    lse [n, Hq]) for the query rows `rows` (all T rows if None)."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    seqs, pos = row_map(seq_lens, q_lens)
    if q.shape[0] != seqs.size:
        raise ValueError("q must have sum(q_lens) rows")
    rows = np.arange(seqs.size) if rows is None else np.asarray(rows, dtype=np.int64)
    bt = np.asarray(block_table, dtype=np.int32)
    virt_bt = np.ascontiguousarray(bt[seqs[rows]]) if rows.size else np.zeros((0, bt.shape[1]), np.int32)
    virt_lens = (pos[rows] + 1).astype(np.int32)
    return oracle.decode_attn(q[rows], k_pool, v_pool, virt_bt, virt_lens, scale, nthreads=nthreads)


def kv_store(k_pool, v_pool, block_table, seq_lens, q_lens, k_new, v_new) -> None:
    """Writes every new token's keys and values into its page slot (in place)."""
    seqs, pos = row_map(seq_lens, q_lens)
    for r in range(seqs.size):
        p = int(pos[r])
        page = int(block_table[seqs[r], p // PAGE])
        write_token(k_pool, v_pool, page, p % PAGE, k_new[r], v_new[r])
