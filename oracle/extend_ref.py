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

extend_attn_dense evaluates the same definition for whole sequences at once:
the sequence's cache gathered densely by the decode oracle's gather, the
scores of all its new rows as one float64 matrix product, the causal limit
applied as a mask, and the softmax and the product with V written out. It
exists because a decode per row costs too much for the longest sequences of
a full-size re-prefill; it is pinned against extend_attn.

Store of the new tokens (before the attention reads them): token j of
sequence s, whose key and value for KV head kvh are k_new[r][kvh] and
v_new[r][kvh] (uint16 bf16 bits [T][Hkv][D]), goes to page
block_table[s][p // 16], slot p % 16, with the layouts of the decode oracle.
"""
from __future__ import annotations

import os

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


def _widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) to float64, exactly."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def extend_attn_dense(q, k_pool, v_pool, block_table, seq_lens, q_lens, scale, seqs, nthreads: int = 0,
                      tok_chunk: int = 128):
    """fp64 extend attention of every new row of the sequences `seqs`.

    Returns (rows, out [n, Hq, D], lse [n, Hq]) with rows the query-row
    indices (in row order of each listed sequence, sequences in the given
    order). Per (sequence, KV head): K_s and V_s gathered densely ([L, D]),
    then for a chunk of new tokens j0 .. j1 - 1 and the g query heads of
    the group, z = scale * Q K_s[:P + j1]^T, key t of token j masked unless
    t <= P + j, m = row max, w = exp(z - m), out = (w V_s) / sum w over the
    keys t <= P + j only, and lse = m + log(sum w)."""
    from concurrent.futures import ThreadPoolExecutor

    q = np.ascontiguousarray(q, dtype=np.uint16)
    lens = np.asarray(seq_lens, np.int64)
    qls = np.asarray(q_lens, np.int64)
    cu = cu_lens(qls)
    hq, d = q.shape[1], q.shape[2]
    hkv = k_pool.shape[1]
    g = hq // hkv
    seqs = [int(s) for s in seqs]
    rows = np.concatenate([np.arange(cu[s], cu[s + 1]) for s in seqs]) if seqs else np.zeros(0, np.int64)
    out = np.empty((rows.size, hq, d), np.float64)
    lse = np.empty((rows.size, hq), np.float64)
    base, jobs = 0, []
    for s in seqs:
        L, e = int(lens[s]), int(qls[s])
        for kvh in range(hkv):
            jobs.append((s, kvh, L, e, base))
        base += e

    def run(job):
        s, kvh, L, e, row_base = job
        if e == 0:
            return
        p0 = L - e
        kd, vd = oracle.gather(k_pool, v_pool, block_table, s, kvh, L)
        K, V = _widen(kd), _widen(vd)
        Q = _widen(q[cu[s]:cu[s + 1], kvh * g:(kvh + 1) * g])           # [e, g, D]
        for j0 in range(0, e, tok_chunk):
            j1 = min(e, j0 + tok_chunk)
            nk = p0 + j1
            z = scale * (Q[j0:j1].reshape(-1, d) @ K[:nk].T)             # [(j1 - j0) g, nk]
            limit = np.repeat(p0 + np.arange(j0, j1), g)
            z[np.arange(nk)[None, :] > limit[:, None]] = -np.inf
            m = z.max(axis=1)
            w = np.exp(z - m[:, None])
            l = w.sum(axis=1)
            # keys [0, common) are inside every row's limit: one product; the
            # rest row by row, over the keys each row sees only (a masked key's
            # value is never multiplied, even by a zero weight)
            common = p0 + j0 + 1
            acc = w[:, :common] @ V[:common]
            for jj in range(j0, j1):
                hi = p0 + jj + 1
                if hi > common:
                    r = slice((jj - j0) * g, (jj - j0 + 1) * g)
                    acc[r] += w[r, common:hi] @ V[common:hi]
            o = acc / l[:, None]
            out[row_base + j0:row_base + j1, kvh * g:(kvh + 1) * g] = o.reshape(j1 - j0, g, d)
            lse[row_base + j0:row_base + j1, kvh * g:(kvh + 1) * g] = (m + np.log(l)).reshape(j1 - j0, g)

    # the longest jobs first, so the pool's tail is short; one BLAS thread per
    # job (the jobs themselves run in parallel)
    jobs.sort(key=lambda j: -j[2] * j[3])
    if nthreads <= 0:
        nthreads = min(16, len(os.sched_getaffinity(0)))
    try:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(1)
    except ImportError:
        limit = None
    try:
        with ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(run, jobs))
    finally:
        if limit is not None:
            limit.restore_original_limits()
    return rows, out, lse


def kv_store(k_pool, v_pool, block_table, seq_lens, q_lens, k_new, v_new) -> None:
    """Writes every new token's keys and values into its page slot (in place)."""
    seqs, pos = row_map(seq_lens, q_lens)
    for r in range(seqs.size):
        p = int(pos[r])
        page = int(block_table[seqs[r], p // PAGE])
        write_token(k_pool, v_pool, page, p % PAGE, k_new[r], v_new[r])
