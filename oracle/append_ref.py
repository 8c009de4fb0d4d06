"""KV append, page allocation and the growing-cache decode loop, written plainly.

TEST INFRASTRUCTURE ONLY. In a batched decode step every running trajectory
produces one new token (App. B.1), so its cached keys and values grow by one
token per step; the cache lives in fixed-size pages drawn from a pool of
bounded size and is released when the trajectory leaves (the KV-cache budget
and release of Sec. 5.2). This module states that bookkeeping in plain Python
for the tests to compare the HIP path against, bit for bit:

  page allocator: a last-in-first-out free list. A new pool hands out pages
      in increasing id order; a released page is handed out again before any
      page released earlier. claim() takes given pages out of the free list
      (the prompt's pages), keeping the order of the rest.
  append of token t of sequence s: page index t // 16, slot t % 16. If
      t % 16 == 0 the page is new: one page is allocated and recorded in the
      block table. The key's dim d goes to k_pool[page, kvh, d // 8, slot, d % 8]
      and the value's to v_pool[page, kvh, d, slot].
  decode loop step t >= 1: first every sequence that was active at t - 1 and
      is not at t releases its pages (ascending sequence order, each in
      block-table order); then every active sequence appends token
      L_s + t - 1 (ascending sequence order).
"""
from __future__ import annotations

import numpy as np

PAGE = 16


class PagePoolRef:
    """LIFO page allocator over page ids 0 .. num_pages - 1."""

    def __init__(self, num_pages: int):
        self.num_pages = int(num_pages)
        self.free = list(range(self.num_pages - 1, -1, -1))  # top of the stack = end of the list
        self.used = set()

    def available(self) -> int:
        return len(self.free)

    def claim(self, pages) -> None:
        pages = [int(p) for p in pages]
        if len(set(pages)) != len(pages) or any(p in self.used or not 0 <= p < self.num_pages for p in pages):
            raise ValueError("claim: page out of range, repeated or already in use")
        taken = set(pages)
        self.free = [p for p in self.free if p not in taken]
        self.used |= taken

    def alloc(self, n: int) -> list:
        if n < 0 or n > len(self.free):
            raise ValueError("alloc: not enough free pages")
        out = [self.free.pop() for _ in range(n)]
        self.used |= set(out)
        return out

    def release(self, pages) -> None:
        pages = [int(p) for p in pages]
        if len(set(pages)) != len(pages) or any(p not in self.used for p in pages):
            raise ValueError("release: page not in use or repeated")
        for p in pages:
            self.used.remove(p)
            self.free.append(p)


def write_token(k_pool, v_pool, page, slot, k_tok, v_tok) -> None:
    """Stores one token's keys and values (uint16 bf16 bits, [Hkv, D]) into a page slot."""
    hkv, d = k_tok.shape
    for kvh in range(hkv):
        k_pool[page, kvh, :, slot, :] = np.asarray(k_tok[kvh]).reshape(d // 8, 8)
        v_pool[page, kvh, :, slot] = v_tok[kvh]


def append_token(k_pool, v_pool, block_table, pool: PagePoolRef, s: int, t: int, k_tok, v_tok):
    """Appends token t of sequence s; returns the newly allocated page or -1."""
    new = -1
    if t % PAGE == 0:
        new = pool.alloc(1)[0]
        block_table[s, t // PAGE] = new
    write_token(k_pool, v_pool, int(block_table[s, t // PAGE]), t % PAGE, k_tok, v_tok)
    return new


class DecodeLoopRef:
    """Replays a growing-cache decode schedule on CPU copies of the pools.

    lens0 [B], caps [B]; k_pool, v_pool: uint16 arrays (modified in place);
    block_table int32 [B, stride] with each sequence's prompt pages (modified
    in place); num_pages: pool size. k_new, v_new: uint16 [steps, B, Hkv, D].
    """

    def __init__(self, lens0, caps, k_pool, v_pool, block_table, k_new, v_new):
        self.lens0 = np.asarray(lens0, dtype=np.int64)
        self.caps = np.asarray(caps, dtype=np.int64)
        self.k_pool, self.v_pool, self.bt = k_pool, v_pool, block_table
        self.k_new, self.v_new = k_new, v_new
        self.pool = PagePoolRef(k_pool.shape[0])
        prompt = []
        for s, L in enumerate(self.lens0):
            prompt += [int(p) for p in block_table[s, : -(-int(L) // PAGE)]]
        self.pool.claim(prompt)
        self.t = 0
        self.new_pages = np.full(self.lens0.size, -1, dtype=np.int32)  # pages allocated by the last step

    def active(self, t):
        return self.lens0 + t <= self.caps

    def lengths(self, t):
        return np.where(self.active(t), self.lens0 + t, 0).astype(np.int32)

    def advance(self):
        """Moves from step t to t + 1: releases, then appends."""
        t = self.t + 1
        was, now = self.active(t - 1), self.active(t)
        for s in np.nonzero(was & ~now)[0]:
            npg = -(-int(self.lens0[s] + t - 1) // PAGE)
            self.pool.release(self.bt[s, :npg])
        self.new_pages[:] = -1
        for s in np.nonzero(now)[0]:
            self.new_pages[s] = append_token(self.k_pool, self.v_pool, self.bt, self.pool, int(s),
                                             int(self.lens0[s] + t - 1), self.k_new[t, s], self.v_new[t, s])
        self.t = t
