"""Seeded synthetic decode batches: lengths, paged KV pools, block tables, queries.

This module only draws inputs. It holds none of the attention arithmetic, so
both the HIP path and the CPU oracle can consume the very same bits.

The five workloads mirror the rollout decode step the paper times (one new
token per running trajectory, attending over its cached keys/values; App. B.1,
per-step latency model) with head geometries of the paper's model families
(Table of models, Sec. 6.1) and length distributions that reproduce the
within-instance length skew the paper motivates (Sec. 2.3, Fig. "skewness").
None of the paper's datasets or weights are used: every value is drawn here.

Layouts (all row-major, bf16 stored as torch.bfloat16 on the CPU):
  q        [B, Hq, D]
  k_pool   [N_pages, Hkv, D/8, P, 8]   key of slot t, dim d at [.., d/8, t, d%8]
  v_pool   [N_pages, Hkv, D, P]        value of slot t, dim d at [.., d, t]
  block_table int32 [B, stride]   physical page of logical page j, -1 = unused
  seq_lens int32 [B]              cached tokens per sequence (incl. the current one)

Random-draw recipe (fixed, machine independent):
  rng = numpy PCG64(seed); lengths first, then the page permutation, all from rng.
  q, K and V values come from SeedSequence(seed).spawn(3)[i] for i = 0, 1, 2,
  each split into a fixed number of sub-streams filling consecutive slices of
  the flat tensor with float32 N(0,1) draws, which are multiplied by the
  config's K factor (K only) and rounded to bf16 (round-to-nearest-even).
  Page-tile slots past a sequence's allocated length and pool pages that no
  sequence owns are overwritten with a bf16 quiet NaN, and block-table entries
  past a sequence's pages with -1, so any stray read shows up as NaN or a fault
  the host can see.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np
import torch

PAGE = 16
NAN_BF16 = 0x7FC0
_SUBSTREAMS = 64
_SUBSTREAM_MIN = 1 << 16

# name -> (index, B, Hq, Hkv, D); seeds are 1000 + index
CONFIGS = {
    "tiny": (0, 4, 4, 1, 64),
    "gqa7b": (1, 64, 28, 4, 128),
    "longtail": (2, 256, 28, 4, 128),
    "gqa32b": (3, 128, 40, 8, 128),
    "straggler": (4, 512, 28, 4, 128),
}
STRAGGLER_STEPS = 64


def config_seed(name: str) -> int:
    return 1000 + CONFIGS[name][0]


# ----------------------------------------------------------------------------
# length samplers
# ----------------------------------------------------------------------------
def _lognormal_lengths(rng, n, median, sigma, lo, hi):
    z = rng.standard_normal(n)
    return np.clip(np.rint(np.exp(math.log(median) + sigma * z)), lo, hi).astype(np.int64)


def sample_lengths(name: str, rng: np.random.Generator) -> np.ndarray:
    """Per-sequence KV lengths for a named workload (int64 [B])."""
    if name == "tiny":
        return np.array([17, 64, 130, 300], dtype=np.int64)
    if name == "gqa7b":
        return rng.integers(512, 4096, size=64, endpoint=True).astype(np.int64)
    if name == "longtail":
        return _lognormal_lengths(rng, 256, 2048, 1.0, 256, 16384)
    if name == "gqa32b":
        return _lognormal_lengths(rng, 128, 4096, 0.8, 512, 32768)
    if name == "straggler":
        short = rng.integers(1, 2048, size=502, endpoint=True)
        lens = np.concatenate([short, np.full(10, 32768)])
        return lens[rng.permutation(lens.size)].astype(np.int64)
    raise KeyError(name)


def uniform_lengths_like(lens: np.ndarray) -> np.ndarray:
    """Equal-total-token batch of the same size: floor(T/B) + [i < T mod B]."""
    b = lens.size
    t = int(lens.sum())
    out = np.full(b, t // b, dtype=np.int64)
    out[: t % b] += 1
    return out


# ----------------------------------------------------------------------------
# value draws
# ----------------------------------------------------------------------------
def _fill_normal(seedseq: np.random.SeedSequence, n: int, mult: float) -> torch.Tensor:
    """n float32 N(0,1) draws (times mult) rounded to bf16; fixed sub-stream split."""
    buf = np.empty(n, dtype=np.float32)
    nsub = max(1, min(_SUBSTREAMS, n // _SUBSTREAM_MIN))
    subs = seedseq.spawn(nsub)
    bounds = [n * i // nsub for i in range(nsub + 1)]

    def fill(i):
        seg = buf[bounds[i]:bounds[i + 1]]
        np.random.Generator(np.random.PCG64(subs[i])).standard_normal(out=seg, dtype=np.float32)
        if mult != 1.0:
            seg *= np.float32(mult)

    workers = min(16, os.cpu_count() or 1, nsub)
    if workers > 1:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(nsub)))
    else:
        for i in range(nsub):
            fill(i)
    return torch.from_numpy(buf).to(torch.bfloat16)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """uint16 view of a contiguous CPU bf16 tensor (no copy)."""
    assert t.dtype == torch.bfloat16 and t.is_contiguous() and t.device.type == "cpu"
    return t.view(torch.int16).numpy().view(np.uint16)


# ----------------------------------------------------------------------------
# batches
# ----------------------------------------------------------------------------
@dataclass
class Batch:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_lens: np.ndarray          # int32 [B]
    block_table: np.ndarray       # int32 [B, stride]
    q: torch.Tensor               # bf16 [B, Hq, D]
    k_pool: torch.Tensor          # bf16 [N, Hkv, D/8, P, 8]
    v_pool: torch.Tensor          # bf16 [N, Hkv, D, P]
    scale: float
    alloc_lens: np.ndarray = field(default=None)  # int64 [B] tokens backed by pages
    extra: dict = field(default_factory=dict)

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.size)

    @property
    def num_pages(self) -> int:
        return int(self.k_pool.shape[0])

    def kv_bytes(self, lens=None) -> int:
        """Algorithmic K+V bytes one decode step must read (bf16)."""
        lens = self.seq_lens if lens is None else lens
        return int(np.asarray(lens, dtype=np.int64).sum()) * self.num_kv_heads * self.head_dim * 2 * 2


def build_batch(lens, num_q_heads, num_kv_heads, head_dim, seed, *, name="custom",
                pool_pages=None, k_mult=1.0, alloc_lens=None, poison=True,
                rng=None, num_queries=1) -> Batch:
    """Paged batch for the given lengths.

    alloc_lens (>= lens) is how many tokens each sequence's pages back; the
    pool holds exactly sum(ceil(alloc/16)) pages unless pool_pages is larger,
    in which case the used pages are scattered over the larger pool.
    num_queries > 1 draws that many query sets ([n, B, Hq, D]).
    """
    lens = np.asarray(lens, dtype=np.int64)
    alloc = lens.copy() if alloc_lens is None else np.asarray(alloc_lens, dtype=np.int64)
    assert alloc.shape == lens.shape and np.all(alloc >= lens) and np.all(lens >= 0)
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    b = lens.size
    pages = (alloc + PAGE - 1) // PAGE
    used = int(pages.sum())
    n_pool = used if pool_pages is None else int(pool_pages)
    assert n_pool >= used
    stride = max(1, int(pages.max()) if b else 1)
    perm = rng.permutation(n_pool)[:used]
    bt = np.full((b, stride), -1, dtype=np.int32)
    off = 0
    for i in range(b):
        bt[i, : pages[i]] = perm[off: off + pages[i]]
        off += pages[i]

    ss_q, ss_k, ss_v = np.random.SeedSequence(seed).spawn(3)
    hq, hkv, d = num_q_heads, num_kv_heads, head_dim
    qshape = (b, hq, d) if num_queries == 1 else (num_queries, b, hq, d)
    q = _fill_normal(ss_q, int(np.prod(qshape)), 1.0).view(*qshape)
    k_pool = _fill_normal(ss_k, n_pool * hkv * PAGE * d, k_mult).view(n_pool, hkv, d // 8, PAGE, 8)
    v_pool = _fill_normal(ss_v, n_pool * hkv * d * PAGE, 1.0).view(n_pool, hkv, d, PAGE)

    if poison:
        kb = bf16_bits(k_pool)
        vb = bf16_bits(v_pool)
        owned = np.zeros(n_pool, dtype=bool)
        owned[perm] = True
        kb[~owned] = NAN_BF16
        vb[~owned] = NAN_BF16
        for i in range(b):
            tail = int(alloc[i] % PAGE)
            if pages[i] and tail:
                last = bt[i, pages[i] - 1]
                kb[last, :, :, tail:, :] = NAN_BF16
                vb[last, :, :, tail:] = NAN_BF16

    return Batch(name=name, seed=seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                 seq_lens=lens.astype(np.int32), block_table=bt, q=q, k_pool=k_pool,
                 v_pool=v_pool, scale=1.0 / math.sqrt(d), alloc_lens=alloc)


def make_batch(name: str, seed: int | None = None, poison: bool = True) -> Batch:
    """One of the five named workloads at its full size.

    For "straggler" this is the step-0 view of the multi-step run; use
    make_straggler() for the whole 64-step schedule.
    """
    if name == "straggler":
        return make_straggler(seed=seed, poison=poison).step_batch(0)
    idx, b, hq, hkv, d = CONFIGS[name]
    seed = config_seed(name) if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = sample_lengths(name, rng)
    assert lens.size == b
    pool = 64 if name == "tiny" else None
    k_mult = 3.0 if name == "gqa32b" else 1.0
    return build_batch(lens, hq, hkv, d, seed, name=name, pool_pages=pool, k_mult=k_mult,
                       poison=poison, rng=rng)


@dataclass
class StragglerRun:
    """Multi-step decode over a batch with a few very long sequences.

    Sequence i starts at length L_i and stops after reaching its cap
    cap_i = L_i + U_int[0, 64]: at step t it is active iff L_i + t <= cap_i,
    with KV length L_i + t. Inactive sequences are dropped and the batch is
    compacted; pages never move. The pool already holds every token up to
    each cap, so a step only changes lengths, block-table rows and queries.
    """
    base: Batch                   # lengths = L_i, pages back caps
    caps: np.ndarray              # int64 [B0]
    steps: int
    q_all: torch.Tensor           # bf16 [steps, B0, Hq, D]

    def active(self, t: int) -> np.ndarray:
        return np.nonzero(self.base.seq_lens.astype(np.int64) + t <= self.caps)[0]

    def step_batch(self, t: int) -> Batch:
        idx = self.active(t)
        lens = self.base.seq_lens.astype(np.int64)[idx] + t
        pages = (lens + PAGE - 1) // PAGE
        bt = self.base.block_table[idx].copy()
        cols = np.arange(bt.shape[1])[None, :]
        bt[cols >= pages[:, None]] = -1
        q = self.q_all[t][torch.from_numpy(idx)].contiguous()
        return Batch(name=f"{self.base.name}@{t}", seed=self.base.seed,
                     num_q_heads=self.base.num_q_heads, num_kv_heads=self.base.num_kv_heads,
                     head_dim=self.base.head_dim, seq_lens=lens.astype(np.int32),
                     block_table=bt, q=q, k_pool=self.base.k_pool, v_pool=self.base.v_pool,
                     scale=self.base.scale, alloc_lens=self.base.alloc_lens[idx],
                     extra={"step": t, "active": idx})

    def seq_steps(self) -> int:
        return int(sum(self.active(t).size for t in range(self.steps)))


def make_straggler(seed: int | None = None, steps: int = STRAGGLER_STEPS, poison: bool = True,
                   lens=None, cap_extra_max: int = 64, num_q_heads=28, num_kv_heads=4,
                   head_dim=128) -> StragglerRun:
    """The extreme-straggler schedule (defaults: 502 x U[1,2048] + 10 x 32768, 64 steps).

    lens may be given to build a smaller schedule with the same rules.
    """
    seed = config_seed("straggler") if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    if lens is None:
        lens = sample_lengths("straggler", rng)
    lens = np.asarray(lens, dtype=np.int64)
    caps = lens + rng.integers(0, cap_extra_max, size=lens.size, endpoint=True)
    base = build_batch(lens, num_q_heads, num_kv_heads, head_dim, seed, name="straggler",
                       alloc_lens=caps, poison=poison, rng=rng, num_queries=steps)
    q_all = base.q
    base.q = q_all[0]
    return StragglerRun(base=base, caps=caps, steps=steps, q_all=q_all)


@dataclass
class DecodeLoop:
    """Multi-step decode that grows its own cache (same lengths and caps as the
    extreme-straggler schedule).

    The pool starts with only each sequence's first L_i tokens (its pages
    scattered over a pool of sum_i ceil(cap_i / 16) pages, every other page
    free and NaN-filled). Sequence i is active at step t iff L_i + t <= cap_i,
    with KV length L_i + t; at every step t >= 1 each active sequence appends
    one token, position L_i + t - 1, whose key and value are k_new[t, i] and
    v_new[t, i]. Inactive sequences keep their batch row with length 0.
    """
    base: Batch                   # lengths L_i; block table widened to the caps' stride
    caps: np.ndarray              # int64 [B0]
    steps: int
    q_all: torch.Tensor           # bf16 [steps, B0, Hq, D]
    k_new: torch.Tensor           # bf16 [steps, B0, Hkv, D] (row t = 0 unused)
    v_new: torch.Tensor           # bf16 [steps, B0, Hkv, D]

    def active(self, t: int) -> np.ndarray:
        return self.base.seq_lens.astype(np.int64) + t <= self.caps

    def lengths(self, t: int) -> np.ndarray:
        """int32 [B0]: KV length at step t (0 once a sequence has finished)."""
        return np.where(self.active(t), self.base.seq_lens.astype(np.int64) + t, 0).astype(np.int32)

    def seq_steps(self) -> int:
        return int(sum(int(self.active(t).sum()) for t in range(self.steps)))


def make_decode_loop(seed: int | None = None, steps: int = STRAGGLER_STEPS, poison: bool = True,
                     lens=None, cap_extra_max: int = 64, num_q_heads=28, num_kv_heads=4,
                     head_dim=128) -> DecodeLoop:
    """The growing-cache version of make_straggler(): same seed, lengths and caps;
    new-token keys and values come from SeedSequence(seed).spawn(5)[3] and [4]."""
    seed = config_seed("straggler") if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    if lens is None:
        lens = sample_lengths("straggler", rng)
    lens = np.asarray(lens, dtype=np.int64)
    caps = lens + rng.integers(0, cap_extra_max, size=lens.size, endpoint=True)
    n_pool = int(((caps + PAGE - 1) // PAGE).sum())
    base = build_batch(lens, num_q_heads, num_kv_heads, head_dim, seed, name="decode-loop",
                       pool_pages=n_pool, poison=poison, rng=rng, num_queries=steps)
    stride = max(1, int(((caps + PAGE - 1) // PAGE).max()))
    bt = np.full((lens.size, stride), -1, dtype=np.int32)
    bt[:, : base.block_table.shape[1]] = base.block_table
    base.block_table = bt
    q_all = base.q
    base.q = q_all[0]
    ss = np.random.SeedSequence(seed).spawn(5)
    shape = (steps, lens.size, num_kv_heads, head_dim)
    n = int(np.prod(shape))
    k_new = _fill_normal(ss[3], n, 1.0).view(*shape)
    v_new = _fill_normal(ss[4], n, 1.0).view(*shape)
    return DecodeLoop(base=base, caps=caps, steps=steps, q_all=q_all, k_new=k_new, v_new=v_new)


# ----------------------------------------------------------------------------
# extend (re-prefill) batches
# ----------------------------------------------------------------------------
@dataclass
class ExtendBatch:
    """Extend attention input: every sequence's cache holds L_s tokens, the
    last E_s of which are new (positions L_s - E_s .. L_s - 1; query rows in
    sequence order). The pools already hold the new tokens; k_new and v_new
    are those same keys and values ([T, Hkv, D]) for the store path."""
    batch: Batch
    q_lens: np.ndarray            # int32 [B]
    q: torch.Tensor               # bf16 [T, Hq, D]
    k_new: torch.Tensor           # bf16 [T, Hkv, D]
    v_new: torch.Tensor

    @property
    def num_rows(self) -> int:
        return int(self.q_lens.sum())

    def slots(self):
        """(page, slot) of every new token, in row order."""
        pages, slots = [], []
        for s, (L, e) in enumerate(zip(self.batch.seq_lens, self.q_lens)):
            pos = np.arange(int(L) - int(e), int(L))
            pages.append(self.batch.block_table[s, pos // PAGE])
            slots.append(pos % PAGE)
        if not pages:
            return np.zeros(0, np.int64), np.zeros(0, np.int64)
        return np.concatenate(pages).astype(np.int64), np.concatenate(slots).astype(np.int64)

    def causal_flops(self) -> int:
        """Multiply-adds x 2 of the causal QK^T and PV products: each new
        token at position p pairs with p + 1 keys, 4*D flops per pair and head."""
        tot = 0
        for L, e in zip(self.batch.seq_lens.astype(np.int64), self.q_lens.astype(np.int64)):
            p0 = L - e
            tot += int(e * (p0 + 1) + e * (e - 1) // 2)
        return tot * self.batch.num_q_heads * 4 * self.batch.head_dim


def build_extend(lens, q_lens, num_q_heads, num_kv_heads, head_dim, seed, *, name="extend",
                 poison=True, rng=None, pool_pages=None, k_mult=1.0) -> ExtendBatch:
    """Pools as build_batch() for the full lengths, queries for every new
    token from SeedSequence(seed).spawn(6)[5], and the new tokens' keys and
    values copied out of the pools."""
    lens = np.asarray(lens, dtype=np.int64)
    q_lens = np.asarray(q_lens, dtype=np.int64)
    assert q_lens.shape == lens.shape and np.all(q_lens >= 0) and np.all(q_lens <= lens)
    b = build_batch(lens, num_q_heads, num_kv_heads, head_dim, seed, name=name, poison=poison, rng=rng,
                    pool_pages=pool_pages, k_mult=k_mult)
    t = int(q_lens.sum())
    ss = np.random.SeedSequence(seed).spawn(6)[5]
    q = _fill_normal(ss, t * num_q_heads * head_dim, 1.0).view(t, num_q_heads, head_dim)
    eb = ExtendBatch(batch=b, q_lens=q_lens.astype(np.int32), q=q, k_new=None, v_new=None)
    pages, slots = eb.slots()
    kp = b.k_pool.view(torch.int16).numpy()
    vp = b.v_pool.view(torch.int16).numpy()
    kn = kp[pages, :, :, slots, :].reshape(t, num_kv_heads, head_dim)   # [T, Hkv, D/8, 8] -> [T, Hkv, D]
    vn = vp[pages, :, :, slots].reshape(t, num_kv_heads, head_dim)
    eb.k_new = torch.from_numpy(np.ascontiguousarray(kn)).view(torch.bfloat16)
    eb.v_new = torch.from_numpy(np.ascontiguousarray(vn)).view(torch.bfloat16)
    return eb


REPREFILL = dict(num_seqs=32, num_q_heads=28, num_kv_heads=4, head_dim=128)


def make_reprefill(seed: int | None = None, poison: bool = True, num_seqs=None) -> ExtendBatch:
    """Full re-prefill of resumed trajectories: 32 sequences with the long-tail
    lengths (lognormal, median 2048, sigma 1.0, clipped to [256, 16384]), every
    token new (E_s = L_s), 28 query / 4 KV heads, head_dim 128."""
    seed = 1000 + 5 if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    n = REPREFILL["num_seqs"] if num_seqs is None else num_seqs
    lens = _lognormal_lengths(rng, n, 2048, 1.0, 256, 16384)
    return build_extend(lens, lens, REPREFILL["num_q_heads"], REPREFILL["num_kv_heads"], REPREFILL["head_dim"],
                        seed, name="reprefill", poison=poison, rng=rng)


# ----------------------------------------------------------------------------
# fp8 (E4M3) caches for the fp8 decode path
# ----------------------------------------------------------------------------
NAN_FP8 = 0x7F


@dataclass
class Fp8Cache:
    """An fp8 KV cache for a Batch's block table: E4M3 codes, [N, Hkv, 16*D]
    bytes per pool in the fp8 tile layouts (include/sf_decode_attn.h), and
    fp32 scales per (page, KV head)."""
    k8: torch.Tensor              # uint8 [N, Hkv, 16*D]
    v8: torch.Tensor              # uint8 [N, Hkv, 16*D]
    k_scale: torch.Tensor         # float32 [N, Hkv]
    v_scale: torch.Tensor


def fp8_slot_of_offset(d: int):
    """Slot (0..15) of every byte of an fp8 K tile and V tile (int arrays [16*D]).
    K byte ((a * 16 + t) * 16 + b) holds slot t; V byte
    ((c * 4 + t // 4) * 16 + e) * 16 + f * 4 + t % 4 holds slot t."""
    off = np.arange(PAGE * d)
    return (off // 16) % 16, ((off // 256) % 4) * 4 + off % 4


def random_fp8_cache(batch: Batch, seed: int, poison: bool = True) -> Fp8Cache:
    """Random finite codes for every byte of the batch's pool (uniform over
    the 254 finite codes) and scales U[2^-8, 2^-4], from PCG64(seed). When
    poisoned, pages no sequence owns and the slots past each sequence's
    allocation in its last page hold the NaN code 0x7F."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n, hkv, d = batch.num_pages, batch.num_kv_heads, batch.head_dim
    def codes(shape):
        c = rng.integers(0, 256, size=shape, dtype=np.uint16).astype(np.uint8)
        c[(c & 0x7F) == NAN_FP8] ^= 0x01          # NaN codes -> 0x7E / 0xFE
        return c
    k8 = codes((n, hkv, PAGE * d))
    v8 = codes((n, hkv, PAGE * d))
    ks = rng.uniform(2.0 ** -8, 2.0 ** -4, size=(n, hkv)).astype(np.float32)
    vs = rng.uniform(2.0 ** -8, 2.0 ** -4, size=(n, hkv)).astype(np.float32)
    if poison:
        # Owned pages are the block table's entries (a step view of a
        # multi-step run lists only the pages its current lengths use).
        kslot, vslot = fp8_slot_of_offset(d)
        bt = batch.block_table
        owned = np.zeros(n, dtype=bool)
        owned[bt[bt >= 0]] = True
        alloc = batch.alloc_lens if batch.alloc_lens is not None else batch.seq_lens
        for s in range(batch.num_seqs):
            npg = -(-int(alloc[s]) // PAGE)
            tail = int(alloc[s]) % PAGE
            if npg and tail and npg <= bt.shape[1] and bt[s, npg - 1] >= 0:
                last = bt[s, npg - 1]
                k8[last][:, kslot >= tail] = NAN_FP8
                v8[last][:, vslot >= tail] = NAN_FP8
        k8[~owned] = NAN_FP8
        v8[~owned] = NAN_FP8
    return Fp8Cache(k8=torch.from_numpy(k8), v8=torch.from_numpy(v8), k_scale=torch.from_numpy(ks),
                    v_scale=torch.from_numpy(vs))


def page_fill(batch: Batch):
    """(pages, valid slots) of every page some sequence holds: slots of its
    allocation, in block-table order (int32 arrays)."""
    pages, valid = [], []
    alloc = batch.alloc_lens if batch.alloc_lens is not None else batch.seq_lens
    for s in range(batch.num_seqs):
        L = int(alloc[s])
        for j in range(-(-L // PAGE)):
            pages.append(int(batch.block_table[s, j]))
            valid.append(min(PAGE, L - PAGE * j))
    return np.array(pages, np.int32), np.array(valid, np.int32)
