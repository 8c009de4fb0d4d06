"""Extend (re-prefill) planner and argument checks through the C ABI, on the
CPU: the library's work list against the rule re-derived in
oracle/plan_ref.py, bit for bit, and every host-side rejection."""
import ctypes

import numpy as np
import pytest

from oracle import plan_ref
from paper_2601_12784_amd import binding as B


def _plan(lens, qls, hq, hkv, d=128, stride=None, pages=None):
    lens = np.asarray(lens, np.int32)
    stride = stride or max(1, int(-(-lens.max() // 16)) if lens.size else 1)
    pages = pages if pages is not None else max(1, int((-(-lens.astype(np.int64) // 16)).sum()))
    desc = B.make_desc(lens.size, hq, hkv, d, stride, pages, 0.1)
    info, work = B.sf_extend_attn_plan(desc, lens, qls)
    return desc, info, np.asarray(work)[: info.work_bytes // 4].reshape(-1, 8)


@pytest.mark.parametrize("case", [
    ([37, 5, 64], [37, 5, 64], 28, 4),
    ([90, 33, 17, 48], [20, 1, 17, 16], 4, 2),
    ([40, 16, 1, 0], [0, 9, 1, 0], 7, 7),
    ([5000, 300, 1200], [5000, 44, 1], 16, 1),
    ([129], [47], 8, 1),
])
def test_plan_matches_the_rule(case):
    lens, qls, hq, hkv = case
    desc, info, work = _plan(lens, qls, hq, hkv)
    want, per = plan_ref.extend_plan(lens, qls, hkv, hq)
    assert info.tokens_per_item == per
    assert info.num_items == want.shape[0]
    assert info.num_q_rows == sum(qls)
    assert np.array_equal(work, want)


def test_plan_covers_every_new_token_once_per_kv_head():
    rng = np.random.default_rng(1)
    lens = rng.integers(1, 3000, size=40)
    qls = np.minimum(lens, rng.integers(0, 700, size=40))
    desc, info, work = _plan(lens, qls, 28, 4)
    seen = np.zeros((int(qls.sum()), 4), np.int32)
    cu = np.concatenate([[0], np.cumsum(qls)])
    for seq, kvh, t0, nt, prefix, q0, steps, z in work:
        assert q0 == cu[seq] and prefix == lens[seq] - qls[seq] and z == 0
        assert 1 <= nt <= info.tokens_per_item and steps == -(-(prefix + t0 + nt) // 32)
        seen[q0 + t0: q0 + t0 + nt, kvh] += 1
    assert np.all(seen == 1)
    assert np.all(np.diff(work[:, 6]) <= 0)        # longest key walk first


def test_plan_tiny_by_hand():
    # g = 16 -> floor(384 / 16) = 24 tokens per item; sequence 0: P = 10, E = 20 -> one block (t0 = 0, 20 tokens)
    desc, info, work = _plan([30, 3], [20, 3], 16, 1, d=64)
    assert info.tokens_per_item == 24
    # keys [0, 30) and [0, 3): one step of 32 each, so the tie keeps sequence order
    assert work.tolist() == [[0, 0, 0, 20, 10, 0, 1, 0],
                             [1, 0, 0, 3, 0, 20, 1, 0]]
    desc, info, work = _plan([60, 3], [40, 3], 16, 1, d=64)
    # P = 20: blocks t0 = 0 (24 tokens, keys [0, 44): 2 steps), 24 (16 tokens, keys [0, 60): 2 steps)
    assert work[:, 2].tolist() == [0, 24, 0] and work[:, 3].tolist() == [24, 16, 3]
    assert work[:, 6].tolist() == [2, 2, 1]
    desc, info, work = _plan([100, 3], [80, 3], 16, 1, d=64)
    # P = 20: blocks t0 = 0 (keys [0, 44): 2 steps), 24 ([0, 68): 3), 48 ([0, 92): 3), 72 (8 tokens, [0, 100): 4)
    assert work[:, 2].tolist() == [72, 24, 48, 0, 0] and work[:, 6].tolist() == [4, 3, 3, 2, 1]


@pytest.mark.parametrize("lens,qls", [([10], [11]), ([10], [-1]), ([40], [3])])
def test_plan_rejects_bad_lengths(lens, qls):
    desc = B.make_desc(1, 4, 1, 64, 2, 8, 0.1)        # stride 2 -> at most 32 tokens
    with pytest.raises(B.SfError) as e:
        B.sf_extend_attn_plan(desc, lens, qls)
    assert e.value.status == 1


def test_plan_capacity_and_sizes():
    desc = B.make_desc(2, 4, 2, 64, 4, 8, 0.1)
    info = B.sf_extend_info()
    L = B.lib()
    lens = np.array([40, 20], np.int32)
    qls = np.array([40, 5], np.int32)
    assert L.sf_extend_attn_plan(ctypes.byref(desc), lens.ctypes.data, qls.ctypes.data, None, 0,
                                 ctypes.byref(info)) == 0
    assert info.work_bytes == info.num_items * 32 and info.num_items == 4
    small = np.zeros(8, np.int32)
    assert L.sf_extend_attn_plan(ctypes.byref(desc), lens.ctypes.data, qls.ctypes.data, small.ctypes.data,
                                 small.nbytes, ctypes.byref(info)) == 3


def test_attn_rejects_before_launching():
    """Host-visible argument errors come back before any device call."""
    desc = B.make_desc(1, 4, 1, 64, 2, 4, 0.1)
    info, work = B.sf_extend_attn_plan(desc, [20], [20])
    L = B.lib()
    fake = 1 << 20                  # aligned, never dereferenced on an error path
    args = dict(work_host=None, work_dev=fake, q=fake, k_new=None, v_new=None, k_pool=fake, v_pool=fake,
                bt=fake, out=fake, lse=None)

    def call(info_=info, desc_=desc, **kw):
        a = dict(args, **kw)
        return L.sf_extend_attn(ctypes.byref(desc_), ctypes.byref(info_), a["work_host"], a["work_dev"], a["q"],
                                a["k_new"], a["v_new"], a["k_pool"], a["v_pool"], a["bt"], a["out"], a["lse"],
                                None)
    assert call(q=None) == 1
    assert call(out=fake + 4) == 1                          # misaligned
    assert call(k_new=fake) == 1                            # k_new without v_new
    assert call(k_new=fake + 2, v_new=fake) == 1
    other = B.make_desc(1, 4, 1, 64, 3, 4, 0.1)
    assert call(desc_=other) == 4                           # plan mismatch
    bad = B.sf_extend_info.from_buffer_copy(info)
    bad.tokens_per_item += 1
    assert call(info_=bad) == 4
    unsupported = B.make_desc(1, 4, 1, 96, 2, 4, 0.1)
    assert call(desc_=unsupported) == 2
