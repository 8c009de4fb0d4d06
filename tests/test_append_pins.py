"""Pins of the growing-cache oracle (oracle/append_ref.py) on the CPU: the page
allocator against hand-worked sequences, appends against an independent dense
gather, the decode loop's bookkeeping invariants, and the loop against the
already-pinned attention oracle on a schedule whose appended tokens are the
ones a pre-filled pool holds."""
import numpy as np
import pytest

import oracle
from oracle import append_ref, dense_ref
from oracle.append_ref import PagePoolRef
from paper_2601_12784_amd.workloads import bf16_bits, make_decode_loop, make_straggler

PAGE = 16


def test_allocator_hands_out_lowest_first_then_last_released():
    p = PagePoolRef(6)
    p.claim([1, 4])
    assert p.available() == 4
    assert p.alloc(2) == [0, 2]
    p.release([2, 0])          # 0 is now on top, then 2
    assert p.alloc(1) == [0]
    assert p.alloc(2) == [2, 3]
    assert p.alloc(1) == [5]
    assert p.available() == 0
    p.release([4, 1])
    assert p.alloc(2) == [1, 4]


@pytest.mark.parametrize("bad", [
    lambda p: p.alloc(4), lambda p: p.alloc(-1), lambda p: p.release([3]), lambda p: p.release([0, 0]),
    lambda p: p.claim([0]), lambda p: p.claim([9]), lambda p: p.claim([2, 2]),
])
def test_allocator_rejects_without_side_effects(bad):
    p = PagePoolRef(3)
    p.alloc(1)                 # page 0 in use
    before = (list(p.free), set(p.used))
    with pytest.raises(ValueError):
        bad(p)
    assert (p.free, p.used) == before


def test_append_lands_where_the_dense_gather_reads_it():
    rng = np.random.default_rng(3)
    hkv, d, n = 2, 64, 5
    k = rng.integers(0, 0x7F00, size=(n, hkv, d // 8, PAGE, 8)).astype(np.uint16)
    v = rng.integers(0, 0x7F00, size=(n, hkv, d, PAGE)).astype(np.uint16)
    bt = np.array([[3, -1, -1]], np.int32)
    pool = PagePoolRef(n)
    pool.claim([3])
    length = 15
    kd0, vd0 = dense_ref.gather_dense(k, v, bt, 0, 1, length)
    for t in (15, 16, 17):                      # fills page 3, then opens a new page
        kt = rng.integers(0, 0x7F00, size=(hkv, d)).astype(np.uint16)
        vt = rng.integers(0, 0x7F00, size=(hkv, d)).astype(np.uint16)
        new = append_ref.append_token(k, v, bt, pool, 0, t, kt, vt)
        assert new == (0 if t == 16 else -1)
        kd, vd = dense_ref.gather_dense(k, v, bt, 0, 1, t + 1)
        assert np.array_equal(kd[t], dense_ref.widen(kt[1])) and np.array_equal(vd[t], dense_ref.widen(vt[1]))
        assert np.array_equal(kd[:length], kd0) and np.array_equal(vd[:length], vd0)
    assert bt[0, 1] == 0 and pool.used == {0, 3}


def _ref_loop(run):
    b = run.base
    return append_ref.DecodeLoopRef(b.seq_lens, run.caps, bf16_bits(b.k_pool).copy(), bf16_bits(b.v_pool).copy(),
                                    b.block_table.copy(), bf16_bits(run.k_new), bf16_bits(run.v_new))


def test_decode_loop_bookkeeping_invariants():
    run = make_decode_loop(lens=[1, 15, 16, 17, 40, 200, 3], cap_extra_max=40, steps=40, seed=7,
                           num_q_heads=4, num_kv_heads=2, head_dim=64)
    ref = _ref_loop(run)
    n = ref.k_pool.shape[0]
    for t in range(1, run.steps):
        ref.advance()
        lens = ref.lengths(t)
        assert np.array_equal(lens, run.lengths(t))
        held = []
        for s, L in enumerate(lens):
            npg = -(-int(L) // PAGE)
            held += [int(p) for p in ref.bt[s, :npg]]
            if L and (L - 1) % PAGE == 0:
                assert ref.new_pages[s] == ref.bt[s, (L - 1) // PAGE] >= 0
            else:
                assert ref.new_pages[s] == -1
        assert len(held) == len(set(held)) and min(held, default=0) >= 0
        assert set(held) == ref.pool.used and len(held) + ref.pool.available() == n


def test_decode_loop_equals_prefilled_schedule():
    """Appending exactly the tokens a pre-filled pool holds reproduces the
    pre-filled straggler schedule's attention bit for bit (fp64 oracle)."""
    lens = [5, 16, 33, 250, 700, 1]
    pre = make_straggler(lens=lens, steps=24, cap_extra_max=30, seed=11, num_q_heads=8, num_kv_heads=2,
                         head_dim=64)
    b = pre.base
    kb, vb = bf16_bits(b.k_pool), bf16_bits(b.v_pool)
    hkv, d = b.num_kv_heads, b.head_dim
    lens0 = b.seq_lens.astype(np.int64)
    bt0 = b.block_table.copy()
    for s, L in enumerate(lens0):
        bt0[s, -(-int(L) // PAGE):] = -1
    k_new = np.zeros((pre.steps, lens0.size, hkv, d), np.uint16)
    v_new = np.zeros_like(k_new)
    for t in range(1, pre.steps):
        for s in range(lens0.size):
            p = int(lens0[s] + t - 1)
            if p < pre.caps[s]:
                pg = b.block_table[s, p // PAGE]
                k_new[t, s] = kb[pg, :, :, p % PAGE, :].reshape(hkv, d)
                v_new[t, s] = vb[pg, :, :, p % PAGE]
    ref = append_ref.DecodeLoopRef(lens0, pre.caps, kb.copy(), vb.copy(), bt0, k_new, v_new)
    qb_all = bf16_bits(pre.q_all)
    for t in range(pre.steps):
        if t:
            ref.advance()
        step = pre.step_batch(t)
        want_o, want_l = oracle.decode_attn(bf16_bits(step.q), kb, vb, step.block_table, step.seq_lens, b.scale)
        got_o, got_l = oracle.decode_attn(qb_all[t], ref.k_pool, ref.v_pool, ref.bt, ref.lengths(t), b.scale)
        idx = step.extra["active"]
        assert np.array_equal(got_o[idx], want_o) and np.array_equal(got_l[idx], want_l), t
        gone = np.setdiff1d(np.arange(lens0.size), idx)
        assert not got_o[gone].any() and np.all(got_l[gone] == -np.inf)


def test_released_pages_are_reused_in_the_same_step():
    """Sequence 0 (L = 20, cap 25) is last active at step 5 and releases its two
    pages at step 6, where sequence 1 (L = 11) appends token 16 and needs a
    page: it gets sequence 0's second page, the last one released."""
    run = make_decode_loop(lens=[20, 11], steps=8, seed=5, num_q_heads=2, num_kv_heads=1, head_dim=64)
    run.caps = np.array([25, 100])
    ref = _ref_loop(run)
    pages0 = ref.bt[0, :2].copy()
    for _ in range(6):
        ref.advance()
    assert ref.t == 6 and ref.lengths(6).tolist() == [0, 17]
    assert ref.new_pages.tolist() == [-1, pages0[1]] and ref.bt[1, 1] == pages0[1]
