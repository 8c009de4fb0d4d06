"""Host-only checks of the page allocator and the append entry point: the C
allocator against the LIFO model in oracle/append_ref.py over random operation
sequences, its error behaviour, and argument checks of sf_decode_attn_append
that must fail before anything reaches the device."""
import ctypes

import numpy as np
import pytest

from oracle.append_ref import PagePoolRef
from paper_2601_12784_amd import binding as B

FAKE = 0x10000  # aligned, never dereferenced


@pytest.mark.parametrize("seed", range(5))
def test_allocator_matches_model(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 200))
    c, m = B.PagePool(n), PagePoolRef(n)
    first = rng.choice(n, size=int(rng.integers(0, n + 1)), replace=False)
    c.claim(first)
    m.claim(first)
    held = list(first)
    for _ in range(300):
        op = rng.integers(0, 3)
        if op == 0:
            k = int(rng.integers(0, 8))
            ok = k <= m.available()
            if ok:
                got = c.alloc(k).tolist()
                assert got == m.alloc(k)
                held += got
            else:
                with pytest.raises(B.SfError):
                    c.alloc(k)
        elif op == 1 and held:
            k = int(rng.integers(1, min(8, len(held)) + 1))
            pick = [held.pop(int(rng.integers(0, len(held)))) for _ in range(k)]
            c.release(pick)
            m.release(pick)
        else:  # an invalid call changes nothing
            bad = [int(rng.integers(-3, n + 3))]
            if bad[0] in held:
                bad = bad * 2
            with pytest.raises(B.SfError):
                c.release(bad)
        assert c.available() == m.available()
    assert c.alloc(m.available()).tolist() == m.alloc(m.available())


def test_allocator_rejects_bad_calls():
    p = B.PagePool(4)
    p.alloc(1)                                   # page 0 in use
    for bad in ([0], [5], [-1], [1, 1]):
        with pytest.raises(B.SfError):
            p.claim(bad)
    for bad in ([1], [0, 0], [9]):
        with pytest.raises(B.SfError):
            p.release(bad)
    with pytest.raises(B.SfError):
        p.alloc(4)
    assert p.available() == 3 and p.alloc(3).tolist() == [1, 2, 3]
    L = B.lib()
    out = ctypes.c_void_p()
    assert L.sf_page_pool_create(-1, ctypes.byref(out)) == 1
    assert L.sf_page_pool_create(3, None) == 1
    assert L.sf_page_pool_available(None) == -1
    assert L.sf_page_pool_alloc(None, 1, FAKE) == 1
    empty = B.PagePool(0)
    assert empty.available() == 0 and empty.alloc(0).size == 0


def _planned():
    lens = np.array((40, 3000), np.int32)
    desc = B.make_desc(2, 8, 2, 128, 200, 400, 0.1)
    info, work = B.sf_decode_attn_plan(desc, lens, B.make_opts(num_cus=4, chunk_pages=16))
    return desc, info


@pytest.mark.parametrize("kw", [dict(k_new=None), dict(v_new=None), dict(k_new=FAKE + 8),
                                dict(v_new=FAKE + 2), dict(pages=FAKE + 2), dict(bt=None), dict(k=None),
                                dict(lse=None), dict(lse=FAKE + 2)])
def test_append_rejects_bad_arguments(kw):
    desc, info = _planned()
    a = dict(k_new=FAKE, v_new=FAKE, pages=None, k=FAKE, v=FAKE, bt=FAKE, lse=FAKE)
    a.update(kw)
    st = B.lib().sf_decode_attn_append(ctypes.byref(desc), ctypes.byref(info), None, FAKE, FAKE, a["k_new"],
                                        a["v_new"], a["pages"], a["k"], a["v"], a["bt"], FAKE, a["lse"], FAKE,
                                        1 << 30, None)
    assert st == 1


def test_page_table_follows_the_oracle_loop():
    """The runner's host bookkeeping (library allocator) hands out the same
    pages, step by step, as the oracle's replay of the schedule."""
    from oracle.append_ref import DecodeLoopRef
    from paper_2601_12784_amd.workloads import bf16_bits, make_decode_loop
    run = make_decode_loop(lens=[1, 15, 16, 17, 40, 200, 3, 700, 33, 2047], steps=60, cap_extra_max=50,
                           seed=23, num_q_heads=4, num_kv_heads=1, head_dim=64)
    b = run.base
    ref = DecodeLoopRef(b.seq_lens, run.caps, bf16_bits(b.k_pool).copy(), bf16_bits(b.v_pool).copy(),
                        b.block_table.copy(), bf16_bits(run.k_new), bf16_bits(run.v_new))
    table = B.PageTable(b.num_pages, b.block_table, b.seq_lens)
    reused = 0
    for t in range(1, run.steps):
        ref.advance()
        free_before = table.pool.available()
        pages = table.advance(run.lengths(t))
        assert np.array_equal(pages, ref.new_pages), t
        reused += int((pages >= 0).sum() > free_before - table.pool.available())
        for s, L in enumerate(run.lengths(t)):
            npg = -(-int(L) // 16)
            assert np.array_equal(table.bt[s, :npg], ref.bt[s, :npg])
        assert table.pool.available() == ref.pool.available()
    assert reused > 0  # some steps took pages that sequences released in the same step


def test_block_table_check_accepts_what_a_step_reads_and_names_the_first_bad_sequence():
    """sf_check_block_table: entries 0 .. ceil(L/16) - 1 of every sequence must
    lie in [0, num_pages); entries past that, and rows of empty sequences, are
    never read and may hold anything."""
    desc = B.make_desc(4, 8, 2, 128, 3, 10, 0.1)
    bt = np.array([[0, 1, -1], [9, -7, 55], [2, 3, 4], [-1, -1, -1]], np.int32)
    lens = np.array([17, 16, 48, 0], np.int32)
    B.check_block_table(desc, bt, lens)                      # all in range where read
    for s, (row, col, val) in enumerate([(0, 1, 10), (1, 0, -1), (2, 2, 10)]):
        bad = bt.copy()
        bad[row, col] = val
        with pytest.raises(B.SfError) as e:
            B.check_block_table(desc, bad, lens)
        assert f"sequence {row}" in str(e.value) and e.value.status == 1
    longer = lens.copy()
    longer[2] = 49                                           # needs a 4th page: more than the stride
    with pytest.raises(B.SfError) as e:
        B.check_block_table(desc, bt, longer)
    assert "sequence 2" in str(e.value)
    # the first bad sequence is the one named
    bad = bt.copy()
    bad[2, 0] = 10
    bad[0, 0] = -3
    with pytest.raises(B.SfError) as e:
        B.check_block_table(desc, bad, lens)
    assert "sequence 0" in str(e.value)
    # raw call: NULL arrays and a bad descriptor
    L = B.lib()
    out = ctypes.c_int32(5)
    assert L.sf_check_block_table(ctypes.byref(desc), None, lens.ctypes.data, ctypes.byref(out)) == 1
    assert out.value == -1
    bad_desc = B.make_desc(4, 8, 3, 128, 3, 10, 0.1)       # 8 q heads over 3 kv heads
    assert L.sf_check_block_table(ctypes.byref(bad_desc), bt.ctypes.data, lens.ctypes.data, None) == 1
