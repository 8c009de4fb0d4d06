"""Host-only checks of the C ABI: exported symbols, the split-K planner
(bit-exact against the re-derivation in oracle/plan_ref.py), and argument
checks that must reject bad calls before anything reaches the device."""
import ctypes

import numpy as np
import pytest

from oracle import plan_ref
from paper_2601_12784_amd import binding as B

PAGE = 16


@pytest.fixture(scope="module")
def lib():
    return B.lib()


def test_exports_every_declared_function(lib):
    names = B.header_functions()
    assert {"sf_decode_attn_plan", "sf_decode_attn", "sf_decode_attn_combine",
            "sf_debug_gather_kv", "sf_status_string", "sf_version"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_status_strings(lib):
    assert B.version() >> 16 == 1
    for st in range(6):
        assert B.status_string(st)
    assert B.status_string(99) == "unknown status"


def test_struct_sizes_match_header():
    assert ctypes.sizeof(B.sf_attn_desc) == 32
    assert ctypes.sizeof(B.sf_plan_opts) == 20
    assert ctypes.sizeof(B.sf_plan_info) == 48


# ---------------------------------------------------------------------------
# planner parity
# ---------------------------------------------------------------------------
def _plan_both(lens, hq, hkv, d, num_cus=256, chunk=0, wpc=0, mn=0, stride=None, skew=0):
    lens = np.asarray(lens, dtype=np.int32)
    if stride is None:
        stride = max(1, int(((lens.astype(np.int64) + PAGE - 1) // PAGE).max(initial=1)))
    desc = B.make_desc(lens.size, hq, hkv, d, stride, 1, 0.1)
    opts = B.make_opts(num_cus=num_cus, chunk_pages=chunk, workers_per_cu=wpc, min_chunk_pages=mn,
                       xcd_parity_skew=skew)
    info, work = B.sf_decode_attn_plan(desc, lens, opts)
    ref = plan_ref.plan(lens, hkv, hq, d, num_cus, chunk, wpc or None, mn or None, skew)
    return info, work[: info.work_bytes // 4].reshape(-1, 8), ref


def _split(info, work):
    t = info.num_workers
    return work[:t], work[t:t + info.num_work], work[t + info.num_work:]


def _assert_same(info, work, ref):
    assert info.num_workers == ref["num_workers"]
    assert info.workers_per_group == ref["workers_per_group"]
    assert info.chunk_pages == ref["chunk_pages"]
    assert info.num_work == ref["items"].shape[0]
    assert info.num_combine == ref["combine"].shape[0]
    assert info.num_partials == ref["num_partials"]
    assert info.workspace_bytes == ref["workspace_bytes"]
    assert info.work_bytes == ref["work_bytes"]
    table, items, comb = _split(info, work)
    assert np.array_equal(table, ref["table"])
    assert np.array_equal(items, ref["items"])
    assert np.array_equal(comb, ref["combine"])


@pytest.mark.parametrize("seed", range(6))
def test_plan_matches_rederivation_random(seed):
    rng = np.random.default_rng(seed)
    b = int(rng.integers(1, 300))
    lens = np.exp(rng.normal(np.log(1500), 1.2, size=b)).astype(np.int64).clip(0, 40000)
    lens[rng.random(b) < 0.05] = 0
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 4, 5, 7, 16]))
    info, work, ref = _plan_both(lens, hkv * g, hkv, 128, num_cus=int(rng.choice([8, 80, 256])))
    _assert_same(info, work, ref)


@pytest.mark.parametrize("chunk", [1, 2, 7, 64, 1 << 20])
def test_plan_matches_rederivation_forced_chunk(chunk):
    lens = [17, 64, 130, 300, 0, 1, 16, 33]
    info, work, ref = _plan_both(lens, 4, 1, 64, chunk=chunk)
    _assert_same(info, work, ref)


def test_plan_matches_rederivation_knobs():
    lens = np.arange(0, 5000, 37)
    info, work, ref = _plan_both(lens, 28, 4, 128, num_cus=32, wpc=3, mn=5)
    _assert_same(info, work, ref)
    assert info.num_workers == 96


def test_plan_skew_kept_or_dropped_by_cut_count():
    """A skew is dropped where equal slices fall on pair boundaries (equal,
    page-aligned lengths: one pair per worker, no cut) and it would cut more
    than W / 8 pairs more; on skewed lengths it is kept."""
    aligned = [1600] * 8
    for skew in (20, -20):
        a, wa, _ = _plan_both(aligned, 28, 4, 128, num_cus=8, skew=skew)
        e, we, _ = _plan_both(aligned, 28, 4, 128, num_cus=8)
        assert (a.num_workers, a.num_work, a.num_combine) == (32, 32, 0) and np.array_equal(wa, we)
    rng = np.random.default_rng(5)
    lens = np.exp(rng.normal(np.log(1500), 1.0, size=24)).astype(np.int64).clip(16, 12000)
    e, we, _ = _plan_both(lens, 28, 4, 128, num_cus=8)
    for skew in (20, -20):
        s, ws, _ = _plan_both(lens, 28, 4, 128, num_cus=8, skew=skew)
        assert s.chunk_pages > e.chunk_pages                 # kept: the favoured workers own more
        assert s.num_combine - e.num_combine <= s.num_workers // 8


def test_plan_skew_dropped_where_a_worker_would_get_no_page():
    """Slices near one page (minimum slice 1, as many workers as pages): a skew
    would leave some workers without a page, so the plan takes equal slices.
    Every worker then has at least one segment and no segment is empty, and
    the plan oracle agrees. Where the skew leaves every worker a page, it is
    kept."""
    lens = [48] * 40                      # 2 KV heads x 40 x 3 pages: T = 240
    for skew in (100, -100, 250):
        s, ws, ref = _plan_both(lens, 4, 2, 128, num_cus=64, wpc=4, mn=1, skew=skew)
        e, we, _ = _plan_both(lens, 4, 2, 128, num_cus=64, wpc=4, mn=1)
        _assert_same(s, ws, ref)
        assert s.num_workers == 240 and np.array_equal(ws, we)
        table, items, _ = _split(s, ws)
        assert table[:, 1].min() >= 1 and np.all(items[:, 3] > items[:, 2])
    # three pages per worker on skewed lengths: 750 per mille still leaves each two
    rng = np.random.default_rng(5)
    skewed = np.exp(rng.normal(np.log(300), 1.0, size=24)).astype(np.int64).clip(16, 3000)
    s, ws, ref = _plan_both(skewed, 4, 2, 128, num_cus=256, wpc=8, mn=3, skew=250)
    e, we, _ = _plan_both(skewed, 4, 2, 128, num_cus=256, wpc=8, mn=3)
    _assert_same(s, ws, ref)
    assert s.num_workers == e.num_workers and s.chunk_pages > e.chunk_pages
    table, items, _ = _split(s, ws)
    assert table[:, 1].min() >= 1 and np.all(items[:, 3] > items[:, 2])


@pytest.mark.parametrize("skew", [-250, -30, 1, 50, 250])
@pytest.mark.parametrize("num_cus,wpc,group,nseq", [(64, 0, 4, 180), (64, 8, 8, 180), (64, 6, 2, 180),
                                                   (64, 5, 1, 180), (2048, 0, 1, 40)])
def test_plan_matches_rederivation_parity_skew(skew, num_cus, wpc, group, nseq):
    rng = np.random.default_rng(400 + skew)
    lens = np.exp(rng.normal(np.log(2000), 1.0, size=nseq)).astype(np.int64).clip(0, 16384)
    info, work, ref = _plan_both(lens, 28, 4, 128, num_cus=num_cus, wpc=wpc, skew=skew)
    assert info.workers_per_group == group
    _assert_same(info, work, ref)
    # a forced slice size ignores the skew: the same plan with and without it
    a, wa, _ = _plan_both(lens, 28, 4, 128, chunk=400, skew=skew)
    b, wb, _ = _plan_both(lens, 28, 4, 128, chunk=400)
    assert a.num_workers == b.num_workers and np.array_equal(wa, wb)


def test_plan_all_empty_and_no_sequences():
    info, work, ref = _plan_both([0, 0, 0], 8, 2, 128)
    _assert_same(info, work, ref)
    assert info.num_workers == 1 and info.num_work == 6 and info.num_combine == 0
    desc = B.make_desc(0, 8, 2, 128, 1, 1, 0.1)
    info0, _ = B.sf_decode_attn_plan(desc, np.zeros(0, np.int32))
    assert info0.num_workers == 0 and info0.num_work == 0


def test_tiny_plan_by_hand():
    """L = {17, 64, 130, 300}, one KV head: pages {2, 4, 9, 19} laid end to end
    give T = 34 global pages. W = min(8 * 256, ceil(34 / 8)) = 5 workers own
    [0,6) [6,13) [13,20) [20,27) [27,34); pair 2 ([6,15)) is cut once and
    pair 3 ([15,34)) twice."""
    info, work, _ = _plan_both([17, 64, 130, 300], 4, 1, 64)
    assert (info.num_workers, info.num_work, info.num_combine, info.num_partials, info.chunk_pages) == \
        (5, 7, 2, 5, 7)
    table, items, comb = _split(info, work)
    # per worker: first item, count, then the first item's seq, kv_head, pages, length, slot
    assert np.array_equal(table, np.array([[0, 2, 0, 0, 0, 2, 17, -1],
                                           [2, 1, 2, 0, 0, 7, 130, 0],
                                           [3, 2, 2, 0, 7, 9, 130, 1],
                                           [5, 1, 3, 0, 5, 12, 300, 3],
                                           [6, 1, 3, 0, 12, 19, 300, 4]], np.int32))
    expect = [[0, 0, 0, 2, 17, -1, -1, 1],
              [1, 0, 0, 4, 64, -1, -1, 1],
              [2, 0, 0, 7, 130, 0, 0, 2],
              [2, 0, 7, 9, 130, 1, 0, 2],
              [3, 0, 0, 5, 300, 2, 1, 3],
              [3, 0, 5, 12, 300, 3, 1, 3],
              [3, 0, 12, 19, 300, 4, 1, 3]]
    assert np.array_equal(items, np.array(expect, np.int32))
    assert np.array_equal(comb, np.array([[2, 0, 0, 2, 130, 0, 0, 0], [3, 0, 2, 3, 300, 0, 0, 0]], np.int32))
    assert info.workspace_bytes == 5 * 4 * 64 * 4 + 256


@pytest.mark.parametrize("seed,skew,wpc", [(0, 0, 0), (1, 0, 0), (2, -40, 0), (3, 0, 8), (4, 120, 0),
                                           (5, 60, 8), (6, -90, 4), (7, 70, 6), (8, -50, 2), (9, 30, 5)])
def test_plan_invariants(seed, skew, wpc):
    """Every worker owns its share of the T pages to within one page: T / W
    without a parity skew; with skew p, a worker of group floor(w / G) weighs
    1000 + p if the group is even and 1000 - p if it is odd, and owns T times
    its weight over the sum of all weights; G is 8, 4 or 1 as W reaches 8 or
    4 workers per CU; the slices tile [0, T) in order; each pair's segments
    tile [0, pages) in worker order; slots of cut pairs are consecutive; every
    pair appears; empty pairs have one empty item."""
    rng = np.random.default_rng(100 + seed)
    lens = rng.integers(0, 20000, size=int(rng.integers(1, 200)))
    lens[rng.random(lens.size) < 0.1] = 0
    hkv = 4
    num_cus = int(rng.integers(1, 300))
    info, work, _ = _plan_both(lens, 28, hkv, 128, num_cus=num_cus, wpc=wpc, skew=skew)
    table, items, comb = _split(info, work)
    tab = table[:, :2]
    # each worker's row repeats the first six ints of its first item
    assert np.array_equal(table[:, 2:], items[tab[:, 0], :6])
    pages = (lens.astype(np.int64) + PAGE - 1) // PAGE
    total = int(pages.sum()) * hkv
    W = info.num_workers
    assert np.array_equal(tab[:, 0], np.concatenate([[0], np.cumsum(tab[:, 1])[:-1]]))
    assert tab[:, 1].sum() == info.num_work
    G = info.workers_per_group
    assert G == next((g for g in (8, 4, 2) if W >= g * num_cus and W % (g * num_cus) == 0), 1)
    p = skew
    weight = [1000 + p if (w // G) % 2 == 0 else 1000 - p for w in range(W)]
    owned = []
    for w in range(W):
        seg = items[tab[w, 0]: tab[w, 0] + tab[w, 1]]
        got = int((seg[:, 3] - seg[:, 2]).sum())
        share = total * weight[w] / sum(weight)
        assert abs(got - share) < 1.0, (w, got, share)
        owned.append(got)
    assert sum(owned) == total
    if p == 0:
        assert set(owned) <= {total // W, -(-total // W)}
    for s, L in enumerate(lens):
        npg = int(pages[s])
        for kvh in range(hkv):
            mine = items[(items[:, 0] == s) & (items[:, 1] == kvh)]  # in worker order
            n = mine.shape[0]
            assert n >= 1 and np.all(mine[:, 7] == n) and np.all(mine[:, 4] == (L if npg else 0))
            if npg == 0:
                assert n == 1 and mine[0, 2] == mine[0, 3] == 0 and mine[0, 5] == -1
                continue
            assert mine[0, 2] == 0 and mine[-1, 3] == npg
            assert np.all(mine[1:, 2] == mine[:-1, 3]) and np.all(mine[:, 3] > mine[:, 2])
            if n > 1:
                row = comb[mine[0, 6]]
                assert row[0] == s and row[1] == kvh and row[3] == n and row[4] == L
                assert np.array_equal(mine[:, 5], row[2] + np.arange(n))
            else:
                assert mine[0, 5] == -1 and mine[0, 6] == -1
    slots = items[items[:, 5] >= 0, 5]
    assert np.array_equal(np.sort(slots), np.arange(info.num_partials))


def test_plan_rejects_bad_knobs(lib):
    desc = B.make_desc(2, 8, 2, 128, 10, 4, 0.1)
    lens = np.array([10, 20], np.int32)
    info = B.sf_plan_info()
    for field, value in (("num_cus", -1), ("chunk_pages", -1), ("workers_per_cu", -1),
                         ("min_chunk_pages", -1), ("xcd_parity_skew", -251), ("xcd_parity_skew", 251)):
        opts = B.make_opts()
        setattr(opts, field, value)
        assert lib.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, ctypes.byref(opts), None, 0,
                                       ctypes.byref(info)) == 1, field


def test_plan_size_query_and_capacity(lib):
    lens = np.array([100, 5000, 3], np.int32)
    desc = B.make_desc(3, 8, 2, 128, 400, 1, 0.1)
    info = B.sf_plan_info()
    st = lib.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, None, None, 0, ctypes.byref(info))
    assert st == 0 and info.work_bytes > 0
    small = np.zeros(info.work_bytes // 4 - 1, np.int32)
    st = lib.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, None, small.ctypes.data,
                                 small.nbytes, ctypes.byref(info))
    assert st == 3  # SF_ERR_CAPACITY


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 2), ("page_size", 32, 2), ("num_q_heads", 34, 2),
    ("num_q_heads", 31, 1), ("num_seqs", -1, 1), ("block_table_stride", 0, 1),
    ("softmax_scale", float("nan"), 1), ("softmax_scale", float("inf"), 1),
    ("softmax_scale", -2.4e38, 1),  # finite, but scale * log2(e) is not
])
def test_plan_rejects_bad_descriptor(lib, field, value, status):
    desc = B.make_desc(2, 8, 2, 128, 10, 4, 0.1)
    setattr(desc, field, value)
    lens = np.array([10, 20], np.int32)
    info = B.sf_plan_info()
    assert lib.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, None, None, 0,
                                   ctypes.byref(info)) == status


def test_plan_rejects_bad_lengths(lib):
    desc = B.make_desc(2, 8, 2, 128, 2, 4, 0.1)
    info = B.sf_plan_info()
    for lens in ([10, -1], [10, 33]):  # negative; 3 pages > stride 2
        arr = np.array(lens, np.int32)
        assert lib.sf_decode_attn_plan(ctypes.byref(desc), arr.ctypes.data, None, None, 0,
                                       ctypes.byref(info)) == 1


# ---------------------------------------------------------------------------
# sf_decode_attn / combine argument checks (all fail before any HIP call)
# ---------------------------------------------------------------------------
FAKE = 0x10000  # aligned, never dereferenced: every case below must be rejected first


def _planned(lens=(40, 3000)):
    lens = np.array(lens, np.int32)
    desc = B.make_desc(len(lens), 8, 2, 128, 200, 400, 0.1)
    info, work = B.sf_decode_attn_plan(desc, lens, B.make_opts(num_cus=4, chunk_pages=16))
    return desc, info, work


def _call(lib, desc, info, **kw):
    a = dict(work_host=None, work_dev=FAKE, q=FAKE, k=FAKE, v=FAKE, bt=FAKE, out=FAKE, lse=None,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return lib.sf_decode_attn(ctypes.byref(desc), ctypes.byref(info), a["work_host"], a["work_dev"],
                              a["q"], a["k"], a["v"], a["bt"], a["out"], a["lse"], a["ws"],
                              a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), 1), (dict(k=None), 1), (dict(v=None), 1), (dict(bt=None), 1),
    (dict(out=None), 1), (dict(work_dev=None), 1),
    (dict(q=FAKE + 8), 1), (dict(out=FAKE + 4), 1), (dict(bt=FAKE + 2), 1), (dict(lse=FAKE + 1), 1),
    (dict(ws_bytes=0), 3), (dict(ws=None), 1), (dict(ws=FAKE + 8), 1),
])
def test_attn_rejects_bad_arguments(lib, kw, status):
    desc, info, _ = _planned()
    assert info.workspace_bytes > 0
    assert _call(lib, desc, info, **kw) == status


def test_attn_rejects_mismatched_plan(lib):
    desc, info, _ = _planned()
    other = B.make_desc(desc.num_seqs, desc.num_q_heads, desc.num_kv_heads, desc.head_dim,
                        desc.block_table_stride + 1, desc.num_pages, desc.softmax_scale)
    assert _call(lib, other, info) == 4
    bad = B.sf_plan_info.from_buffer_copy(info)
    bad.work_bytes += 32
    assert _call(lib, desc, bad) == 4
    for group in (0, 3, 16):           # the launch packs 1, 2, 4 or 8 waves per workgroup, nothing else
        bad = B.sf_plan_info.from_buffer_copy(info)
        bad.workers_per_group = group
        assert _call(lib, desc, bad) == 4


def test_combine_rejects_bad_arguments(lib):
    desc, info, _ = _planned()
    assert info.num_combine > 0
    c = lib.sf_decode_attn_combine
    assert c(ctypes.byref(desc), ctypes.byref(info), FAKE, FAKE, 0, FAKE, None, None) == 3
    assert c(ctypes.byref(desc), ctypes.byref(info), None, FAKE, 1 << 30, FAKE, None, None) == 1
    assert c(ctypes.byref(desc), ctypes.byref(info), FAKE, FAKE, 1 << 30, FAKE + 4, None, None) == 1
    # a plan without cut pairs makes the combine call a no-op
    lens1 = np.array((40, 200), np.int32)
    one, _ = B.sf_decode_attn_plan(desc, lens1, B.make_opts(num_cus=4, chunk_pages=1 << 20))
    assert one.num_combine == 0
    assert c(ctypes.byref(desc), ctypes.byref(one), None, None, 0, None, None, None) == 0


def test_scratch_step_checks_everything_before_touching_the_device(lib):
    """sf_decode_attn_scratch rejects bad arguments, and a plan whose partials
    exceed its array, before its first HIP call (this runs without a GPU)."""
    desc, info, _ = _planned()
    assert 0 < info.workspace_bytes <= B.SCRATCH_BYTES
    f = lib.sf_decode_attn_scratch

    def call(d=desc, i=info, work=FAKE, q=FAKE, k=FAKE, v=FAKE, bt=FAKE, out=FAKE, lse=None):
        return f(ctypes.byref(d), None if i is None else ctypes.byref(i), work, q, k, v, bt, out, lse, None)

    assert call(i=None) == 1
    assert call(q=None) == 1 and call(work=None) == 1 and call(out=FAKE + 4) == 1 and call(lse=FAKE + 2) == 1
    other = B.make_desc(desc.num_seqs, desc.num_q_heads, desc.num_kv_heads, desc.head_dim,
                        desc.block_table_stride + 1, desc.num_pages, desc.softmax_scale)
    assert call(d=other) == 4
    lens = np.full(64, 4096, np.int32)
    big_desc = B.make_desc(64, 28, 4, 128, 256, 64 * 256, 0.1)
    big, _ = B.sf_decode_attn_plan(big_desc, lens, B.make_opts(num_cus=256, chunk_pages=1))
    assert big.workspace_bytes > B.SCRATCH_BYTES
    assert call(d=big_desc, i=big) == 3
    # a batch of no sequences launches nothing and needs no array
    none_desc = B.make_desc(0, 28, 4, 128, 1, 0, 0.1)
    none, _ = B.sf_decode_attn_plan(none_desc, np.zeros(0, np.int32))
    assert none.num_workers == 0
    assert call(d=none_desc, i=none, work=None, q=None, k=None, v=None, bt=None, out=None) == 0


def test_gather_rejects_bad_arguments(lib):
    desc = B.make_desc(2, 8, 2, 128, 4, 10, 0.1)
    g = lib.sf_debug_gather_kv
    assert g(ctypes.byref(desc), FAKE, FAKE, FAKE, 2, 0, 5, FAKE, FAKE, None) == 1   # seq out of range
    assert g(ctypes.byref(desc), FAKE, FAKE, FAKE, 0, 2, 5, FAKE, FAKE, None) == 1   # kv head
    assert g(ctypes.byref(desc), FAKE, FAKE, FAKE, 0, 0, 65, FAKE, FAKE, None) == 1  # > stride pages
    assert g(ctypes.byref(desc), FAKE, FAKE, FAKE, 0, 0, 5, FAKE + 8, FAKE, None) == 1


def test_empty_pool_only_for_empty_batches(lib):
    info = B.sf_plan_info()
    desc = B.make_desc(2, 8, 2, 128, 1, 0, 0.1)
    zero = np.zeros(2, np.int32)
    assert lib.sf_decode_attn_plan(ctypes.byref(desc), zero.ctypes.data, None, None, 0,
                                   ctypes.byref(info)) == 0
    one = np.array([0, 1], np.int32)
    assert lib.sf_decode_attn_plan(ctypes.byref(desc), one.ctypes.data, None, None, 0,
                                   ctypes.byref(info)) == 1
    # pools may be NULL only with num_pages == 0
    d2 = B.make_desc(2, 8, 2, 128, 1, 5, 0.1)
    info2, _ = B.sf_decode_attn_plan(d2, zero)
    assert _call(lib, d2, info2, k=None) == 1


def test_binding_refuses_host_tensors():
    import torch
    desc, info, work = _planned()
    q = torch.zeros((2, 8, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        B.sf_decode_attn(desc, info, work, torch.zeros(16, dtype=torch.int32), q, q, q,
                         torch.zeros((2, 200), dtype=torch.int32), torch.zeros((2, 8, 128)))
