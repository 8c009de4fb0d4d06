"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Acceptance for floating point (bf16 inputs, fp32 accumulation and output):
elementwise |gpu - ref| <= 2e-3 + 1e-2 * |ref| for out and for lse.
Integer and byte work (block-table gathers, plans) must match bit for bit.
"""
import functools
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2601_12784_amd import binding as B
from paper_2601_12784_amd.workloads import (PAGE, bf16_bits, build_batch, make_batch,
                                            make_straggler)

pytestmark = pytest.mark.gpu

ATOL, RTOL = 2e-3, 1e-2


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    _need_gpu()
    B.lib()
    yield
    torch.cuda.synchronize()


def _say(msg):
    print(msg, flush=True)


def to_dev(batch):
    return dict(q=batch.q.cuda(), k=batch.k_pool.cuda(), v=batch.v_pool.cuda(),
                bt=torch.from_numpy(batch.block_table).cuda())


def run_gpu(batch, dev=None, chunk_pages=None, runner=None, lse=True):
    dev = dev or to_dev(batch)
    runner = runner or B.DecodeAttention(batch.num_q_heads, batch.num_kv_heads, batch.head_dim)
    lse_t = torch.empty((batch.num_seqs, batch.num_q_heads), dtype=torch.float32, device="cuda") if lse else None
    out = runner(dev["q"], dev["k"], dev["v"], dev["bt"], batch.seq_lens, batch.scale, lse=lse_t,
                 chunk_pages=chunk_pages)
    torch.cuda.synchronize()
    return out.cpu().numpy(), (lse_t.cpu().numpy() if lse else None), runner


def run_oracle(batch):
    return oracle.decode_attn(bf16_bits(batch.q), bf16_bits(batch.k_pool), bf16_bits(batch.v_pool),
                              batch.block_table, batch.seq_lens, batch.scale)


def assert_close(gpu, ref, what=""):
    gpu = np.asarray(gpu, dtype=np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(gpu), fin), f"{what}: finiteness differs"
    assert np.array_equal(gpu[~fin], ref[~fin]), f"{what}: non-finite values differ"
    err = np.abs(gpu[fin] - ref[fin])
    bound = ATOL + RTOL * np.abs(ref[fin])
    worst = float((err / bound).max(initial=0.0))
    _say(f"  {what}: max|err| {err.max(initial=0):.3e}  worst err/bound {worst:.3f}  n={err.size}")
    assert worst <= 1.0, f"{what}: tolerance exceeded ({worst:.3f} of bound)"


def check_batch(batch, ref=None, chunk_pages=None, dev=None):
    ref = ref or run_oracle(batch)
    out, lse, runner = run_gpu(batch, dev=dev, chunk_pages=chunk_pages)
    tag = f"{batch.name} chunk={chunk_pages}"
    assert_close(out, ref[0], f"{tag} out")
    assert_close(lse, ref[1], f"{tag} lse")
    return out, lse, runner.last_info


@functools.lru_cache(maxsize=None)
def named(name):
    return make_batch(name)


@functools.lru_cache(maxsize=None)
def named_ref(name):
    return run_oracle(named(name))


# ---------------------------------------------------------------------------
# block-table translation: bit exact
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("which", ["tiny", "d128"])
def test_gather_is_bit_exact(which):
    if which == "tiny":
        b = named("tiny")
    else:
        b = build_batch([1, 15, 16, 17, 300, 33], 8, 2, 128, 31, pool_pages=80)
    dev = to_dev(b)
    desc = B.make_desc(b.num_seqs, b.num_q_heads, b.num_kv_heads, b.head_dim,
                       b.block_table.shape[1], b.num_pages, b.scale)
    for s in range(b.num_seqs):
        L = int(b.seq_lens[s])
        for kvh in range(b.num_kv_heads):
            kd = torch.empty((L, b.head_dim), dtype=torch.bfloat16, device="cuda")
            vd = torch.empty_like(kd)
            B.sf_debug_gather_kv(desc, dev["k"], dev["v"], dev["bt"], s, kvh, L, kd, vd)
            torch.cuda.synchronize()
            rk, rv = oracle.gather(bf16_bits(b.k_pool), bf16_bits(b.v_pool), b.block_table, s, kvh, L)
            assert np.array_equal(bf16_bits(kd.cpu()), rk)
            assert np.array_equal(bf16_bits(vd.cpu()), rv)


# ---------------------------------------------------------------------------
# the tiny config, every chunking
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("chunk", [None, 1, 2, 7, 64, 1 << 20])
def test_tiny_parity(chunk):
    _say(f"tiny chunk={chunk}")
    check_batch(named("tiny"), named_ref("tiny"), chunk_pages=chunk)


def test_uploaded_plan_is_reusable():
    """Rerunning a plan already on the device (work_host = NULL) gives the same bits."""
    b = build_batch([5, 700, 3000, 9000], 28, 4, 128, 43)
    dev = to_dev(b)
    desc = B.make_desc(b.num_seqs, 28, 4, 128, b.block_table.shape[1], b.num_pages, b.scale)
    info, work = B.sf_decode_attn_plan(desc, b.seq_lens, B.make_opts(num_cus=256, chunk_pages=5))
    assert info.num_combine > 0
    pinned = torch.from_numpy(work[: info.work_bytes // 4].copy()).pin_memory()
    work_dev = torch.empty(info.work_bytes // 4, dtype=torch.int32, device="cuda")
    ws = torch.empty(info.workspace_bytes, dtype=torch.uint8, device="cuda")
    outs = []
    for rep in range(3):
        out = torch.empty((b.num_seqs, 28, 128), dtype=torch.float32, device="cuda")
        lse = torch.empty((b.num_seqs, 28), dtype=torch.float32, device="cuda")
        B.sf_decode_attn(desc, info, pinned if rep == 0 else None, work_dev, dev["q"], dev["k"], dev["v"],
                         dev["bt"], out, lse, ws)
        B.sf_decode_attn_combine(desc, info, work_dev, ws, out, lse)
        torch.cuda.synchronize()
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
        # the pass leaves the whole work list, queue row included, as planned
        assert np.array_equal(work_dev.cpu().numpy(), pinned.numpy()), f"work list changed (rep {rep})"
    ref = run_oracle(b)
    assert_close(outs[0][0], ref[0], "reused plan")
    assert_close(outs[0][1], ref[1], "reused plan lse")
    for o, l in outs[1:]:
        assert np.array_equal(o, outs[0][0]) and np.array_equal(l, outs[0][1])


def test_few_workers_walk_many_segments():
    """Four workers (one CU) each walk several segments, most of them cut."""
    _say("few workers, many segments")
    b = build_batch([3, 17, 250, 1000, 4096, 0, 777], 28, 4, 128, 44)
    dev = to_dev(b)
    desc = B.make_desc(b.num_seqs, 28, 4, 128, b.block_table.shape[1], b.num_pages, b.scale)
    info, work = B.sf_decode_attn_plan(desc, b.seq_lens, B.make_opts(num_cus=1))
    assert info.num_workers == 4 and info.num_work >= 28 and info.num_combine > 0
    pinned = torch.from_numpy(work[: info.work_bytes // 4].copy()).pin_memory()
    work_dev = torch.empty(info.work_bytes // 4, dtype=torch.int32, device="cuda")
    ws = torch.empty(info.workspace_bytes, dtype=torch.uint8, device="cuda")
    out = torch.empty((b.num_seqs, 28, 128), dtype=torch.float32, device="cuda")
    lse = torch.empty((b.num_seqs, 28), dtype=torch.float32, device="cuda")
    for rep in range(2):
        B.sf_decode_attn(desc, info, pinned if rep == 0 else None, work_dev, dev["q"], dev["k"], dev["v"],
                         dev["bt"], out, lse, ws)
        B.sf_decode_attn_combine(desc, info, work_dev, ws, out, lse)
        torch.cuda.synchronize()
        assert np.array_equal(work_dev.cpu().numpy(), pinned.numpy())
        ref = run_oracle(b)
        assert_close(out.cpu().numpy(), ref[0], f"few workers rep {rep}")
        assert_close(lse.cpu().numpy(), ref[1], f"few workers lse rep {rep}")


def test_chunk_count_invariance():
    b = build_batch([1, 17, 100, 513, 2000, 4099], 28, 4, 128, 32)
    dev = to_dev(b)
    ref = run_oracle(b)
    base, base_lse, _ = run_gpu(b, dev=dev, chunk_pages=1 << 20)
    assert_close(base, ref[0], "unsplit")
    for chunk in (1, 2, 7, 64):
        out, lse, runner = run_gpu(b, dev=dev, chunk_pages=chunk)
        assert runner.last_info.num_combine > 0
        assert_close(out, ref[0], f"chunk={chunk}")
        assert_close(lse, ref[1], f"lse chunk={chunk}")
        assert np.allclose(out, base, rtol=1e-4, atol=1e-5), f"chunk={chunk} drifts from unsplit"


# ---------------------------------------------------------------------------
# exact special cases
# ---------------------------------------------------------------------------
def test_length_one_returns_v_row_bitwise():
    b = build_batch([1] * 9, 28, 4, 128, 33)
    out, lse, _ = run_gpu(b)
    g = 7
    vb = bf16_bits(b.v_pool)
    for s in range(9):
        pg = b.block_table[s, 0]
        for h in range(28):
            v = (vb[pg, h // g, :, 0].astype(np.uint32) << 16).view(np.float32)
            assert np.array_equal(out[s, h], v)


def test_dominant_key_returns_its_v_row_bitwise():
    d, length, hot = 128, 200, 137
    b = build_batch([length], 4, 1, d, 34)
    q = np.zeros(d, np.float32)
    q[0] = 64.0
    bf16_bits(b.q)[0, :] = (q.view(np.uint32) >> 16).astype(np.uint16)
    kb = bf16_bits(b.k_pool)  # [N, Hkv, D/8, 16, 8]: dim 0 of slot t at [.., 0, t, 0]
    for t in range(length):
        kb[b.block_table[0, t // PAGE], 0, 0, t % PAGE, 0] = 0x4280 if t == hot else 0  # 64.0 / 0.0
    out, _, _ = run_gpu(b)
    pg = b.block_table[0, hot // PAGE]
    v = (bf16_bits(b.v_pool)[pg, 0, :, hot % PAGE].astype(np.uint32) << 16).view(np.float32)
    for h in range(4):
        assert np.array_equal(out[0, h], v)


def test_empty_sequences_give_zero_and_neg_inf():
    b = build_batch([0, 40, 0, 1, 0], 8, 2, 128, 35)
    ref = run_oracle(b)
    out, lse, _ = run_gpu(b)
    assert np.all(out[[0, 2, 4]] == 0.0) and np.all(np.isneginf(lse[[0, 2, 4]]))
    assert_close(out, ref[0], "with empties")
    assert_close(lse, ref[1], "lse with empties")


def test_all_empty_batch():
    b = build_batch([0, 0], 8, 2, 64, 36)
    out, lse, _ = run_gpu(b)
    assert np.all(out == 0.0) and np.all(np.isneginf(lse))


def test_page_permutation_is_bitwise_invariant():
    b = named("tiny")
    out0, lse0, _ = run_gpu(b)
    perm = np.random.default_rng(5).permutation(b.num_pages)
    k2 = torch.empty_like(b.k_pool)
    v2 = torch.empty_like(b.v_pool)
    k2[torch.from_numpy(perm)] = b.k_pool
    v2[torch.from_numpy(perm)] = b.v_pool
    bt2 = b.block_table.copy()
    bt2[bt2 >= 0] = perm[bt2[bt2 >= 0]]
    dev = dict(q=b.q.cuda(), k=k2.cuda(), v=v2.cuda(), bt=torch.from_numpy(bt2).cuda())
    out1, lse1, _ = run_gpu(b, dev=dev)
    assert np.array_equal(out0, out1) and np.array_equal(lse0, lse1)


def test_run_to_run_bitwise_determinism():
    b = build_batch([3000, 17, 800, 12000], 28, 4, 128, 37)
    dev = to_dev(b)
    o1, l1, _ = run_gpu(b, dev=dev)
    o2, l2, _ = run_gpu(b, dev=dev)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_nan_poisoned_tails_do_not_leak():
    b = build_batch([1, 15, 17, 31, 33, 47], 8, 2, 128, 38, pool_pages=20)
    assert np.any(np.isnan(b.k_pool.float().numpy()))
    out, lse, _ = run_gpu(b)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))


# ---------------------------------------------------------------------------
# ragged mid-size shapes: several tiles and partial pages, every group size
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("hq,hkv,d", [(28, 4, 128), (40, 8, 128), (16, 1, 128), (8, 8, 128),
                                      (4, 1, 64), (32, 2, 64), (7, 7, 64), (64, 4, 128)])
def test_ragged_shapes(hq, hkv, d):
    lens = [1, 2, 15, 16, 17, 31, 32, 33, 255, 257, 1000, 4097]
    b = build_batch(lens, hq, hkv, d, 40 + hq + hkv + d, pool_pages=sum((L + 15) // 16 for L in lens) + 7)
    ref = run_oracle(b)
    _say(f"ragged hq={hq} hkv={hkv} d={d}")
    check_batch(b, ref)
    check_batch(b, ref, chunk_pages=3)


@pytest.mark.parametrize("hq,hkv", [(28, 4), (8, 1)])
def test_one_very_long_sequence(hq, hkv):
    """A 200k-token sequence next to a 1-token one: the default plan cuts each
    of the long sequence's pairs into hundreds of segments (about a thousand
    with one KV head), so one combine row merges that many partials."""
    lens = np.array([200_000, 1], np.int64)
    b = build_batch(lens, hq, hkv, 128, 44)
    ref = run_oracle(b)
    _say(f"very long sequence hq={hq} hkv={hkv}")
    out, lse, info = check_batch(b, ref)
    assert info.num_combine == hkv
    assert info.num_partials >= 250 * hkv


def test_sharp_softmax_scaled_keys():
    """Keys scaled by 3 (the 32B-like workload's sharpening) at mid size."""
    lens = np.random.default_rng(9).integers(1, 6000, size=24)
    b = build_batch(lens, 40, 8, 128, 41, k_mult=3.0)
    check_batch(b)



@pytest.mark.parametrize("chunk", [None, 3])
def test_rising_scores_across_split_pairs(chunk):
    """Scores that climb along the keys (about 130 log2 units over 3000 keys):
    a pair cut into many segments then has partials whose maxima lie far
    apart, so the combine weights its early partials by factors that
    underflow to zero, and the last keys carry the row."""
    lens = np.array([3000, 1000, 17, 1], np.int32)
    b = build_batch(lens, 8, 2, 128, 43)
    kp = b.k_pool.view(torch.int16).numpy()   # [page, KV head, D/8, slot, 8], shares memory
    for s, L in enumerate(lens):
        pos = np.arange(int(L))
        ramp = torch.from_numpy(pos * 0.15).float().to(torch.bfloat16).view(torch.int16).numpy()
        for h in range(b.num_kv_heads):
            kp[b.block_table[s, pos // 16], h, 0, pos % 16, 0] = ramp
    b.q[:, :, 0] = 4.0
    _say(f"rising scores chunk={chunk}")
    check_batch(b, chunk_pages=chunk)

# ---------------------------------------------------------------------------
# the named workloads at full size
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["gqa7b", "longtail", "gqa32b"])
def test_full_size_workload(name):
    _say(f"full-size {name}: generating")
    b = named(name)
    _say(f"  {b.num_seqs} seqs, {int(b.seq_lens.sum())} tokens, {b.kv_bytes() / 1e9:.2f} GB KV")
    ref = named_ref(name)
    out, lse, info = check_batch(b, ref)
    _say(f"  plan: {info.num_work} items, chunk {info.chunk_pages} pages, {info.num_combine} split pairs")


def test_straggler_steps():
    _say("straggler: generating")
    run = make_straggler()
    runner = B.DecodeAttention(28, 4, 128)
    dev = dict(k=run.base.k_pool.cuda(), v=run.base.v_pool.cuda())
    for t in (0, 1, 31, 63):
        b = run.step_batch(t)
        _say(f"  step {t}: {b.num_seqs} active")
        d = dict(dev, q=b.q.cuda(), bt=torch.from_numpy(b.block_table).cuda())
        ref = run_oracle(b)
        out, lse, _ = run_gpu(b, dev=d, runner=runner)
        assert_close(out, ref[0], f"straggler@{t}")
        assert_close(lse, ref[1], f"straggler@{t} lse")


# ---------------------------------------------------------------------------
# measurement support: the streaming-read probe
# ---------------------------------------------------------------------------
def test_stream_read_probe_runs_and_checks_its_arguments():
    _say("stream-read probe")
    buf = torch.full((1 << 20,), 0x5A, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(64, dtype=torch.uint8, device="cuda")
    for blocks in (1, 7, 4096):
        B.sf_debug_stream_read(buf, sink, blocks)
    B.sf_debug_stream_read(buf[: 16 * 1000 + 16], sink, 3)          # ragged tail of the grid-stride loop
    torch.cuda.synchronize()
    assert not sink.any()                                             # 0x5A... XOR-reduces to 0: nothing stored
    L = B.lib()
    addr, sk = buf.data_ptr(), sink.data_ptr()
    assert L.sf_debug_stream_read(addr, 0, sk, 1, None, None, None) == 0           # empty: nothing launched
    assert L.sf_debug_stream_read(addr + 8, 1024, sk, 1, None, None, None) == 1    # misaligned buffer
    assert L.sf_debug_stream_read(addr, 1000, sk, 1, None, None, None) == 1        # not a multiple of 16
    assert L.sf_debug_stream_read(addr, 1024, sk, 0, None, None, None) == 1        # no blocks
    assert L.sf_debug_stream_read(addr, 1024, sk, 65537, None, None, None) == 1    # too many blocks
    assert L.sf_debug_stream_read(addr, 1024, None, 1, None, None, None) == 1      # no sink


def _elapsed_inside(inner, outer):
    """Both intervals in ms; the kernel-timed one must be positive and lie
    within the one that brackets the whole call."""
    t_in, t_out = inner[0].elapsed_time(inner[1]), outer[0].elapsed_time(outer[1])
    _say(f"  kernel {t_in * 1e3:.1f} us inside a {t_out * 1e3:.1f} us bracket")
    assert 0.0 < t_in <= t_out
    assert outer[0].elapsed_time(inner[0]) >= 0.0 and inner[1].elapsed_time(outer[1]) >= 0.0


def _events(n=2):
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "fp8"])
def test_kernel_timed_events_leave_the_step_unchanged(fp8):
    """Timing events handed to a runner step are filled by the attention
    launch itself (the kernel's own start and end): that launch path must give
    bit-identical results to the plain one, match the oracle, and time an
    interval inside a bracket around the whole step."""
    from paper_2601_12784_amd.workloads import random_fp8_cache
    b = build_batch([3000, 17, 1, 700, 16, 2049], 28, 4, 128, 77, pool_pages=420)
    _say(f"timed launch, fp8={fp8}: lens {b.seq_lens.tolist()}")
    dev = to_dev(b)
    if fp8:
        cache = random_fp8_cache(b, seed=19)
        k, v = cache.k8.cuda(), cache.v8.cuda()
        scales = (cache.k_scale.cuda(), cache.v_scale.cuda())
        ref = oracle.decode_attn_fp8(bf16_bits(b.q), cache.k8.numpy(), cache.v8.numpy(), cache.k_scale.numpy(),
                                     cache.v_scale.numpy(), b.block_table, b.seq_lens, b.scale)
    else:
        k, v, scales, ref = dev["k"], dev["v"], None, run_oracle(b)
    runner = B.DecodeAttention(b.num_q_heads, b.num_kv_heads, b.head_dim)
    stream = torch.cuda.Stream()
    outs = []
    for timed in (False, True):
        out = torch.full((b.num_seqs, b.num_q_heads, b.head_dim), float("nan"), device="cuda")
        lse = torch.full((b.num_seqs, b.num_q_heads), float("nan"), device="cuda")
        inner, outer = _events(), _events()
        outer[0].record(stream)
        runner(dev["q"], k, v, dev["bt"], b.seq_lens, b.scale, out=out, lse=lse, chunk_pages=40, stream=stream,
               attn_events=inner if timed else None, fp8=scales)
        outer[1].record(stream)
        torch.cuda.synchronize()
        assert runner.last_info.num_combine > 0             # cut pairs: the combine launch follows
        if timed:
            _elapsed_inside(inner, outer)
        outs.append((out.cpu().numpy(), lse.cpu().numpy()))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    assert_close(outs[1][0], ref[0], "timed out")
    assert_close(outs[1][1], ref[1], "timed lse")


def test_kernel_timed_events_on_the_read_probe():
    stream = torch.cuda.Stream()
    buf = torch.full((64 << 20,), 0x5A, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(64, dtype=torch.uint8, device="cuda")
    inner, outer = _events(), _events()
    outer[0].record(stream)
    B.sf_debug_stream_read(buf, sink, 2048, stream, events=inner)
    outer[1].record(stream)
    torch.cuda.synchronize()
    _elapsed_inside(inner, outer)
    assert not sink.any()


def test_runner_ring_reuse_with_growing_and_shrinking_plans():
    """One runner, consecutive steps whose work lists grow and shrink (its
    pinned ring slots are rewritten, and regrown, only after the step that read
    them ended): every step against the oracle."""
    runner = B.DecodeAttention(28, 4, 128)
    sizes = [3, 40, 7, 120, 1, 64, 200, 5, 90, 2, 150, 30]
    for i, nseq in enumerate(sizes):
        rng = np.random.default_rng(900 + i)
        lens = np.exp(rng.normal(np.log(600), 1.0, size=nseq)).astype(np.int64).clip(0, 6000)
        lens[rng.random(nseq) < 0.1] = 0
        b = build_batch(lens, 28, 4, 128, 910 + i)
        _say(f"ring reuse step {i}: {nseq} sequences, {int(lens.sum())} tokens")
        o, l, _ = run_gpu(b, runner=runner, chunk_pages=(None if i % 3 else 5))
        ref = run_oracle(b)
        assert_close(o, ref[0], f"ring step {i} out")
        assert_close(l, ref[1], f"ring step {i} lse")


def test_runner_takes_every_plan_option():
    """DecodeAttention hands all of its planner options to its native runner:
    its plan (widest slice, cut pairs) is the host planner's for the same
    options, with no XCD-parity skew and with -120 and 200 per mille. Every
    plan against the oracle."""
    rng = np.random.default_rng(5)
    lens = np.exp(rng.normal(np.log(1500), 1.0, size=24)).astype(np.int64).clip(16, 12000)
    b = build_batch(lens, 28, 4, 128, 78)
    ref = run_oracle(b)
    desc = B.make_desc(b.num_seqs, 28, 4, 128, b.block_table.shape[1], b.num_pages, b.scale)
    widest = set()
    for skew in (-120, 0, 200):
        opts = B.make_opts(num_cus=8, xcd_parity_skew=skew)
        host, _ = B.sf_decode_attn_plan(desc, b.seq_lens, opts)
        runner = B.DecodeAttention(28, 4, 128, opts=opts)
        out, lse, _ = run_gpu(b, runner=runner)
        assert_close(out, ref[0], f"skew {skew} out")
        assert_close(lse, ref[1], f"skew {skew} lse")
        got = runner.last_info
        assert (got.num_workers, got.num_work, got.num_combine, got.chunk_pages) == \
            (host.num_workers, host.num_work, host.num_combine, host.chunk_pages)
        widest.add(got.chunk_pages)
    assert len(widest) == 3   # three different plans reached the kernels


@pytest.mark.parametrize("wpc,group", [(1, 1), (2, 2), (4, 4), (5, 1), (6, 2), (8, 8)])
def test_every_launch_group_size(wpc, group):
    """The plan packs 8, 4 or 2 workers into each attention workgroup when
    that fills whole rounds of one workgroup per CU, else 1; the launch takes
    that size from the plan.
    Each size, with equal slices and with a group-parity skew, against the
    oracle."""
    rng = np.random.default_rng(6)
    lens = np.exp(rng.normal(np.log(1500), 1.0, size=24)).astype(np.int64).clip(16, 12000)
    b = build_batch(lens, 28, 4, 128, 79)
    ref = run_oracle(b)
    for skew in (0, 60):
        runner = B.DecodeAttention(28, 4, 128, opts=B.make_opts(num_cus=8, workers_per_cu=wpc, xcd_parity_skew=skew))
        out, lse, _ = run_gpu(b, runner=runner)
        info = runner.last_info
        _say(f"group {group} skew {skew}: {info.num_workers} workers, {info.num_combine} cut pairs")
        assert info.workers_per_group == group and info.num_workers == 8 * wpc
        assert_close(out, ref[0], f"group {group} skew {skew} out")
        assert_close(lse, ref[1], f"group {group} skew {skew} lse")


def test_runner_steps_switching_streams_in_order():
    """Forty runner steps that move between two streams every five steps, each
    switch ordered by an event wait on the stream before (no host
    synchronization): the runner closes its run of marked steps at every
    switch, so a ring slot is rewritten only after its last reader ended on
    whichever stream that was. Every step against the oracle."""
    runner = B.DecodeAttention(28, 4, 128)
    sizes = [3, 40, 120, 1, 64, 90, 2, 30]
    batches = []
    for i, nseq in enumerate(sizes):
        rng = np.random.default_rng(2900 + i)
        lens = np.exp(rng.normal(np.log(600), 1.0, size=nseq)).astype(np.int64).clip(0, 6000)
        lens[rng.random(nseq) < 0.1] = 0
        batches.append(build_batch(lens, 28, 4, 128, 2910 + i))
    devs = [to_dev(b) for b in batches]
    which = [i % len(batches) for i in range(40)]
    outs = [torch.full((batches[j].num_seqs, 28, 128), float("nan"), device="cuda") for j in which]
    lses = [torch.full((batches[j].num_seqs, 28), float("nan"), device="cuda") for j in which]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    _say("runner steps on two streams, switching every five steps")
    cur = streams[0]
    for i, j in enumerate(which):
        if i and i % 5 == 0:
            nxt = streams[(i // 5) % 2]
            ev = torch.cuda.Event()
            ev.record(cur)
            nxt.wait_event(ev)
            cur = nxt
        b, d = batches[j], devs[j]
        runner(d["q"], d["k"], d["v"], d["bt"], b.seq_lens, b.scale, out=outs[i], lse=lses[i], stream=cur)
    torch.cuda.synchronize()
    refs = [run_oracle(b) for b in batches]
    for i, j in enumerate(which):
        assert_close(outs[i].cpu().numpy(), refs[j][0], f"two-stream step {i} (batch {j}) out")
        assert_close(lses[i].cpu().numpy(), refs[j][1], f"two-stream step {i} (batch {j}) lse")


@pytest.mark.parametrize("reserve", [False, True])
def test_runner_steps_in_flight_with_growing_and_shrinking_plans(reserve):
    """Ninety-six runner steps enqueued back to back, with no synchronization
    between them, cycling over batches whose plans grow and shrink: each step
    plans into a ring slot (32 per runner) while earlier steps still run,
    waits for the step that last read the slot (through the event that marks
    its run of 16 steps, recycling those events as it goes), and regrows
    slots (reserve=False) while other slots are in use. The default-chunk
    runner takes 64 of the steps, twice round its ring. Every step writes its
    own out and lse; one synchronization at the end, then every step against
    the oracle. With reserve=True the runner is sized for the largest batch
    first (sf_runner_reserve)."""
    runner = B.DecodeAttention(28, 4, 128)
    sizes = [3, 40, 7, 120, 1, 64, 200, 5, 90, 2, 150, 30]
    num_steps = 8 * len(sizes)
    batches = []
    for i, nseq in enumerate(sizes):
        rng = np.random.default_rng(1900 + i)
        lens = np.exp(rng.normal(np.log(600), 1.0, size=nseq)).astype(np.int64).clip(0, 6000)
        lens[rng.random(nseq) < 0.1] = 0
        batches.append(build_batch(lens, 28, 4, 128, 1910 + i))
    devs = [to_dev(b) for b in batches]
    which = [i % len(batches) for i in range(num_steps)]
    outs = [torch.full((batches[j].num_seqs, 28, 128), float("nan"), device="cuda") for j in which]
    lses = [torch.full((batches[j].num_seqs, 28), float("nan"), device="cuda") for j in which]
    stream = torch.cuda.Stream()
    if reserve:
        big = max(range(len(batches)), key=lambda i: int(batches[i].seq_lens.sum()))
        for chunk in (None, 5):
            runner.reserve(batches[big].seq_lens, batches[big].num_pages, batches[big].block_table.shape[1],
                           chunk_pages=chunk, stream=stream)
    torch.cuda.synchronize()
    _say(f"in-flight runner steps (reserve={reserve})")
    for i, j in enumerate(which):
        b, d = batches[j], devs[j]
        runner(d["q"], d["k"], d["v"], d["bt"], b.seq_lens, b.scale, out=outs[i], lse=lses[i],
               chunk_pages=(None if i % 3 else 5), stream=stream)
    torch.cuda.synchronize()
    refs = [run_oracle(b) for b in batches]
    for i, j in enumerate(which):
        assert_close(outs[i].cpu().numpy(), refs[j][0], f"in-flight step {i} (batch {j}) out")
        assert_close(lses[i].cpu().numpy(), refs[j][1], f"in-flight step {i} (batch {j}) lse")
