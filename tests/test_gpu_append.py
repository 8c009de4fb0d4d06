"""Append-then-attend on the GPU, through the C ABI, against the oracle's
replay of the same growing-cache schedule (oracle/append_ref.py).

Bar: the pools and block tables the kernels write equal the oracle's bit for
bit; every step's out and lse satisfy |gpu - ref| <= 2e-3 + 1e-2 * |ref|.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import append_ref
from paper_2601_12784_amd import binding as B
from paper_2601_12784_amd.workloads import PAGE, bf16_bits, make_decode_loop

pytestmark = pytest.mark.gpu

ATOL, RTOL = 2e-3, 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    yield
    torch.cuda.synchronize()


def _say(msg):
    print(msg, flush=True)


def assert_close(gpu, ref, what):
    gpu = np.asarray(gpu, dtype=np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(gpu), fin), f"{what}: finiteness differs"
    assert np.array_equal(gpu[~fin], ref[~fin]), f"{what}: non-finite values differ"
    err = np.abs(gpu[fin] - ref[fin])
    worst = float((err / (ATOL + RTOL * np.abs(ref[fin]))).max(initial=0.0))
    assert worst <= 1.0, f"{what}: tolerance exceeded ({worst:.3f} of bound)"
    return worst


def run_loop(run, check_steps, chunk_pages=None, opts=None):
    b = run.base
    hq, hkv, d = b.num_q_heads, b.num_kv_heads, b.head_dim
    ref = append_ref.DecodeLoopRef(b.seq_lens, run.caps, bf16_bits(b.k_pool).copy(), bf16_bits(b.v_pool).copy(),
                                   b.block_table.copy(), bf16_bits(run.k_new), bf16_bits(run.v_new))
    k, v = b.k_pool.cuda(), b.v_pool.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    attn = B.DecodeAttention(hq, hkv, d, opts=opts) if opts is not None else None
    runner = B.DecodeLoopRunner(hq, hkv, d, k, v, bt, b.block_table, b.seq_lens, b.scale, attn=attn)
    if chunk_pages is not None:
        runner.attn.opts.chunk_pages = chunk_pages
    q_all, k_new, v_new = run.q_all.cuda(), run.k_new.cuda(), run.v_new.cuda()
    qb_all = bf16_bits(run.q_all)
    worst = 0.0
    for t in range(run.steps):
        if t:
            ref.advance()
        lens = run.lengths(t)
        lse = torch.empty((lens.size, hq), dtype=torch.float32, device="cuda")
        out = runner.step(q_all[t], lens, k_new[t] if t else None, v_new[t] if t else None, lse=lse)
        if t in check_steps:
            torch.cuda.synchronize()
            want_o, want_l = oracle.decode_attn(qb_all[t], ref.k_pool, ref.v_pool, ref.bt, ref.lengths(t), b.scale)
            worst = max(worst, assert_close(out.cpu().numpy(), want_o, f"out@{t}"),
                        assert_close(lse.cpu().numpy(), want_l, f"lse@{t}"))
    torch.cuda.synchronize()
    _say(f"  worst err/bound {worst:.3f} over steps {sorted(check_steps)}")
    assert np.array_equal(bf16_bits(k.cpu()), ref.k_pool), "K pool differs from the oracle's"
    assert np.array_equal(bf16_bits(v.cpu()), ref.v_pool), "V pool differs from the oracle's"
    lens = run.lengths(run.steps - 1)
    bt_dev = bt.cpu().numpy()
    for s, L in enumerate(lens):
        npg = -(-int(L) // PAGE)
        assert np.array_equal(bt_dev[s, :npg], ref.bt[s, :npg]), f"block table row {s}"
        assert np.array_equal(runner.bt_host[s, :npg], ref.bt[s, :npg]), f"host block table row {s}"
    assert runner.pool.available() == ref.pool.available()


@pytest.mark.parametrize("hq,hkv,d", [(28, 4, 128), (8, 2, 64), (16, 1, 128)])
def test_decode_loop_small(hq, hkv, d):
    _say(f"decode loop small {hq}/{hkv} d={d}")
    run = make_decode_loop(lens=[1, 15, 16, 17, 40, 200, 3, 700, 33, 2047], steps=40, cap_extra_max=40,
                           seed=21, num_q_heads=hq, num_kv_heads=hkv, head_dim=d)
    run_loop(run, check_steps=set(range(40)))


@pytest.mark.parametrize("chunk", [1, 3])
def test_decode_loop_split_pairs(chunk):
    """Forced small chunks: the newest token's page is read by the last of many segments."""
    _say(f"decode loop chunk={chunk}")
    run = make_decode_loop(lens=[5, 16, 100, 333], steps=20, cap_extra_max=20, seed=22)
    run_loop(run, check_steps=set(range(20)), chunk_pages=chunk)


def test_decode_loop_eight_wave_groups_with_skew():
    """Appending steps launched as eight-wave workgroups (eight workers per CU
    on an 8-CU plan) with a group-parity skew: pools, tables and every step
    against the oracle."""
    _say("decode loop, groups of 8, skew 40")
    run = make_decode_loop(lens=[1, 15, 16, 17, 40, 200, 3, 700, 33, 2047, 5000, 90], steps=24, cap_extra_max=24,
                           seed=23)
    run_loop(run, check_steps=set(range(24)), opts=B.make_opts(num_cus=8, workers_per_cu=8, xcd_parity_skew=40))


def test_decode_loop_full_straggler():
    """The extreme-straggler lengths and caps with a growing cache: 512
    sequences, 64 steps, pages released and reused as sequences finish."""
    _say("decode loop full size: generating")
    run = make_decode_loop()
    _say(f"  {run.base.num_seqs} sequences, {run.base.num_pages} pages, {run.seq_steps()} seq-steps")
    run_loop(run, check_steps={0, 1, 2, 17, 31, 63})
