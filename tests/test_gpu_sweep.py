"""Seeded sweep of the decode path over drawn shapes and planner options.

Each case draws, from its seed:
- a head layout (KV heads 1..8, group size 1..16) and head dim (64 or 128);
- a batch of 1..40 sequences with lognormal lengths (median and spread drawn per case),
  some empty, some of length 1 and some whole pages;
- a softmax scale of either sign;
- planner options: CU count, workers per CU, a forced slice width or the free rule,
  minimum slice, and group-parity skew.

The CPU test checks that the library's plan for every case is the plan oracle's, bit
for bit. The GPU test runs the bf16 and the fp8 attention through the C ABI with the
same options and compares out and lse with the fp64 oracle, elementwise within
2e-3 + 1e-2 |ref|.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import plan_ref
from paper_2601_12784_amd import binding as B
from paper_2601_12784_amd.workloads import PAGE, bf16_bits, build_batch, random_fp8_cache

ATOL, RTOL = 2e-3, 1e-2
SEEDS = range(24)


def sweep_case(seed):
    rng = np.random.default_rng(1000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 16]))
    d = int(rng.choice([64, 128]))
    b = int(rng.integers(1, 41))
    median = float(np.exp(rng.uniform(np.log(20), np.log(2000))))
    sigma = float(rng.uniform(0.3, 1.5))
    lens = np.exp(rng.normal(np.log(median), sigma, size=b)).astype(np.int64).clip(1, 4000)
    u = rng.random(b)
    lens[u < 0.08] = 0
    lens[(u >= 0.08) & (u < 0.16)] = 1
    whole = (u >= 0.16) & (u < 0.26)
    lens[whole] = np.maximum(PAGE, lens[whole] // PAGE * PAGE)
    scale = float(rng.choice([1.0, -1.0, 0.5, 2.5])) / math.sqrt(d)
    opts = dict(num_cus=int(rng.choice([1, 3, 8, 64, 256])),
                workers_per_cu=int(rng.choice([0, 1, 2, 3, 4, 5, 6, 8])),
                chunk_pages=int(rng.integers(1, 41)) if rng.random() < 0.3 else 0,
                min_chunk_pages=int(rng.choice([0, 1, 2, 4, 16])),
                xcd_parity_skew=int(rng.choice([0, 20, -20, 60, -60, 150, -150, 250])))
    return dict(seed=seed, hq=hkv * g, hkv=hkv, d=d, lens=lens, scale=scale, opts=opts)


def _describe(c):
    return (f"sweep {c['seed']}: hq={c['hq']} hkv={c['hkv']} d={c['d']} B={c['lens'].size} "
            f"tokens={int(c['lens'].sum())} scale={c['scale']:+.4f} opts={c['opts']}")


@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_plan_matches_oracle(seed):
    """Every sweep case's plan, from the library and from the plan oracle."""
    c = sweep_case(seed)
    lens = c["lens"].astype(np.int32)
    stride = max(1, int(((lens.astype(np.int64) + PAGE - 1) // PAGE).max(initial=1)))
    o = c["opts"]
    desc = B.make_desc(lens.size, c["hq"], c["hkv"], c["d"], stride, 1, c["scale"])
    info, work = B.sf_decode_attn_plan(desc, lens, B.make_opts(**o))
    ref = plan_ref.plan(lens, c["hkv"], c["hq"], c["d"], o["num_cus"], o["chunk_pages"],
                        o["workers_per_cu"] or None, o["min_chunk_pages"] or None, o["xcd_parity_skew"])
    rows = work[: info.work_bytes // 4].reshape(-1, 8)
    t, n = info.num_workers, info.num_work
    assert (info.num_workers, info.workers_per_group, info.chunk_pages, info.num_partials) == \
        (ref["num_workers"], ref["workers_per_group"], ref["chunk_pages"], ref["num_partials"])
    assert np.array_equal(rows[:t], ref["table"])
    assert np.array_equal(rows[t:t + n], ref["items"])
    assert np.array_equal(rows[t + n:], ref["combine"])


def _assert_close(gpu, ref, what):
    gpu = np.asarray(gpu, dtype=np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(gpu), fin), f"{what}: finiteness differs"
    assert np.array_equal(gpu[~fin], ref[~fin]), f"{what}: non-finite values differ"
    err = np.abs(gpu[fin] - ref[fin])
    worst = float((err / (ATOL + RTOL * np.abs(ref[fin]))).max(initial=0.0))
    print(f"  {what}: max|err| {err.max(initial=0):.3e}  worst err/bound {worst:.3f}", flush=True)
    assert worst <= 1.0, f"{what}: tolerance exceeded ({worst:.3f} of bound)"


@pytest.mark.gpu
@pytest.mark.parametrize("seed", SEEDS)
def test_sweep_attention_matches_oracle(seed):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = sweep_case(seed)
    print(_describe(c), flush=True)
    batch = build_batch(c["lens"], c["hq"], c["hkv"], c["d"], 5000 + seed,
                        pool_pages=int(((c["lens"] + PAGE - 1) // PAGE).sum()) + 5)
    batch = dataclasses.replace(batch, scale=c["scale"])
    opts = B.make_opts(**c["opts"])
    q = batch.q.cuda()
    bt = torch.from_numpy(batch.block_table).cuda()
    hq = c["hq"]

    ro, rl = oracle.decode_attn(bf16_bits(batch.q), bf16_bits(batch.k_pool), bf16_bits(batch.v_pool),
                                batch.block_table, batch.seq_lens, batch.scale)
    runner = B.DecodeAttention(hq, c["hkv"], c["d"], opts=opts)
    lse = torch.empty((batch.num_seqs, hq), dtype=torch.float32, device="cuda")
    out = runner(q, batch.k_pool.cuda(), batch.v_pool.cuda(), bt, batch.seq_lens, batch.scale, lse=lse)
    torch.cuda.synchronize()
    info = runner.last_info
    print(f"  bf16: {info.num_workers} workers in groups of {info.workers_per_group}, "
          f"{info.num_work} segments, {info.num_combine} cut pairs", flush=True)
    _assert_close(out.cpu().numpy(), ro, "bf16 out")
    _assert_close(lse.cpu().numpy(), rl, "bf16 lse")

    cache = random_fp8_cache(batch, seed=6000 + seed)
    ro8, rl8 = oracle.decode_attn_fp8(bf16_bits(batch.q), cache.k8.numpy(), cache.v8.numpy(),
                                      cache.k_scale.numpy(), cache.v_scale.numpy(), batch.block_table,
                                      batch.seq_lens, batch.scale)
    runner8 = B.DecodeAttention(hq, c["hkv"], c["d"], opts=opts)
    lse8 = torch.empty_like(lse)
    out8 = runner8(q, cache.k8.cuda(), cache.v8.cuda(), bt, batch.seq_lens, batch.scale, lse=lse8,
                   fp8=(cache.k_scale.cuda(), cache.v_scale.cuda()))
    torch.cuda.synchronize()
    info8 = runner8.last_info
    print(f"  fp8: {info8.num_workers} workers in groups of {info8.workers_per_group}, "
          f"{info8.num_work} segments, {info8.num_combine} cut pairs", flush=True)
    _assert_close(out8.cpu().numpy(), ro8, "fp8 out")
    _assert_close(lse8.cpu().numpy(), rl8, "fp8 lse")


# ---------------------------------------------------------------------------
# extend (re-prefill) attention: drawn prefixes and new-token counts
# ---------------------------------------------------------------------------
EXTEND_SEEDS = range(12)


def extend_case(seed):
    rng = np.random.default_rng(2000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 3, 5, 7, 8, 16]))
    while hkv * g > 64:
        hkv //= 2
    d = int(rng.choice([64, 128]))
    b = int(rng.integers(1, 7))
    prefix = np.where(rng.random(b) < 0.3, 0, rng.integers(0, 1500, size=b))
    new = rng.integers(0, 500, size=b)
    u = rng.random(b)
    new[u < 0.15] = 0
    new[(u >= 0.15) & (u < 0.3)] = 1
    lens = prefix + new
    scale = float(rng.choice([1.0, -1.0, 2.0])) / math.sqrt(d)
    return dict(seed=seed, hq=hkv * g, hkv=hkv, d=d, lens=lens, q_lens=new, scale=scale,
                k_mult=float(rng.choice([1.0, 3.0])), store=bool(rng.random() < 0.5))


@pytest.mark.parametrize("seed", EXTEND_SEEDS)
def test_sweep_extend_plan_matches_oracle(seed):
    c = extend_case(seed)
    lens = c["lens"].astype(np.int32)
    stride = max(1, int(-(-lens.max() // PAGE)))
    pages = max(1, int((-(-lens.astype(np.int64) // PAGE)).sum()))
    desc = B.make_desc(lens.size, c["hq"], c["hkv"], c["d"], stride, pages, c["scale"])
    info, work = B.sf_extend_attn_plan(desc, lens, c["q_lens"])
    want, per = plan_ref.extend_plan(lens, c["q_lens"], c["hkv"], c["hq"])
    assert info.tokens_per_item == per and info.num_items == want.shape[0]
    assert np.array_equal(np.asarray(work)[: info.work_bytes // 4].reshape(-1, 8), want)


@pytest.mark.gpu
@pytest.mark.parametrize("seed", EXTEND_SEEDS)
def test_sweep_extend_matches_oracle(seed):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from oracle import extend_ref
    from paper_2601_12784_amd.workloads import build_extend
    c = extend_case(seed)
    print(f"extend sweep {seed}: hq={c['hq']} hkv={c['hkv']} d={c['d']} lens={c['lens'].tolist()} "
          f"new={c['q_lens'].tolist()} scale={c['scale']:+.4f} k_mult={c['k_mult']} store={c['store']}", flush=True)
    eb = build_extend(c["lens"], c["q_lens"], c["hq"], c["hkv"], c["d"], seed=7000 + seed, k_mult=c["k_mult"])
    b = eb.batch
    runner = B.ExtendAttention(c["hq"], c["hkv"], c["d"])
    kp, vp = b.k_pool.cuda(), b.v_pool.cuda()
    rows = eb.num_rows
    lse = torch.empty((rows, c["hq"]), dtype=torch.float32, device="cuda")
    out = runner(eb.q.cuda(), kp, vp, torch.from_numpy(b.block_table).cuda(), b.seq_lens, eb.q_lens, c["scale"],
                 lse=lse, k_new=eb.k_new.cuda() if c["store"] else None,
                 v_new=eb.v_new.cuda() if c["store"] else None)
    torch.cuda.synchronize()
    ro, rl = extend_ref.extend_attn(bf16_bits(eb.q), bf16_bits(b.k_pool), bf16_bits(b.v_pool), b.block_table,
                                    b.seq_lens, eb.q_lens, c["scale"])
    assert out.shape == (rows, c["hq"], c["d"])
    if rows:
        _assert_close(out.cpu().numpy(), ro, "extend out")
        _assert_close(lse.cpu().numpy(), rl, "extend lse")
    # the new tokens' keys and values are copies of their pool slots: a store
    # leaves the pools bit for bit as they were
    assert np.array_equal(bf16_bits(kp.cpu()), bf16_bits(b.k_pool))
    assert np.array_equal(bf16_bits(vp.cpu()), bf16_bits(b.v_pool))


# ---------------------------------------------------------------------------
# growing-cache decode loop (append): drawn batches, caps and planner options
# ---------------------------------------------------------------------------
LOOP_SEEDS = range(8)


def loop_case(seed):
    rng = np.random.default_rng(3000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 3, 7, 8, 16]))
    while hkv * g > 64:
        hkv //= 2
    d = int(rng.choice([64, 128]))
    b = int(rng.integers(2, 21))
    median = float(np.exp(rng.uniform(np.log(5), np.log(800))))
    lens = np.exp(rng.normal(np.log(median), 1.0, size=b)).astype(np.int64).clip(1, 3000)
    opts = dict(num_cus=int(rng.choice([1, 8, 64, 256])),
                workers_per_cu=int(rng.choice([0, 1, 2, 4, 6, 8])),
                chunk_pages=int(rng.integers(1, 9)) if rng.random() < 0.25 else 0,
                min_chunk_pages=int(rng.choice([0, 1, 4])),
                xcd_parity_skew=int(rng.choice([0, 40, -40, 250])))
    return dict(seed=seed, hq=hkv * g, hkv=hkv, d=d, lens=lens, steps=int(rng.integers(6, 21)),
                cap_extra_max=int(rng.choice([3, 10, 40])), opts=opts)


@pytest.mark.gpu
@pytest.mark.parametrize("seed", LOOP_SEEDS)
def test_sweep_decode_loop_matches_oracle(seed):
    """Every step's out and lse against the fp64 oracle on the oracle's own
    appended pools; the final pools, block tables and free-page count bit for
    bit (the growing-cache loop's checks, with drawn options)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2601_12784_amd.workloads import make_decode_loop
    from test_gpu_append import run_loop
    c = loop_case(seed)
    print(f"loop sweep {seed}: hq={c['hq']} hkv={c['hkv']} d={c['d']} B={c['lens'].size} "
          f"steps={c['steps']} caps+{c['cap_extra_max']} opts={c['opts']}", flush=True)
    run = make_decode_loop(lens=c["lens"], steps=c["steps"], cap_extra_max=c["cap_extra_max"], seed=8000 + seed,
                           num_q_heads=c["hq"], num_kv_heads=c["hkv"], head_dim=c["d"])
    run_loop(run, check_steps=set(range(c["steps"])), opts=B.make_opts(**c["opts"]))
