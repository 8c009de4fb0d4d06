"""GPU parity of the fp8 (OCP E4M3) KV path against the fp64 oracle, through the C ABI.

Attention over an fp8 cache: every code widens exactly to bf16 and the
kernel then runs the bf16 path, with each page's K scale in the score scale
and its V scale in the P.V operand (one extra fp32 rounding). The acceptance
bound is the decode path's: |gpu - ref| <= 2e-3 + 1e-2 * |ref| for out and
lse. The quantizer is byte work: codes and scales must match bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import fp8_ref
from paper_2601_12784_amd import binding as B
from paper_2601_12784_amd.workloads import (bf16_bits, build_batch, make_batch, page_fill, random_fp8_cache)

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
    _say(f"  {what}: max|err| {err.max(initial=0):.3e}  worst err/bound {worst:.3f}  n={err.size}")
    assert worst <= 1.0, f"{what}: tolerance exceeded ({worst:.3f} of bound)"


def run_fp8(batch, cache, chunk_pages=None, opts=None):
    runner = B.DecodeAttention(batch.num_q_heads, batch.num_kv_heads, batch.head_dim, opts=opts)
    lse = torch.empty((batch.num_seqs, batch.num_q_heads), dtype=torch.float32, device="cuda")
    out = runner(batch.q.cuda(), cache.k8.cuda(), cache.v8.cuda(), torch.from_numpy(batch.block_table).cuda(),
                 batch.seq_lens, batch.scale, lse=lse, chunk_pages=chunk_pages,
                 fp8=(cache.k_scale.cuda(), cache.v_scale.cuda()))
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy(), runner.last_info


def ref_fp8(batch, cache):
    return oracle.decode_attn_fp8(bf16_bits(batch.q), cache.k8.numpy(), cache.v8.numpy(), cache.k_scale.numpy(),
                                  cache.v_scale.numpy(), batch.block_table, batch.seq_lens, batch.scale)


@pytest.mark.parametrize("name", ["tiny", "gqa7b", "longtail", "gqa32b", "straggler"])
def test_fp8_attention_named_workloads(name):
    batch = make_batch(name)
    cache = random_fp8_cache(batch, seed=300 + len(name))
    _say(f"fp8 attention {name}")
    out, lse, info = run_fp8(batch, cache)
    ro, rl = ref_fp8(batch, cache)
    assert_close(out, ro, f"{name} out")
    assert_close(lse, rl, f"{name} lse")


@pytest.mark.parametrize("chunk", [1, 3, 64])
def test_fp8_attention_split_pairs(chunk):
    batch = make_batch("gqa7b")
    cache = random_fp8_cache(batch, seed=41)
    _say(f"fp8 attention gqa7b chunk={chunk}")
    out, lse, info = run_fp8(batch, cache, chunk_pages=chunk)
    assert info.num_combine > 0 or chunk == 64
    ro, rl = ref_fp8(batch, cache)
    assert_close(out, ro, f"chunk {chunk} out")
    assert_close(lse, rl, f"chunk {chunk} lse")


def test_fp8_attention_one_very_long_sequence():
    """A 200k-token sequence beside a 1-token one over the fp8 cache: each
    pair is cut into hundreds of segments (eight workers per CU)."""
    batch = build_batch([200_000, 1], 28, 4, 128, seed=45)
    cache = random_fp8_cache(batch, seed=46)
    _say("fp8 attention, one very long sequence")
    out, lse, info = run_fp8(batch, cache)
    assert info.num_combine == 4 and info.num_partials >= 1000
    ro, rl = ref_fp8(batch, cache)
    assert_close(out, ro, "very long out")
    assert_close(lse, rl, "very long lse")


@pytest.mark.parametrize("wpc,group", [(1, 1), (2, 2), (4, 4), (6, 2), (0, 8)])
def test_fp8_attention_every_launch_group_size(wpc, group):
    """fp8 steps plan eight workers per CU by default (eight waves per
    workgroup); four and one per CU give groups of 4 and 1. Each, with equal
    slices and with a group-parity skew, against the oracle."""
    rng = np.random.default_rng(7)
    lens = np.exp(rng.normal(np.log(1500), 1.0, size=24)).astype(np.int64).clip(16, 12000)
    batch = build_batch(lens, 28, 4, 128, 80)
    cache = random_fp8_cache(batch, seed=47)
    ro, rl = ref_fp8(batch, cache)
    for skew in (0, -60):
        out, lse, info = run_fp8(batch, cache, opts=B.make_opts(num_cus=8, workers_per_cu=wpc, xcd_parity_skew=skew))
        _say(f"fp8 group {group} skew {skew}: {info.num_workers} workers, {info.num_combine} cut pairs")
        assert info.workers_per_group == group
        assert_close(out, ro, f"fp8 group {group} skew {skew} out")
        assert_close(lse, rl, f"fp8 group {group} skew {skew} lse")


@pytest.mark.parametrize("shape", [(8, 2, 64), (16, 1, 128), (7, 7, 64), (5, 1, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_fp8_attention_head_shapes(shape):
    hq, hkv, d = shape
    rng = np.random.Generator(np.random.PCG64(9))
    lens = rng.integers(0, 700, size=13)
    lens[3] = 0
    batch = build_batch(lens, hq, hkv, d, seed=17 + hq)
    cache = random_fp8_cache(batch, seed=5)
    _say(f"fp8 attention shape {shape}")
    out, lse, _ = run_fp8(batch, cache, chunk_pages=5)
    ro, rl = ref_fp8(batch, cache)
    assert_close(out, ro, f"{shape} out")
    assert_close(lse, rl, f"{shape} lse")


def _quantize_gpu(batch, pages, valid):
    n, hkv, d = batch.num_pages, batch.num_kv_heads, batch.head_dim
    desc = B.make_desc(batch.num_seqs, batch.num_q_heads, hkv, d, batch.block_table.shape[1], n, batch.scale)
    k8 = torch.full((n, hkv, 16 * d), 0xAA, dtype=torch.uint8, device="cuda")
    v8 = torch.full((n, hkv, 16 * d), 0xAA, dtype=torch.uint8, device="cuda")
    ks = torch.full((n, hkv), -1.0, dtype=torch.float32, device="cuda")
    vs = torch.full((n, hkv), -1.0, dtype=torch.float32, device="cuda")
    B.sf_kv_quantize_fp8(desc, batch.k_pool.cuda(), batch.v_pool.cuda(), torch.from_numpy(pages).cuda(),
                         torch.from_numpy(valid).cuda(), k8, v8, ks, vs)
    torch.cuda.synchronize()
    return k8.cpu().numpy(), v8.cpu().numpy(), ks.cpu().numpy(), vs.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny", "gqa7b"])
def test_quantizer_bit_exact(name):
    """Every page a sequence holds (partial last pages included; their other
    slots hold NaN in the bf16 pools and must not count); pages not listed
    stay untouched."""
    batch = make_batch(name)
    pages, valid = page_fill(batch)
    _say(f"fp8 quantizer {name}: {pages.size} pages")
    k8, v8, ks, vs = _quantize_gpu(batch, pages, valid)
    n, hkv, d = batch.num_pages, batch.num_kv_heads, batch.head_dim
    rk = np.full(k8.shape, 0xAA, np.uint8)
    rv = np.full(v8.shape, 0xAA, np.uint8)
    rks = np.full((n, hkv), -1.0, np.float32)
    rvs = np.full((n, hkv), -1.0, np.float32)
    fp8_ref.quantize_pages(bf16_bits(batch.k_pool), bf16_bits(batch.v_pool), pages, valid, rk, rv, rks, rvs)
    assert np.array_equal(ks, rks) and np.array_equal(vs, rvs), "scales differ"
    assert np.array_equal(k8, rk), "key codes differ"
    assert np.array_equal(v8, rv), "value codes differ"


def test_quantizer_zero_tile_and_extremes():
    batch = make_batch("tiny")
    k = bf16_bits(batch.k_pool).copy()
    v = bf16_bits(batch.v_pool).copy()
    pages, valid = page_fill(batch)
    p0, p1 = int(pages[0]), int(pages[2])
    k[p0] = 0                                        # an all-zero K tile: scale 1, codes 0
    v[p1, 0, 0, 0] = 0x7F7F                          # the largest finite bf16
    v[p1, 0, 1, 0] = 0x0001                          # the smallest subnormal bf16
    batch.k_pool = torch.from_numpy(k.view(np.int16)).view(torch.bfloat16)
    batch.v_pool = torch.from_numpy(v.view(np.int16)).view(torch.bfloat16)
    _say("fp8 quantizer extremes")
    k8, v8, ks, vs = _quantize_gpu(batch, pages, valid)
    rk = np.full(k8.shape, 0xAA, np.uint8)
    rv = np.full(v8.shape, 0xAA, np.uint8)
    rks = np.full(ks.shape, -1.0, np.float32)
    rvs = np.full(vs.shape, -1.0, np.float32)
    fp8_ref.quantize_pages(k, v, pages, valid, rk, rv, rks, rvs)
    assert ks[p0, 0] == 1.0 and not k8[p0].any()
    assert np.array_equal(ks, rks) and np.array_equal(vs, rvs)
    assert np.array_equal(k8, rk) and np.array_equal(v8, rv)


def test_quantize_then_attend_end_to_end():
    """The library's quantizer, then its fp8 attention, on the full 32B-like
    cache: every page's codes and scales against the oracle's quantizer bit
    for bit, then the GPU attention over the GPU's codes against the oracle's
    attention over the oracle's own codes."""
    batch = make_batch("gqa32b")
    pages, valid = page_fill(batch)
    _say(f"fp8 quantize + attend gqa32b: {pages.size} pages")
    k8, v8, ks, vs = _quantize_gpu(batch, pages, valid)
    rk = np.full(k8.shape, 0xAA, np.uint8)
    rv = np.full(v8.shape, 0xAA, np.uint8)
    rks = np.full(ks.shape, -1.0, np.float32)
    rvs = np.full(vs.shape, -1.0, np.float32)
    fp8_ref.quantize_pages_batched(bf16_bits(batch.k_pool), bf16_bits(batch.v_pool), pages, valid, rk, rv, rks, rvs)
    assert np.array_equal(ks, rks) and np.array_equal(vs, rvs), "scales differ"
    assert np.array_equal(k8, rk), "key codes differ"
    assert np.array_equal(v8, rv), "value codes differ"

    from paper_2601_12784_amd.workloads import Fp8Cache
    gpu_cache = Fp8Cache(torch.from_numpy(k8), torch.from_numpy(v8), torch.from_numpy(ks), torch.from_numpy(vs))
    ref_cache = Fp8Cache(torch.from_numpy(rk), torch.from_numpy(rv), torch.from_numpy(rks), torch.from_numpy(rvs))
    out, lse, _ = run_fp8(batch, gpu_cache)
    ro, rl = ref_fp8(batch, ref_cache)
    assert_close(out, ro, "quantized gqa32b out")
    assert_close(lse, rl, "quantized gqa32b lse")
