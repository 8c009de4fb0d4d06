"""sf_decode_attn_scratch, the decode step that allocates nothing, against
sf_decode_attn + sf_decode_attn_combine on a caller workspace (the entry
points it stands in for) and against the fp64 oracle, through the C ABI.

Two calls in a row, the second with a smaller batch, so the second runs on
the array the first left behind. The scratch variant launches the same
kernels over the same plan, so its results must equal the workspace path's
bit for bit; both must meet |err| <= 2e-3 + 1e-2 |ref| against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2601_12784_amd import binding as B
from paper_2601_12784_amd.workloads import bf16_bits, build_batch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    yield
    torch.cuda.synchronize()


def _say(msg):
    print(msg, flush=True)


def _step_both_ways(b, opts):
    desc = B.make_desc(b.num_seqs, b.num_q_heads, b.num_kv_heads, b.head_dim, b.block_table.shape[1],
                       b.num_pages, b.scale)
    info, work = B.sf_decode_attn_plan(desc, b.seq_lens, opts)
    assert info.workspace_bytes <= B.SCRATCH_BYTES
    q, k, v = b.q.cuda(), b.k_pool.cuda(), b.v_pool.cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    work_dev = torch.from_numpy(np.ascontiguousarray(work[: info.work_bytes // 4])).cuda()
    shape_o, shape_l = (b.num_seqs, b.num_q_heads, b.head_dim), (b.num_seqs, b.num_q_heads)
    out_ws = torch.full(shape_o, float("nan"), device="cuda")
    lse_ws = torch.full(shape_l, float("nan"), device="cuda")
    ws = torch.empty(max(16, info.workspace_bytes), dtype=torch.uint8, device="cuda")
    B.sf_decode_attn(desc, info, None, work_dev, q, k, v, bt, out_ws, lse_ws, ws)
    B.sf_decode_attn_combine(desc, info, work_dev, ws, out_ws, lse_ws)
    out_sc = torch.full(shape_o, float("nan"), device="cuda")
    lse_sc = torch.full(shape_l, float("nan"), device="cuda")
    B.sf_decode_attn_scratch(desc, info, work_dev, q, k, v, bt, out_sc, lse_sc)
    torch.cuda.synchronize()
    return info, (out_ws.cpu().numpy(), lse_ws.cpu().numpy()), (out_sc.cpu().numpy(), lse_sc.cpu().numpy())


def _check(b, info, ws, sc, what):
    ro, rl = oracle.decode_attn(bf16_bits(b.q), bf16_bits(b.k_pool), bf16_bits(b.v_pool), b.block_table,
                                b.seq_lens, b.scale)
    assert np.array_equal(sc[0], ws[0]) and np.array_equal(sc[1], ws[1]), f"{what}: scratch != workspace path"
    # an empty sequence has lse = -inf on both sides; compare the rest
    empty = np.isneginf(rl)
    assert np.array_equal(np.isneginf(sc[1]), empty) and np.all(sc[0][b.seq_lens == 0] == 0)
    for got, ref, name in ((sc[0], ro, "out"), (sc[1][~empty], rl[~empty], "lse")):
        err = np.abs(np.asarray(got, np.float64) - ref)
        worst = float((err / (2e-3 + 1e-2 * np.abs(ref))).max())
        _say(f"  {what} {name}: max|err| {err.max():.3e}  worst err/bound {worst:.4f}")
        assert worst <= 1.0


def test_scratch_step_matches_the_workspace_step_twice_then_smaller():
    opts = B.make_opts(num_cus=torch.cuda.get_device_properties(0).multi_processor_count)
    rng = np.random.default_rng(5)
    lens1 = np.concatenate([rng.integers(1, 4096, size=60), [16384, 9000, 0, 1]])
    b1 = build_batch(lens1, 28, 4, 128, seed=501)
    _say(f"scratch call 1: {b1.num_seqs} sequences, {int(b1.seq_lens.sum())} tokens")
    info1, ws1, sc1 = _step_both_ways(b1, opts)
    assert info1.num_combine > 0 and info1.workspace_bytes > 0
    _check(b1, info1, ws1, sc1, "call 1")

    lens2 = rng.integers(1, 600, size=9)
    b2 = build_batch(lens2, 8, 2, 64, seed=502)
    _say(f"scratch call 2 (smaller): {b2.num_seqs} sequences, {int(b2.seq_lens.sum())} tokens")
    info2, ws2, sc2 = _step_both_ways(b2, B.make_opts(num_cus=4))
    assert info2.num_combine > 0 and 0 < info2.workspace_bytes < info1.workspace_bytes
    _check(b2, info2, ws2, sc2, "call 2")


def test_scratch_step_rejects_a_plan_beyond_its_array():
    """A plan that needs more partial space than the array holds is refused
    before anything is launched."""
    b = build_batch([4096] * 64, 28, 4, 128, seed=503)
    desc = B.make_desc(b.num_seqs, 28, 4, 128, b.block_table.shape[1], b.num_pages, b.scale)
    info, work = B.sf_decode_attn_plan(desc, b.seq_lens, B.make_opts(num_cus=256, chunk_pages=1))
    assert info.workspace_bytes > B.SCRATCH_BYTES
    dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty((b.num_seqs, 28, 128), device="cuda")
    with pytest.raises(B.SfError) as e:
        B.sf_decode_attn_scratch(desc, info, torch.zeros(info.work_bytes // 4, dtype=torch.int32, device="cuda"),
                                 b.q.cuda(), b.k_pool.cuda(), b.v_pool.cuda(),
                                 torch.from_numpy(b.block_table).cuda(), out)
    assert e.value.status == 3   # SF_ERR_CAPACITY
    del dev


def test_scratch_step_over_the_sweep_cases():
    """The seeded sweep's drawn decode cases (head layouts, head dims, length
    mixes, scales of either sign, planner options), one call after another on
    the one array, large and small in turn: each equal to the workspace path
    bit for bit and within the bound of the oracle. Cases whose partials do
    not fit the array are left out (the refusal has its own test)."""
    import dataclasses
    from test_gpu_sweep import SEEDS, sweep_case
    from paper_2601_12784_amd.workloads import PAGE
    ran = 0
    for seed in SEEDS:
        c = sweep_case(seed)
        b = build_batch(c["lens"], c["hq"], c["hkv"], c["d"], 5000 + seed,
                        pool_pages=int(((c["lens"] + PAGE - 1) // PAGE).sum()) + 5)
        b = dataclasses.replace(b, scale=c["scale"])
        opts = B.make_opts(**c["opts"])
        desc = B.make_desc(b.num_seqs, b.num_q_heads, b.num_kv_heads, b.head_dim, b.block_table.shape[1],
                           b.num_pages, b.scale)
        info, _ = B.sf_decode_attn_plan(desc, b.seq_lens, opts)
        if info.workspace_bytes > B.SCRATCH_BYTES:
            continue
        _say(f"scratch sweep {seed}: hq={c['hq']} hkv={c['hkv']} d={c['d']} B={b.num_seqs} opts={c['opts']}")
        info, ws, sc = _step_both_ways(b, opts)
        _check(b, info, ws, sc, f"sweep {seed}")
        ran += 1
    assert ran >= len(SEEDS) // 2
