"""GPU parity of extend (re-prefill) attention and the new-token store against
the fp64 oracle, through the C ABI.

Acceptance, elementwise for out and for lse (natural log), the same bound as
every decode-attention test:
    |gpu - ref| <= 2e-3 + 1e-2 * |ref|
The kernel rounds the softmax weights to fp16 (relative error <= 2^-11) for
the P.V product, and its sums are fp32; the worst error seen stays well
inside the bound (the largest err/bound is printed for each case). The
stores are byte work and must match bit for bit.
"""
import copy

import numpy as np
import pytest
import torch

from oracle import extend_ref
from paper_2601_12784_amd import binding as B
from paper_2601_12784_amd.workloads import bf16_bits, build_extend, make_reprefill

pytestmark = pytest.mark.gpu

NAN_BF16 = 0x7FC0


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    yield
    torch.cuda.synchronize()


def _say(msg):
    print(msg, flush=True)


def run_gpu(eb, scale=None, store=False, k_pool=None, v_pool=None, lse=True):
    b = eb.batch
    runner = B.ExtendAttention(b.num_q_heads, b.num_kv_heads, b.head_dim)
    kp = (b.k_pool if k_pool is None else k_pool).cuda()
    vp = (b.v_pool if v_pool is None else v_pool).cuda()
    bt = torch.from_numpy(b.block_table).cuda()
    t = eb.num_rows
    lse_t = torch.empty((t, b.num_q_heads), dtype=torch.float32, device="cuda") if lse else None
    out = runner(eb.q.cuda(), kp, vp, bt, b.seq_lens, eb.q_lens, b.scale if scale is None else scale, lse=lse_t,
                 k_new=eb.k_new.cuda() if store else None, v_new=eb.v_new.cuda() if store else None)
    torch.cuda.synchronize()
    return out.cpu().numpy(), (lse_t.cpu().numpy() if lse else None), kp.cpu(), vp.cpu(), runner.last_info


def run_oracle(eb, rows=None, scale=None):
    b = eb.batch
    q, k, v = bf16_bits(eb.q), bf16_bits(b.k_pool), bf16_bits(b.v_pool)
    s = b.scale if scale is None else scale
    return extend_ref.extend_attn(q, k, v, b.block_table, b.seq_lens, eb.q_lens, s, rows=rows)


def assert_close(out, lse, ref, what):
    ro, rl = ref
    out = np.asarray(out, np.float64)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(ro)), f"{what}: non-finite output"
    err = np.abs(out - ro)
    worst = float((err / (2e-3 + 1e-2 * np.abs(ro))).max(initial=0.0))
    _say(f"  {what} out: max|err| {err.max(initial=0):.3e}  worst err/bound {worst:.3f}  n={err.size}")
    assert worst <= 1.0, f"{what}: out tolerance exceeded ({worst:.3f} of bound)"
    if lse is not None:
        le = np.abs(np.asarray(lse, np.float64) - rl)
        lw = float((le / (2e-3 + 1e-2 * np.abs(rl))).max(initial=0.0))
        _say(f"  {what} lse: max|err| {le.max(initial=0):.3e}  worst err/bound {lw:.3f}")
        assert lw <= 1.0, f"{what}: lse tolerance exceeded ({lw:.3f} of bound)"


SHAPES = [(28, 4, 128), (8, 2, 64), (16, 1, 128), (7, 7, 64), (5, 1, 64)]
CASES = {
    # name: (lens, q_lens)
    "reprefill": ([37, 300, 64, 1], [37, 300, 64, 1]),
    "chunked": ([900, 233, 517, 48], [200, 1, 117, 16]),
    "mixed": ([40, 16, 1, 0, 700], [0, 9, 1, 0, 333]),
    # with one query head per KV head an item holds 384 tokens: several full items and ragged tails
    "wide": ([1000, 777], [900, 777]),
}


@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_extend_small(case, shape):
    hq, hkv, d = shape
    lens, qls = CASES[case]
    _say(f"extend {case} hq={hq} hkv={hkv} d={d}")
    eb = build_extend(lens, qls, hq, hkv, d, seed=71 + len(case) + hq)
    out, lse, *_ = run_gpu(eb)
    assert_close(out, lse, run_oracle(eb), f"{case} {shape}")


@pytest.mark.parametrize("shape", [(28, 4, 128), (16, 1, 128)], ids=lambda s: "x".join(map(str, s)))
def test_extend_after_a_long_prefix(shape):
    """New tokens after a 100k-token cache: the items walk about 6250 pages
    of keys each, the longest key walks the kernel takes."""
    hq, hkv, d = shape
    eb = build_extend([100_000, 5_000], [40, 700], hq, hkv, d, seed=91 + hq)
    _say(f"extend after a long prefix hq={hq} hkv={hkv}")
    out, lse, *_ = run_gpu(eb)
    assert_close(out, lse, run_oracle(eb), f"long prefix {shape}")


def test_extend_with_no_new_tokens_launches_nothing():
    eb = build_extend([40, 16], [0, 0], 8, 2, 64, seed=3)
    _say("extend empty")
    out, lse, kp, vp, info = run_gpu(eb, store=True)
    assert info.num_items == 0 and out.shape == (0, 8, 64)
    assert np.array_equal(bf16_bits(kp), bf16_bits(eb.batch.k_pool))


def test_extend_store_then_attend():
    """New-token slots start as NaN; the store launch must write exactly the
    bytes the oracle's store writes, and the attention must read them."""
    eb = build_extend([700, 40, 333, 17], [300, 40, 1, 17], 28, 4, 128, seed=5)
    b = eb.batch
    pages, slots = eb.slots()
    k0 = bf16_bits(b.k_pool).copy()
    v0 = bf16_bits(b.v_pool).copy()
    kh, vh = k0.copy(), v0.copy()
    kh[pages, :, :, slots, :] = NAN_BF16
    vh[pages, :, :, slots] = NAN_BF16
    k_in = torch.from_numpy(kh.view(np.int16)).view(torch.bfloat16)
    v_in = torch.from_numpy(vh.view(np.int16)).view(torch.bfloat16)
    _say("extend store+attend 28x4x128")
    out, lse, kp, vp, _ = run_gpu(eb, store=True, k_pool=k_in, v_pool=v_in)
    # the oracle's store applied to the NaN-filled copy gives back the original pools
    kref, vref = kh.copy(), vh.copy()
    extend_ref.kv_store(kref, vref, b.block_table, b.seq_lens, eb.q_lens, bf16_bits(eb.k_new), bf16_bits(eb.v_new))
    assert np.array_equal(kref, k0) and np.array_equal(vref, v0)
    assert np.array_equal(bf16_bits(kp), kref), "stored keys differ"
    assert np.array_equal(bf16_bits(vp), vref), "stored values differ"
    assert_close(out, lse, run_oracle(eb), "store+attend")


@pytest.mark.parametrize("scale", [-0.0883883, 0.0, 0.5])
def test_extend_scale_sign_and_zero(scale):
    eb = build_extend([300, 70], [300, 22], 8, 2, 64, seed=9)
    _say(f"extend scale={scale}")
    out, lse, *_ = run_gpu(eb, scale=scale)
    assert_close(out, lse, run_oracle(eb, scale=scale), f"scale {scale}")


def test_extend_peaked_scores():
    eb = build_extend([1200, 333], [1200, 100], 28, 4, 128, seed=13, k_mult=3.0)
    _say("extend peaked (K x 3)")
    out, lse, *_ = run_gpu(eb)
    assert_close(out, lse, run_oracle(eb), "peaked")



def test_extend_rising_scores_move_the_reference():
    """Scores that climb along the keys (about 90 log2 units over 1200 keys)
    make each row move its softmax reference several times during its walk, and
    make the last keys of a row its heaviest."""
    eb = build_extend([1200, 333], [1200, 333], 28, 4, 128, seed=17)
    pages, slots = eb.slots()
    pos = np.concatenate([np.arange(1200), np.arange(333)])
    ramp = torch.from_numpy(pos * 0.15).float().to(torch.bfloat16).view(torch.int16).numpy()
    kp = eb.batch.k_pool.view(torch.int16).numpy()   # [page, KV head, D/8, slot, 8], shares memory
    for h in range(kp.shape[1]):
        kp[pages, h, 0, slots, 0] = ramp
    eb.q[:, :, 0] = 4.0
    _say("extend rising scores")
    out, lse, *_ = run_gpu(eb)
    assert_close(out, lse, run_oracle(eb), "rising")

def test_extend_page_order_does_not_matter():
    """Physical page ids are only addresses: the same pages moved to other
    slots of a larger pool (block table rewritten to match) give the same bits."""
    a = build_extend([500, 90], [500, 31], 28, 4, 128, seed=17)
    ba = a.batch
    n = ba.k_pool.shape[0]
    rng = np.random.default_rng(2)
    dest = rng.permutation(n + 37)[:n]                 # page p moves to dest[p]
    kb, vb = bf16_bits(ba.k_pool), bf16_bits(ba.v_pool)
    k2 = np.full((n + 37,) + kb.shape[1:], NAN_BF16, np.uint16)
    v2 = np.full((n + 37,) + vb.shape[1:], NAN_BF16, np.uint16)
    k2[dest], v2[dest] = kb, vb
    bt2 = np.where(ba.block_table >= 0, dest[np.maximum(ba.block_table, 0)], -1).astype(np.int32)
    b = copy.copy(a)
    b.batch = copy.copy(ba)
    b.batch.k_pool = torch.from_numpy(k2.view(np.int16)).view(torch.bfloat16)
    b.batch.v_pool = torch.from_numpy(v2.view(np.int16)).view(torch.bfloat16)
    b.batch.block_table = bt2
    _say("extend page permutation")
    oa, la, *_ = run_gpu(a)
    ob, lb, *_ = run_gpu(b)
    assert np.array_equal(oa, ob) and np.array_equal(la, lb)


def test_extend_value_range_of_the_fp16_product():
    """Values are widened to fp16 for the P.V product: bf16 values up to
    65280 in magnitude and down to 2^-17 convert exactly, smaller ones round
    by at most 2^-25. Values of 49152 and about -1.1 * 2^-20 in the cache, checked
    against the oracle on the same bits."""
    eb = build_extend([300, 70], [300, 22], 8, 2, 64, seed=19)
    vp = eb.batch.v_pool.view(torch.int16).numpy()   # shares memory
    pages, slots = eb.slots()
    big = np.int16(torch.tensor([49152.0]).to(torch.bfloat16).view(torch.int16).item())
    tiny = np.int16(torch.tensor([-1.1 * 2.0 ** -20]).to(torch.bfloat16).view(torch.int16).item())
    vp[pages[::3], :, :, slots[::3]] = big
    vp[pages[1::3], :, 5, slots[1::3]] = tiny
    _say("extend value range")
    out, lse, *_ = run_gpu(eb)
    assert_close(out, lse, run_oracle(eb), "value range")


@pytest.fixture(scope="module")
def reprefill_run():
    """The 32-sequence full re-prefill at its real size, computed twice on the
    GPU (the two runs must agree bit for bit)."""
    eb = make_reprefill()
    _say(f"reprefill full size: {eb.num_rows} rows")
    out, lse, *_, info = run_gpu(eb)
    out2, lse2, *_ = run_gpu(eb)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2), "not deterministic"
    return eb, out, lse


def test_reprefill_full_size_longest_and_shortest_sequences(reprefill_run):
    """Every row of the four longest and the four shortest sequences against
    the whole-sequence fp64 oracle."""
    eb, out, lse = reprefill_run
    b = eb.batch
    order = np.argsort(b.seq_lens, kind="stable")
    seqs = [int(s) for s in np.concatenate([order[-4:][::-1], order[:4]])]
    _say(f"reprefill: full rows of sequences {seqs} (lengths {[int(b.seq_lens[s]) for s in seqs]})")
    rows, ro, rl = extend_ref.extend_attn_dense(bf16_bits(eb.q), bf16_bits(b.k_pool), bf16_bits(b.v_pool),
                                                b.block_table, b.seq_lens, eb.q_lens, b.scale, seqs)
    assert_close(out[rows], lse[rows], (ro, rl), f"reprefill full rows n={rows.size}")


def test_reprefill_full_size_random_rows(reprefill_run):
    """2048 random rows of the whole batch, plus each sequence's first and
    last row, against the per-row oracle."""
    eb, out, lse = reprefill_run
    cu = np.concatenate([[0], np.cumsum(eb.q_lens.astype(np.int64))])
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([cu[:-1], cu[1:] - 1, rng.choice(eb.num_rows, size=2048, replace=False)]))
    assert rows.size >= 2048
    ref = run_oracle(eb, rows=rows)
    assert_close(out[rows], lse[rows], ref, f"reprefill random rows={rows.size}")
