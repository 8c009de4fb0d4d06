"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Each check is chosen so that a plausible slip in the oracle (a dropped scale,
a wrong GQA head mapping, a transposed V tile, a page/slot index mix-up, a
missing max subtraction, a wrong log-normaliser) fails at least one of them.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import dense_ref, exact_ref, merge_ref
from paper_2601_12784_amd.workloads import build_batch, bf16_bits, NAN_BF16, PAGE
from tests.conftest import f32_to_bf16_exact

pytestmark = pytest.mark.usefixtures("oracle_lib")


def _bits(batch):
    return bf16_bits(batch.q), bf16_bits(batch.k_pool), bf16_bits(batch.v_pool)


def _run(batch, scale=None):
    q, k, v = _bits(batch)
    return oracle.decode_attn(q, k, v, batch.block_table, batch.seq_lens,
                              batch.scale if scale is None else scale)


def _widen(bits):
    return dense_ref.widen(bits)


def _k_row(batch, s, kvh, t):
    """uint16 key row of token t (the K tile stores 8-dim pieces per slot)."""
    pg = batch.block_table[s, t // PAGE]
    return bf16_bits(batch.k_pool)[pg, kvh, :, t % PAGE, :].reshape(-1)


def _set_k_row(batch, s, kvh, t, row_bits):
    pg = batch.block_table[s, t // PAGE]
    bf16_bits(batch.k_pool)[pg, kvh, :, t % PAGE, :] = np.asarray(row_bits).reshape(-1, 8)


def _set_v_row(batch, s, kvh, t, row_bits):
    pg = batch.block_table[s, t // PAGE]
    bf16_bits(batch.v_pool)[pg, kvh, :, t % PAGE] = row_bits


def _grid_values(rng, shape, lim=64, den=16):
    """Values k/den, |k| <= lim: exact in bf16 and under small sums."""
    return rng.integers(-lim, lim + 1, size=shape).astype(np.float32) / np.float32(den)


# ---------------------------------------------------------------------------
# brute force: decimal (60 digits) and dense numpy on tiny inputs
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", [1, 2, 3])
def test_matches_decimal_brute_force(seed):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, 21, size=3)
    lens[0] = 1
    b = build_batch(lens, 4, 2, 16, seed, pool_pages=int(((lens + 15) // 16).sum()) + 3)
    out, lse = _run(b)
    ex_out, ex_lse, _ = exact_ref.decode_attn(*_bits(b), b.block_table, b.seq_lens, b.scale)
    assert np.all(np.abs(out - ex_out) <= 1e-14 * np.maximum(1.0, np.abs(ex_out)))
    assert np.all(np.abs(lse - ex_lse) <= 1e-14 * np.maximum(1.0, np.abs(ex_lse)))


@pytest.mark.parametrize("seed", [4, 5])
def test_matches_dense_numpy(seed):
    lens = np.array([1, 15, 16, 17, 40, 0, 100])
    b = build_batch(lens, 6, 2, 32, seed, pool_pages=40)
    out, lse = _run(b)
    d_out, d_lse = dense_ref.decode_attn(*_bits(b), b.block_table, b.seq_lens, b.scale)
    assert np.allclose(out, d_out, rtol=1e-12, atol=1e-13)
    fin = np.isfinite(d_lse)
    assert np.array_equal(fin, np.isfinite(lse))
    assert np.allclose(lse[fin], d_lse[fin], rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------------------
# closed forms and special cases
# ---------------------------------------------------------------------------
def test_length_one_returns_v_row_exactly():
    b = build_batch([1, 1, 1], 8, 2, 64, 11)
    out, lse = _run(b)
    g = 4
    for s in range(3):
        pg = b.block_table[s, 0]
        for h in range(8):
            v = _widen(bf16_bits(b.v_pool)[pg, h // g, :, 0])
            assert np.array_equal(out[s, h], v)
            # lse of one token is its own score
            qv = _widen(bf16_bits(b.q)[s, h])
            kv = _widen(_k_row(b, s, h // g, 0))
            assert lse[s, h] == pytest.approx(b.scale * float(qv @ kv), rel=1e-14, abs=1e-15)


def test_gqa_head_mapping_contiguous_groups():
    hq, hkv = 12, 3
    b = build_batch([1, 5], hq, hkv, 64, 12)
    for s in range(2):
        for kvh in range(hkv):
            for t in range(int(b.seq_lens[s])):
                _set_v_row(b, s, kvh, t, f32_to_bf16_exact(np.full(64, kvh + 1.0)))
    out, _ = _run(b)
    g = hq // hkv
    for h in range(hq):
        # exact for the length-1 row; Sum(c*w)/Sum(w) rounds in fp64 otherwise
        assert np.all(out[0, h, :] == h // g + 1.0)
        assert np.allclose(out[1, h, :], h // g + 1.0, rtol=1e-15, atol=0)


@pytest.mark.parametrize("length", [1, 16, 17, 300])
def test_identical_keys_give_exact_mean(length):
    rng = np.random.default_rng(length)
    d = 64
    b = build_batch([length], 4, 1, d, 13)
    key = f32_to_bf16_exact(_grid_values(rng, d))
    vals = _grid_values(rng, (length, d))
    for t in range(length):
        _set_k_row(b, 0, 0, t, key)
        _set_v_row(b, 0, 0, t, f32_to_bf16_exact(vals[t]))
    out, lse = _run(b)
    exact = [float(sum(Fraction(float(x)) for x in vals[:, j]) / length) for j in range(d)]
    for h in range(4):
        assert np.array_equal(out[0, h], np.array(exact))
        z = b.scale * float(_widen(bf16_bits(b.q)[0, h]) @ _widen(key))
        assert lse[0, h] == pytest.approx(z + math.log(length), rel=1e-13)


def test_zero_scale_gives_mean_of_values():
    rng = np.random.default_rng(3)
    length, d = 45, 32
    b = build_batch([length], 2, 1, d, 14)
    vals = _grid_values(rng, (length, d))
    for t in range(length):
        _set_v_row(b, 0, 0, t, f32_to_bf16_exact(vals[t]))
    out, lse = _run(b, scale=0.0)
    exact = np.array([float(sum(Fraction(float(x)) for x in vals[:, j]) / length) for j in range(d)])
    assert np.array_equal(out[0, 0], exact) and np.array_equal(out[0, 1], exact)
    assert lse[0, 0] == pytest.approx(math.log(length), rel=1e-15)


def test_dominant_key_returns_its_value_row():
    """A score gap of thousands underflows every other weight to exactly 0,
    and without the max subtraction exp(4096) would overflow."""
    d, length, hot = 32, 40, 23
    b = build_batch([length], 1, 1, d, 15)
    q = np.zeros(d, np.float32)
    q[0] = 64.0
    bf16_bits(b.q)[0, 0] = f32_to_bf16_exact(q)
    for t in range(length):
        row = _widen(_k_row(b, 0, 0, t)).astype(np.float32)
        row[0] = 64.0 if t == hot else 0.0
        _set_k_row(b, 0, 0, t, f32_to_bf16_exact(row))
    out, lse = _run(b, scale=1.0)
    pg = b.block_table[0, hot // PAGE]
    assert np.array_equal(out[0, 0], _widen(bf16_bits(b.v_pool)[pg, 0, :, hot % PAGE]))
    assert lse[0, 0] == 4096.0


def test_two_token_logistic_closed_form():
    """softmax over two scores is the logistic function of their gap."""
    d = 16
    b = build_batch([2], 1, 1, d, 16)
    q = np.zeros(d, np.float32)
    q[0] = 1.0
    bf16_bits(b.q)[0, 0] = f32_to_bf16_exact(q)
    k0 = np.zeros(d, np.float32)
    k1 = np.zeros(d, np.float32)
    k1[0] = 1.5
    _set_k_row(b, 0, 0, 0, f32_to_bf16_exact(k0))
    _set_k_row(b, 0, 0, 1, f32_to_bf16_exact(k1))
    v0 = np.linspace(-1, 1, d).astype(np.float32)
    v0 = (v0.view(np.uint32) & 0xFFFF0000).view(np.float32)
    v1 = np.full(d, 2.0, np.float32)
    _set_v_row(b, 0, 0, 0, f32_to_bf16_exact(v0))
    _set_v_row(b, 0, 0, 1, f32_to_bf16_exact(v1))
    scale = 0.75
    out, lse = _run(b, scale=scale)
    gap = scale * 1.5
    sig = 1.0 / (1.0 + math.exp(-gap))
    expect = v0.astype(np.float64) + sig * (v1.astype(np.float64) - v0.astype(np.float64))
    assert np.allclose(out[0, 0], expect, rtol=1e-15, atol=1e-15)
    assert lse[0, 0] == pytest.approx(math.log(1.0 + math.exp(gap)), rel=1e-15)


def test_shift_of_values_shifts_output():
    rng = np.random.default_rng(7)
    length, d = 70, 64
    b = build_batch([length], 4, 2, d, 17)
    vals = _grid_values(rng, (2, length, d))
    for kvh in range(2):
        for t in range(length):
            _set_v_row(b, 0, kvh, t, f32_to_bf16_exact(vals[kvh, t]))
    out0, _ = _run(b)
    for kvh in range(2):
        for t in range(length):
            _set_v_row(b, 0, kvh, t, f32_to_bf16_exact(vals[kvh, t] + 2.0))
    out1, _ = _run(b)
    assert np.allclose(out1, out0 + 2.0, rtol=0, atol=1e-13)


def test_linear_in_values():
    rng = np.random.default_rng(8)
    length, d = 33, 32
    b = build_batch([length], 2, 1, d, 18)
    v1 = _grid_values(rng, (length, d))
    v2 = _grid_values(rng, (length, d))
    res = []
    for vals in (v1, v2, v1 + v2):
        for t in range(length):
            _set_v_row(b, 0, 0, t, f32_to_bf16_exact(vals[t]))
        res.append(_run(b)[0])
    assert np.allclose(res[2], res[0] + res[1], rtol=0, atol=1e-13)


def test_empty_sequence_is_zero_and_neg_inf():
    b = build_batch([0, 5, 0], 4, 2, 32, 19)
    out, lse = _run(b)
    assert np.all(out[[0, 2]] == 0.0) and np.all(np.isneginf(lse[[0, 2]]))
    assert np.all(np.isfinite(out[1])) and np.all(np.isfinite(lse[1]))


# ---------------------------------------------------------------------------
# invariances
# ---------------------------------------------------------------------------
def test_physical_page_permutation_is_bitwise_invariant():
    lens = [17, 64, 130, 300]
    b = build_batch(lens, 4, 1, 64, 20, pool_pages=64)
    out0, lse0 = _run(b)
    rng = np.random.default_rng(0)
    perm = rng.permutation(64)
    kb, vb = bf16_bits(b.k_pool).copy(), bf16_bits(b.v_pool).copy()
    bf16_bits(b.k_pool)[perm] = kb
    bf16_bits(b.v_pool)[perm] = vb
    bt = b.block_table.copy()
    b.block_table[bt >= 0] = perm[bt[bt >= 0]]
    out1, lse1 = _run(b)
    assert np.array_equal(out0, out1) and np.array_equal(lse0, lse1)


def test_logical_page_order_changes_only_rounding():
    """Attention is a set function of the (key, value) pairs."""
    b = build_batch([128, 64], 4, 2, 64, 21)
    out0, lse0 = _run(b)
    b.block_table[0, :8] = b.block_table[0, :8][::-1].copy()
    b.block_table[1, :4] = b.block_table[1, [2, 0, 3, 1]].copy()
    out1, lse1 = _run(b)
    assert np.allclose(out0, out1, rtol=1e-13, atol=1e-14)
    assert np.allclose(lse0, lse1, rtol=1e-14, atol=0)


def test_lse_merge_of_page_aligned_halves_equals_whole():
    """Softmax over A u B rebuilt from each half's (out, lse): pins both the
    oracle's log-normaliser and the fp64 merge used for split-K."""
    b = build_batch([96, 160], 6, 3, 64, 22)
    full_o, full_l = _run(b)
    for s, cut_pages in ((0, 2), (1, 7)):
        parts_o, parts_l = [], []
        for lo, hi in ((0, cut_pages), (cut_pages, b.block_table.shape[1])):
            n_tok = min(int(b.seq_lens[s]), hi * PAGE) - lo * PAGE
            sub_bt = np.full((1, b.block_table.shape[1]), -1, np.int32)
            npg = (n_tok + PAGE - 1) // PAGE
            sub_bt[0, :npg] = b.block_table[s, lo:lo + npg]
            q, k, v = _bits(b)
            o, l = oracle.decode_attn(q[s:s + 1], k, v, sub_bt, np.array([n_tok], np.int32), b.scale)
            parts_o.append(o[0])
            parts_l.append(l[0])
        mo, ml = merge_ref.merge(parts_o, parts_l)
        assert np.allclose(mo, full_o[s], rtol=1e-13, atol=1e-14)
        assert np.allclose(ml, full_l[s], rtol=1e-14, atol=0)


def test_merge_ignores_empty_parts():
    o = np.array([[1.0, 2.0], [5.0, 7.0]])
    l = np.array([0.3, -np.inf])
    mo, ml = merge_ref.merge(o[:, None, :], l[:, None])
    assert np.array_equal(mo[0], o[0]) and ml[0] == 0.3


def test_poisoned_slots_and_pages_are_never_read():
    lens = [17, 64, 130, 300, 5]
    clean = build_batch(lens, 4, 1, 64, 23, pool_pages=70, poison=False)
    dirty = build_batch(lens, 4, 1, 64, 23, pool_pages=70, poison=True)
    assert np.any(bf16_bits(dirty.k_pool) == NAN_BF16)
    o0, l0 = _run(clean)
    o1, l1 = _run(dirty)
    assert np.all(np.isfinite(o1)) and np.array_equal(o0, o1) and np.array_equal(l0, l1)


def test_rejects_out_of_range_pages():
    b = build_batch([20], 2, 1, 32, 24)
    b.block_table[0, 1] = b.num_pages
    with pytest.raises(ValueError):
        _run(b)


def test_gather_matches_layout_definition():
    b = build_batch([37, 3], 4, 2, 32, 25, pool_pages=8)
    for s in range(2):
        for kvh in range(2):
            L = int(b.seq_lens[s])
            kd, vd = oracle.gather(bf16_bits(b.k_pool), bf16_bits(b.v_pool), b.block_table, s, kvh, L)
            for t in range(L):
                pg = b.block_table[s, t // PAGE]
                # key dim d of slot t sits at [d // 8, t, d % 8] of its tile
                kt = bf16_bits(b.k_pool)[pg, kvh]
                assert all(kd[t, d] == kt[d // 8, t % PAGE, d % 8] for d in range(32))
                assert np.array_equal(vd[t], bf16_bits(b.v_pool)[pg, kvh, :, t % PAGE])


# ---------------------------------------------------------------------------
# stored high-precision cases (tests/golden/exact_cases.json)
# ---------------------------------------------------------------------------
def test_golden_exact_cases():
    import json
    import os
    from decimal import Decimal
    path = os.path.join(os.path.dirname(__file__), "golden", "exact_cases.json")
    doc = json.load(open(path))
    for c in doc["cases"]:
        q = np.array(c["q"], dtype=np.uint16)
        k = np.array(c["k_pool"], dtype=np.uint16)
        v = np.array(c["v_pool"], dtype=np.uint16)
        out, lse = oracle.decode_attn(q, k, v, np.array(c["block_table"], np.int32),
                                      np.array(c["lens"], np.int32), c["scale"])
        for key, vals in c["out"].items():
            s, h = map(int, key.split(","))
            ref = np.array([float(Decimal(x)) for x in vals])
            assert np.all(np.abs(out[s, h] - ref) <= 4e-16 * np.maximum(1.0, np.abs(ref))), c["name"]
            ref_l = float(Decimal(c["lse"][key]))
            assert abs(lse[s, h] - ref_l) <= 4e-16 * max(1.0, abs(ref_l)), c["name"]
