"""Pins of the extend (re-prefill) oracle, oracle/extend_ref.py, on the CPU.

Checked against what the definition fixes, through code that shares nothing
with the oracle's decode-per-row evaluation: torch's own scaled-dot-product
attention in float64 with an explicit causal mask over an independently
gathered dense cache; the closed form of a sequence's first token (its output
is its own value row); the dense numpy decode path for a sequence's last
token; and, for the store, the dense gather reading back what was written."""
import math

import numpy as np
import pytest
import torch

from oracle import dense_ref, extend_ref

PAGE = 16


def _case(seed, lens, q_lens, hq=4, hkv=2, d=64, pool_extra=3):
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, np.int64)
    pages = -(-lens // PAGE)
    n = int(pages.sum()) + pool_extra
    perm = rng.permutation(n)
    stride = max(1, int(pages.max()))
    bt = np.full((lens.size, stride), -1, np.int32)
    off = 0
    for s in range(lens.size):
        bt[s, : pages[s]] = perm[off: off + pages[s]]
        off += pages[s]
    # finite bf16 bit patterns of moderate size: sign, exponent 120..129, any mantissa
    def draw(*shape):
        sign = rng.integers(0, 2, size=shape) << 15
        expo = rng.integers(120, 130, size=shape) << 7
        mant = rng.integers(0, 128, size=shape)
        return (sign | expo | mant).astype(np.uint16)
    t = int(np.sum(q_lens))
    q = draw(t, hq, d)
    k = draw(n, hkv, d // 8, PAGE, 8)
    v = draw(n, hkv, d, PAGE)
    return q, k, v, bt, lens, np.asarray(q_lens, np.int64), 1.0 / math.sqrt(d)


def _sdpa_reference(q, k, v, bt, lens, q_lens, scale):
    """torch SDPA (float64) per sequence with a boolean mask allowing t <= P + j."""
    hq, d = q.shape[1], q.shape[2]
    hkv = k.shape[1]
    g = hq // hkv
    outs, lses = [], []
    cu = 0
    for s in range(lens.size):
        L, e = int(lens[s]), int(q_lens[s])
        if e == 0:
            continue
        p0 = L - e
        kd = np.stack([dense_ref.gather_dense(k, v, bt, s, kvh, L)[0] for kvh in range(hkv)])   # [Hkv, L, D]
        vd = np.stack([dense_ref.gather_dense(k, v, bt, s, kvh, L)[1] for kvh in range(hkv)])
        kt = torch.from_numpy(kd).repeat_interleave(g, dim=0)                                  # [Hq, L, D]
        vt = torch.from_numpy(vd).repeat_interleave(g, dim=0)
        qt = torch.from_numpy(dense_ref.widen(q[cu: cu + e])).permute(1, 0, 2).contiguous()   # [Hq, E, D]
        j = torch.arange(e).unsqueeze(1)
        t = torch.arange(L).unsqueeze(0)
        mask = t <= p0 + j                                                                     # [E, L]
        o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
        z = (qt @ kt.transpose(1, 2)) * scale
        lse = torch.logsumexp(z.masked_fill(~mask, float("-inf")), dim=-1)                   # [Hq, E]
        outs.append(o.permute(1, 0, 2).numpy())
        lses.append(lse.T.numpy())
        cu += e
    return np.concatenate(outs), np.concatenate(lses)


CASES = [
    # (lens, q_lens): full re-prefill, chunked extend, single-token (decode), empty extend
    ([37, 5, 64], [37, 5, 64]),
    ([90, 33, 17, 48], [20, 1, 17, 16]),
    ([40, 16, 1], [0, 9, 1]),
    ([129], [47]),
]


@pytest.mark.parametrize("ci", range(len(CASES)))
@pytest.mark.parametrize("heads", [(4, 2, 64), (7, 1, 128), (3, 3, 64)])
def test_extend_oracle_matches_torch_sdpa_with_causal_mask(oracle_lib, ci, heads):
    hq, hkv, d = heads
    q, k, v, bt, lens, ql, scale = _case(10 + ci, *CASES[ci], hq=hq, hkv=hkv, d=d)
    out, lse = extend_ref.extend_attn(q, k, v, bt, lens, ql, scale)
    want_o, want_l = _sdpa_reference(q, k, v, bt, lens, ql, scale)
    np.testing.assert_allclose(out, want_o, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse, want_l, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("ci", range(len(CASES)))
@pytest.mark.parametrize("heads", [(4, 2, 64), (7, 1, 128), (3, 3, 64)])
def test_dense_extend_oracle_matches_torch_sdpa_and_the_per_row_oracle(oracle_lib, ci, heads):
    """The whole-sequence fp64 path (matrix products, mask, softmax written
    out) against torch's SDPA and against a decode step per row; chunks of
    new tokens smaller than the sequences, so chunk edges are crossed."""
    hq, hkv, d = heads
    q, k, v, bt, lens, ql, scale = _case(20 + ci, *CASES[ci], hq=hq, hkv=hkv, d=d)
    seqs = list(range(lens.size))[::-1]
    rows, out, lse = extend_ref.extend_attn_dense(q, k, v, bt, lens, ql, scale, seqs, nthreads=3, tok_chunk=7)
    cu = extend_ref.cu_lens(ql)
    assert rows.tolist() == [r for s in seqs for r in range(cu[s], cu[s + 1])]
    want_o, want_l = _sdpa_reference(q, k, v, bt, lens, ql, scale)
    np.testing.assert_allclose(out, want_o[rows], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse, want_l[rows], rtol=1e-12, atol=1e-12)
    o2, l2 = extend_ref.extend_attn(q, k, v, bt, lens, ql, scale, rows=rows)
    np.testing.assert_allclose(out, o2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, l2, rtol=1e-13, atol=1e-13)


# the poisoned +inf key makes inf * 0 products in that key's column of the
# score matmul, a column every earlier row masks out
@pytest.mark.filterwarnings("ignore:invalid value encountered in matmul:RuntimeWarning")
def test_dense_extend_oracle_first_row_and_causal_limit(oracle_lib):
    """A full re-prefill's first row returns its own value row exactly, and a
    key past a row's causal limit changes nothing: poisoning the last key of
    a sequence leaves every earlier row's result unchanged."""
    q, k, v, bt, lens, ql, scale = _case(8, [45], [45], hq=2, hkv=1, d=64)
    rows, out, lse = extend_ref.extend_attn_dense(q, k, v, bt, lens, ql, scale, [0], tok_chunk=16)
    kd, vd = dense_ref.gather_dense(k, v, bt, 0, 0, 1)
    assert np.array_equal(out[0, 0], vd[0]) and np.array_equal(out[0, 1], vd[0])
    k2, v2 = k.copy(), v.copy()
    last = 44
    pg, sl = int(bt[0, last // PAGE]), last % PAGE
    k2[pg, 0, :, sl, :] = 0x7F80   # +inf keys
    v2[pg, 0, :, sl] = 0x7FC0      # NaN values
    _, out2, lse2 = extend_ref.extend_attn_dense(q, k2, v2, bt, lens, ql, scale, [0], tok_chunk=16)
    assert np.array_equal(out2[:last], out[:last]) and np.array_equal(lse2[:last], lse[:last])
    assert not np.all(np.isfinite(out2[last]))


def test_first_token_of_a_full_reprefill_is_its_own_value_row(oracle_lib):
    q, k, v, bt, lens, ql, scale = _case(3, [50, 20], [50, 20], hq=6, hkv=2, d=64)
    out, lse = extend_ref.extend_attn(q, k, v, bt, lens, ql, scale)
    cu = extend_ref.cu_lens(ql)
    for s in range(2):
        for h in range(6):
            kvh = h // 3
            kd, vd = dense_ref.gather_dense(k, v, bt, s, kvh, 1)
            r = int(cu[s])
            assert np.array_equal(out[r, h], vd[0])                       # one term: weight exactly 1
            z = scale * float(np.dot(dense_ref.widen(q[r, h]), kd[0]))
            assert lse[r, h] == pytest.approx(z, rel=1e-14, abs=1e-14)  # ln e^z


def test_last_new_token_is_a_decode_step_over_the_whole_sequence(oracle_lib):
    q, k, v, bt, lens, ql, scale = _case(4, [70, 33, 16], [12, 33, 5], hq=4, hkv=1, d=64)
    out, lse = extend_ref.extend_attn(q, k, v, bt, lens, ql, scale)
    cu = extend_ref.cu_lens(ql)
    last = cu[1:] - 1
    d_out, d_lse = dense_ref.decode_attn(q[last], k, v, bt, lens, scale)
    np.testing.assert_allclose(out[last], d_out, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse[last], d_lse, rtol=1e-13, atol=1e-13)


def test_row_subset_equals_the_full_result(oracle_lib):
    q, k, v, bt, lens, ql, scale = _case(5, [90, 33, 17, 48], [20, 1, 17, 16])
    out, lse = extend_ref.extend_attn(q, k, v, bt, lens, ql, scale)
    rows = np.array([0, 19, 20, 21, 37, 53])
    o2, l2 = extend_ref.extend_attn(q, k, v, bt, lens, ql, scale, rows=rows)
    assert np.array_equal(o2, out[rows]) and np.array_equal(l2, lse[rows])


def test_row_map_by_hand():
    seqs, pos = extend_ref.row_map([5, 3, 4], [2, 0, 4])
    assert seqs.tolist() == [0, 0, 2, 2, 2, 2]
    assert pos.tolist() == [3, 4, 0, 1, 2, 3]
    assert extend_ref.cu_lens([2, 0, 4]).tolist() == [0, 2, 2, 6]
    with pytest.raises(ValueError):
        extend_ref.row_map([3], [4])


def test_store_lands_where_the_dense_gather_reads_it():
    q, k, v, bt, lens, ql, scale = _case(6, [40, 18, 33], [25, 18, 1], hq=2, hkv=2, d=64)
    rng = np.random.default_rng(7)
    t = int(ql.sum())
    k_new = rng.integers(0, 0x7F00, size=(t, 2, 64)).astype(np.uint16)
    v_new = rng.integers(0, 0x7F00, size=(t, 2, 64)).astype(np.uint16)
    k2, v2 = k.copy(), v.copy()
    extend_ref.kv_store(k2, v2, bt, lens, ql, k_new, v_new)
    cu = extend_ref.cu_lens(ql)
    touched = 0
    for s in range(3):
        L, e = int(lens[s]), int(ql[s])
        for kvh in range(2):
            kd, vd = dense_ref.gather_dense(k2, v2, bt, s, kvh, L)
            kd0, vd0 = dense_ref.gather_dense(k, v, bt, s, kvh, L)
            assert np.array_equal(kd[: L - e], kd0[: L - e]) and np.array_equal(vd[: L - e], vd0[: L - e])
            for j in range(e):
                assert np.array_equal(kd[L - e + j], dense_ref.widen(k_new[cu[s] + j, kvh]))
                assert np.array_equal(vd[L - e + j], dense_ref.widen(v_new[cu[s] + j, kvh]))
                touched += 1
    # nothing else in the pools changed: every changed key element is in a stored slot
    assert touched == 2 * t
    changed_k = np.argwhere(k2 != k)
    changed_v = np.argwhere(v2 != v)
    slots = set()
    for s in range(3):
        L, e = int(lens[s]), int(ql[s])
        for p in range(L - e, L):
            slots.add((int(bt[s, p // PAGE]), p % PAGE))
    assert all((int(c[0]), int(c[3])) in slots for c in changed_k)
    assert all((int(c[0]), int(c[3])) in slots for c in changed_v)
