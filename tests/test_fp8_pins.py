"""Pins of the fp8 KV oracle on the CPU: the E4M3 code values and the encoder
against torch's own float8_e4m3fn conversions and hand-worked codes, the
per-page quantizer by hand and within the format's error bound, and fp8
attention against the bf16 oracle and a dense numpy path."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import dense_ref, fp8_ref

PAGE = 16


def test_code_values_match_torch_float8_e4m3fn():
    mine = fp8_ref.values()
    theirs = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(theirs))
    fin = ~np.isnan(mine)
    assert np.array_equal(mine[fin], theirs[fin])
    assert np.isnan(mine[[0x7F, 0xFF]]).all() and np.isnan(mine).sum() == 2


def test_code_values_by_hand():
    v = fp8_ref.values()
    assert (v[0x00], v[0x01], v[0x07], v[0x08], v[0x38], v[0x7E]) == (0.0, 2 ** -9, 7 * 2 ** -9, 2 ** -6, 1.0, 448.0)
    assert v[0xB8] == -1.0 and math.copysign(1.0, v[0x80]) == -1.0


def test_encoder_matches_torch_rounding():
    pos = np.unique(fp8_ref.values()[: 0x7F])
    mids = (pos[:-1] + pos[1:]) / 2
    rng = np.random.default_rng(0)
    xs = [pos, mids, np.nextafter(mids.astype(np.float32), np.float32(0)),
          np.nextafter(mids.astype(np.float32), np.float32(1e9)), rng.uniform(0, 460, 20000),
          np.exp(rng.uniform(np.log(2 ** -12), np.log(460), 20000))]
    x = np.concatenate([a.astype(np.float32) for a in xs])
    x = np.concatenate([x, -x]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(fp8_ref.encode(x), want)


def test_encoder_by_hand():
    x = np.array([0.0, -0.0, 2 ** -10, 3 * 2 ** -11, 1.5 * 2 ** -9, 1.0625, 1.0625 + 1e-3, 448.0, 460.0, 1e6, -7.0],
                 np.float32)
    # ties go to the even code: 2^-10 -> 0, 1.5 * 2^-9 -> 2 * 2^-9, 1 + 1/16 -> 1.0; beyond 448 saturates
    assert fp8_ref.encode(x).tolist() == [0x00, 0x80, 0x00, 0x01, 0x02, 0x38, 0x39, 0x7E, 0x7E, 0x7E, 0xCE]


def _bits(vals):
    a = np.asarray(vals, np.float32).view(np.uint32)
    assert np.all((a & 0xFFFF) == 0)
    return (a >> 16).astype(np.uint16)


def test_quantize_tile_by_hand():
    tile = np.zeros((2, PAGE), np.uint16)                 # a V tile: [dim][slot], D = 2
    tile[0, :3] = _bits([7.0, -3.5, 0.5])
    tile[1, :3] = _bits([0.0, 1.0, -0.25])
    tile[:, 3:] = 0x7FC0                                   # NaN past the 3 valid slots
    codes, scale = fp8_ref.quantize_tile(tile, 3, slot_axis=1)
    # amax 7: scale 7/448 = 2^-6, inv 64; 7 -> 448 (0x7E), -3.5 -> -224 (0xF6), 0.5 -> 32 (0x60),
    # 1 -> 64 (0x68), -0.25 -> -16 (0xD8)
    assert scale == np.float32(2 ** -6)
    assert codes[0, :3].tolist() == [0x7E, 0xF6, 0x60] and codes[1, :3].tolist() == [0x00, 0x68, 0xD8]
    assert not codes[:, 3:].any()
    zero, s0 = fp8_ref.quantize_tile(np.zeros((2, PAGE), np.uint16), 16, slot_axis=1)
    assert s0 == 1.0 and not zero.any()


def test_quantize_error_within_half_a_code_step():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((8, PAGE, 8)) * 3).astype(np.float32)
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)     # truncate to bf16
    xf = fp8_ref.widen_bf16(bits)
    codes, scale = fp8_ref.quantize_tile(bits, PAGE, slot_axis=1)
    back = fp8_ref.values()[codes] * np.float64(scale)
    y = np.abs(xf.astype(np.float64)) * (448 / np.abs(xf).max())
    # relative half-step 2^-4 for normal codes (|y| >= 2^-6), absolute 2^-10 * scale below
    bound = np.where(y >= 2 ** -6, np.abs(xf) * 2 ** -4, 2 ** -10 * float(scale)) * (1 + 1e-6) + 1e-12
    assert np.all(np.abs(back - xf) <= bound)


def _fp8_case(seed, lens, hq=4, hkv=2, d=64, pow2_scales=False):
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, np.int32)
    pages = -(-lens // PAGE)
    n = int(pages.sum()) + 2
    perm = rng.permutation(n)
    bt = np.full((lens.size, max(1, int(pages.max()))), -1, np.int32)
    off = 0
    for s in range(lens.size):
        bt[s, : pages[s]] = perm[off: off + pages[s]]
        off += pages[s]
    finite = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    k8 = rng.choice(finite, size=(n, hkv, PAGE * d))
    v8 = rng.choice(finite, size=(n, hkv, PAGE * d))
    if pow2_scales:
        ks = np.ldexp(1.0, rng.integers(-9, -4, size=(n, hkv))).astype(np.float32)
        vs = np.ldexp(1.0, rng.integers(-9, -4, size=(n, hkv))).astype(np.float32)
    else:
        ks = rng.uniform(1e-3, 3e-2, size=(n, hkv)).astype(np.float32)
        vs = rng.uniform(1e-3, 3e-2, size=(n, hkv)).astype(np.float32)
    qf = rng.standard_normal((lens.size, hq, d)).astype(np.float32)
    q = (qf.view(np.uint32) >> 16).astype(np.uint16)
    return q, k8, v8, ks, vs, bt, lens, 1 / math.sqrt(d)


def _dense_values(k8, v8, ks, vs, d):
    """Cached values as float64 in the bf16 pools' layouts ([N,Hkv,D/8,16,8] and [N,Hkv,D,16])."""
    vals = fp8_ref.values()
    t, dim = np.meshgrid(np.arange(PAGE), np.arange(d), indexing="ij")
    n, hkv = ks.shape
    kd = np.empty((n, hkv, d // 8, PAGE, 8))
    vd = np.empty((n, hkv, d, PAGE))
    kd[:, :, dim // 8, t, dim % 8] = vals[k8[:, :, fp8_ref.k_offset(t, dim)]] * ks[:, :, None, None]
    vd[:, :, dim, t] = vals[v8[:, :, fp8_ref.v_offset(t, dim)]] * vs[:, :, None, None]
    return kd, vd


def test_tile_layouts_are_bijections_with_contiguous_lane_pieces():
    for d in (64, 128):
        t, dim = np.meshgrid(np.arange(PAGE), np.arange(d), indexing="ij")
        for f in (fp8_ref.k_offset, fp8_ref.v_offset):
            assert np.array_equal(np.sort(f(t, dim).ravel()), np.arange(PAGE * d))
        # a key's 8 dims 8j .. 8j+7 of one slot, and a value's 4 slots 4j .. 4j+3 of one dim, are 8 / 4 bytes in a row
        assert np.all(np.diff(fp8_ref.k_offset(3, np.arange(8, 16))) == 1)
        assert np.all(np.diff(fp8_ref.v_offset(np.arange(4, 8), 5)) == 1)


def test_fp8_attention_equals_bf16_attention_on_the_same_values(oracle_lib):
    """With power-of-two scales every cached value is a bf16 value; the bf16
    oracle over those values must give the same bits."""
    q, k8, v8, ks, vs, bt, lens, scale = _fp8_case(2, [37, 16, 1, 50], pow2_scales=True)
    kd, vd = _dense_values(k8, v8, ks, vs, 64)
    kb = _bits(kd.astype(np.float32))
    vb = _bits(vd.astype(np.float32))
    o8, l8 = oracle.decode_attn_fp8(q, k8, v8, ks, vs, bt, lens, scale)
    ob, lb = oracle.decode_attn(q, kb, vb, bt, lens, scale)
    assert np.array_equal(o8, ob) and np.array_equal(l8, lb)


def test_fp8_attention_matches_dense_numpy(oracle_lib):
    q, k8, v8, ks, vs, bt, lens, scale = _fp8_case(3, [23, 40, 16], hq=6, hkv=3, d=128)
    o8, l8 = oracle.decode_attn_fp8(q, k8, v8, ks, vs, bt, lens, scale)
    vals = fp8_ref.values()
    g = 2
    for s, L in enumerate(lens):
        for h in range(6):
            kvh = h // g
            toks = np.arange(L)
            pg = bt[s, toks // PAGE]
            sl = toks % PAGE
            dims = np.arange(128)
            K = vals[k8[pg[:, None], kvh, fp8_ref.k_offset(sl[:, None], dims[None, :])]] * \
                ks[pg, kvh][:, None].astype(np.float64)
            V = vals[v8[pg[:, None], kvh, fp8_ref.v_offset(sl[:, None], dims[None, :])]] * \
                vs[pg, kvh][:, None].astype(np.float64)
            z = scale * (K @ dense_ref.widen(q[s, h]))
            w = np.exp(z - z.max())
            np.testing.assert_allclose(o8[s, h], (w @ V) / w.sum(), rtol=1e-12, atol=1e-15)
            assert l8[s, h] == pytest.approx(z.max() + np.log(w.sum()), rel=1e-13, abs=1e-13)


def test_fp8_scales_act_linearly(oracle_lib):
    q, k8, v8, ks, vs, bt, lens, scale = _fp8_case(4, [33, 7], pow2_scales=True)
    o, l = oracle.decode_attn_fp8(q, k8, v8, ks, vs, bt, lens, scale)
    o2, l2 = oracle.decode_attn_fp8(q, k8, v8, ks, vs * 2, bt, lens, scale)
    assert np.array_equal(o2, 2 * o) and np.array_equal(l2, l)
    o3, l3 = oracle.decode_attn_fp8(q, k8, v8, ks * 2, vs, bt, lens, scale)
    o4, l4 = oracle.decode_attn_fp8(q, k8, v8, ks, vs, bt, lens, scale * 2)
    assert np.array_equal(o3, o4) and np.array_equal(l3, l4)


def test_quantize_pages_places_codes_by_the_layouts():
    rng = np.random.default_rng(8)
    d, n = 64, 3
    kb = (rng.standard_normal((n, 1, d // 8, PAGE, 8)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    vb = (rng.standard_normal((n, 1, d, PAGE)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    k8 = np.zeros((n, 1, PAGE * d), np.uint8)
    v8 = np.zeros((n, 1, PAGE * d), np.uint8)
    ks = np.zeros((n, 1), np.float32)
    vs = np.zeros((n, 1), np.float32)
    fp8_ref.quantize_pages(kb, vb, [1], [16], k8, v8, ks, vs)
    kc, ksc = fp8_ref.quantize_tile(kb[1, 0], 16, slot_axis=1)
    vc, vsc = fp8_ref.quantize_tile(vb[1, 0], 16, slot_axis=1)
    assert ks[1, 0] == ksc and vs[1, 0] == vsc and not k8[0].any() and not k8[2].any()
    for t in (0, 5, 15):
        for dim in (0, 9, 33, 63):
            assert k8[1, 0, fp8_ref.k_offset(t, dim)] == kc[dim // 8, t, dim % 8]
            assert v8[1, 0, fp8_ref.v_offset(t, dim)] == vc[dim, t]


@pytest.mark.parametrize("d,hkv", [(64, 1), (128, 3)])
def test_batched_quantizer_equals_the_per_tile_one(d, hkv):
    """quantize_pages_batched against quantize_pages, bit for bit: partial
    pages (NaN past their valid slots), an all-zero tile, negative zeros, the
    largest and smallest bf16 magnitudes, unlisted pages left alone, and chunk
    edges crossed."""
    rng = np.random.default_rng(31 + d)
    n = 23

    def draw(shape):
        return (rng.standard_normal(shape).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)

    kb = draw((n, hkv, d // 8, PAGE, 8))
    vb = draw((n, hkv, d, PAGE))
    pages = rng.permutation(n)[:17]
    valid = rng.integers(1, PAGE + 1, size=pages.size)
    for pg, nv in zip(pages, valid):
        kb[pg, :, :, nv:, :] = 0x7FC0
        vb[pg, :, :, nv:] = 0x7FC0
    kb[pages[0]] = 0x8000 * (rng.random(kb[pages[0]].shape) < 0.5)   # all-zero tiles, signed zeros
    vb[pages[1], 0, 0, 0], vb[pages[1], 0, 1, 0] = 0x7F7F, 0x0001
    outs = []
    for fn, kw in ((fp8_ref.quantize_pages, {}), (fp8_ref.quantize_pages_batched, {"chunk": 5})):
        k8 = np.full((n, hkv, PAGE * d), 0xAA, np.uint8)
        v8 = np.full((n, hkv, PAGE * d), 0xAA, np.uint8)
        ks = np.full((n, hkv), -1.0, np.float32)
        vs = np.full((n, hkv), -1.0, np.float32)
        fn(kb, vb, pages, valid, k8, v8, ks, vs, **kw)
        outs.append((k8, v8, ks, vs))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
    assert outs[0][2][pages[0], 0] == 1.0
