"""FP8 (OCP E4M3) encoding and the per-page quantizer of the KV cache, written plainly.

TEST INFRASTRUCTURE ONLY. The paper lists KV-cache quantization among the
optimizations its design is compatible with (Sec. 7). This library's variant
stores keys and values as OCP FP8 E4M3 codes with one fp32 scale per
(page, KV head) tile for K and one for V, which halves the bytes a decode step
reads. The code values come from the format definition (oracle.e4m3_value,
written in the C oracle); decode attention over such a cache is
oracle.decode_attn_fp8.

Encoding (round to nearest, ties to the even code; magnitudes above 448, the
largest finite code, saturate to it; the sign of zero is kept): codes 0x00 ..
0x7E have increasing values, so the nearest one is found by bisection over
that table and the sign bit added.

Quantizer of one tile (the valid slots of one page and KV head, bf16 values x):
  amax  = max |x|
  scale = fp32(amax / 448)          inv = fp32(448 / amax)     (both rounded once)
  code  = encode(fp32(x * inv))     (|x * inv| <= 448 up to that rounding)
An all-zero tile gets scale = inv = 1. Slots past the valid count get code 0.

fp8 tile layouts (16 * D bytes per (page, KV head) tile; byte of slot t, dim d):
  K: ((d // 64 * 4 + d % 32 // 8) * 16 + t) * 16 + (d // 32 % 2) * 8 + d % 8
  V: ((d // 64 * 4 + t // 4) * 16 + d % 16) * 16 + (d // 16 % 4) * 4 + t % 4
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

PAGE = 16
MAX_CODE = 0x7E


def values() -> np.ndarray:
    """Value of every code, float64 [256] (NaN for 0x7F and 0xFF)."""
    return np.array([oracle.e4m3_value(c) for c in range(256)])


def encode(x) -> np.ndarray:
    """E4M3 codes (uint8) of float32 values, round to nearest even."""
    x = np.asarray(x, dtype=np.float32)
    mag = np.abs(x.astype(np.float64))
    pos = values()[: MAX_CODE + 1]               # 0, subnormals, normals up to 448
    hi = np.clip(np.searchsorted(pos, mag, side="left"), 0, MAX_CODE)
    lo = np.clip(hi - 1, 0, MAX_CODE)
    d_lo = mag - pos[lo]
    d_hi = pos[hi] - mag
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0) & (hi != lo))
    code = np.where(pick_hi, hi, lo)
    code = np.where(mag >= pos[MAX_CODE], MAX_CODE, code)
    sign = np.signbit(x)
    return (code | np.where(sign, 0x80, 0)).astype(np.uint8)


def widen_bf16(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def quantize_tile(bits, valid_slots: int, slot_axis: int):
    """Codes (uint8, same shape) and scale (float32) of one tile of bf16 bits;
    only slots [0, valid_slots) along slot_axis count and are encoded."""
    xf = widen_bf16(bits)
    idx = [slice(None)] * xf.ndim
    idx[slot_axis] = slice(0, valid_slots)
    live = xf[tuple(idx)]
    amax = np.float32(np.max(np.abs(live))) if live.size else np.float32(0)
    if amax == 0:
        scale = inv = np.float32(1)
    else:
        scale = np.float32(amax) / np.float32(448)
        inv = np.float32(448) / np.float32(amax)
    codes = np.zeros(xf.shape, dtype=np.uint8)
    codes[tuple(idx)] = encode((live * inv).astype(np.float32))
    return codes, np.float32(scale)


def k_offset(t, d):
    t, d = np.asarray(t), np.asarray(d)
    return ((d // 64 * 4 + d % 32 // 8) * 16 + t) * 16 + (d // 32 % 2) * 8 + d % 8


def v_offset(t, d):
    t, d = np.asarray(t), np.asarray(d)
    return ((d // 64 * 4 + t // 4) * 16 + d % 16) * 16 + (d // 16 % 4) * 4 + t % 4


def _slot_dim(d):
    t, dim = np.meshgrid(np.arange(PAGE), np.arange(d), indexing="ij")
    return t.ravel(), dim.ravel()


def quantize_pages(k_bits, v_bits, pages, valid, k8, v8, k_scale, v_scale) -> None:
    """Quantizes the listed pages of bf16 pools (k_bits [N,Hkv,D/8,16,8],
    v_bits [N,Hkv,D,16] uint16) into fp8 pools [N,Hkv,16*D] (fp8 tile
    layouts) and scales [N,Hkv], in place. valid[i]: valid slots (1..16) of
    page pages[i]."""
    hkv, d = k_bits.shape[1], k_bits.shape[2] * 8
    t, dim = _slot_dim(d)
    ko, vo = k_offset(t, dim), v_offset(t, dim)
    for pg, nv in zip(pages, valid):
        pg, nv = int(pg), int(nv)
        for h in range(hkv):
            kc, k_scale[pg, h] = quantize_tile(k_bits[pg, h], nv, slot_axis=1)   # [D/8][16][8]
            vc, v_scale[pg, h] = quantize_tile(v_bits[pg, h], nv, slot_axis=1)   # [D][16]
            k8[pg, h, ko] = kc[dim // 8, t, dim % 8]
            v8[pg, h, vo] = vc[dim, t]


def quantize_pages_batched(k_bits, v_bits, pages, valid, k8, v8, k_scale, v_scale, chunk: int = 1024,
                           nthreads: int = 0) -> None:
    """quantize_pages over many pages at once: the same arithmetic per tile
    (amax over the valid slots, the two fp32 quotients, encode of fp32(x * inv),
    code 0 past the valid slots), with the tiles of `chunk` pages as one array.
    Pinned bit for bit against quantize_pages; used where the per-tile loop
    would take minutes (a full 32B-like cache). Chunks hold distinct pages and
    run in `nthreads` threads (0: the host's cores, at most 16)."""
    pages = np.asarray(pages, dtype=np.int64)
    valid = np.asarray(valid, dtype=np.int64)
    if np.unique(pages).size != pages.size:
        raise ValueError("pages must be distinct")
    hkv, d = k_bits.shape[1], k_bits.shape[2] * 8
    t, dim = _slot_dim(d)
    ko, vo = k_offset(t, dim), v_offset(t, dim)

    def run(i0):
        pg, nv = pages[i0:i0 + chunk], valid[i0:i0 + chunk]
        # K tile [D/8][16][8] (slot axis 1), V tile [D][16] (slot axis 1)
        for bits, dst, scales, offs, shape in ((k_bits, k8, k_scale, ko, (1, 1, 1, PAGE, 1)),
                                               (v_bits, v8, v_scale, vo, (1, 1, 1, PAGE))):
            x = widen_bf16(bits[pg])                                   # [n, Hkv, ...tile]
            slot = np.arange(PAGE).reshape(shape)
            live = slot < nv.reshape((-1,) + (1,) * (x.ndim - 1))
            xl = np.where(live, x, np.float32(0))
            amax = np.abs(xl).reshape(xl.shape[0], hkv, -1).max(axis=2).astype(np.float32)   # [n, Hkv]
            zero = amax == 0
            safe = np.where(zero, np.float32(1), amax)
            scale = np.where(zero, np.float32(1), safe / np.float32(448)).astype(np.float32)
            inv = np.where(zero, np.float32(1), np.float32(448) / safe).astype(np.float32)
            codes = encode((xl * inv.reshape(inv.shape + (1,) * (x.ndim - 2))).astype(np.float32))
            codes = np.where(live, codes, np.uint8(0))
            scales[pg] = scale
            if bits is k_bits:
                dst[pg[:, None, None], np.arange(hkv)[None, :, None], offs[None, None, :]] = codes[:, :, dim // 8, t, dim % 8]
            else:
                dst[pg[:, None, None], np.arange(hkv)[None, :, None], offs[None, None, :]] = codes[:, :, dim, t]

    if nthreads <= 0:
        nthreads = min(16, len(os.sched_getaffinity(0)))
    with ThreadPoolExecutor(nthreads) as ex:
        list(ex.map(run, range(0, pages.size, chunk)))
