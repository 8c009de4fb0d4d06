"""Writes exact_cases.json: tiny paged decode-attention cases with their
60-digit decimal results (oracle/exact_ref.py, the only code it calls).

Inputs are fixed here: values on the grid k/16 (exact in bf16), a two-page
pool with 16-token pages, and one case with large scores so exp(z) without a
max subtraction would overflow double. Run from the repository root:
    python tests/golden/make_exact_cases.py
"""
import json
import os
import struct
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import exact_ref  # noqa: E402

PAGE = 16


def grid_bits(vals):
    out = []
    for v in np.ravel(vals):
        u = struct.unpack("<I", struct.pack("<f", float(v)))[0]
        assert u & 0xFFFF == 0
        out.append(u >> 16)
    return np.array(out, dtype=np.uint16).reshape(np.shape(vals))


def case(name, lens, hq, hkv, d, n_pages, bt, scale, seed, q_mult=1.0):
    rng = np.random.default_rng(seed)
    q = grid_bits(rng.integers(-32, 33, size=(len(lens), hq, d)) / 16.0 * q_mult)
    k = grid_bits(rng.integers(-32, 33, size=(n_pages, hkv, d // 8, PAGE, 8)) / 16.0)
    v = grid_bits(rng.integers(-32, 33, size=(n_pages, hkv, d, PAGE)) / 16.0)
    bt = np.array(bt, dtype=np.int32)
    out, lse, dec = exact_ref.decode_attn(q, k, v, bt, np.array(lens), scale)
    return {
        "name": name,
        "lens": list(map(int, lens)), "num_q_heads": hq, "num_kv_heads": hkv, "head_dim": d,
        "scale": scale, "block_table": bt.tolist(),
        "q": q.tolist(), "k_pool": k.tolist(), "v_pool": v.tolist(),
        "out": {f"{s},{h}": [str(x) for x in dec[(s, h)][0]] for (s, h) in dec},
        "lse": {f"{s},{h}": str(dec[(s, h)][1]) for (s, h) in dec},
    }


def main():
    cases = [
        case("two_seqs_cross_page", [3, 18], 2, 1, 8, 3, [[2, -1], [0, 1]], 0.25, 1),
        case("gqa_g2", [5], 4, 2, 8, 1, [[0]], 0.5, 2),
        case("large_scores", [4], 1, 1, 8, 1, [[0]], 4.0, 3, q_mult=8.0),
    ]
    doc = {
        "about": "Decode attention (App. B.1 decode step: one query per sequence over its "
                 "paged cache) evaluated at 60 significant digits by oracle/exact_ref.py. "
                 "Layouts: q [B][Hq][D], k_pool [N][Hkv][D/8][16][8], v_pool [N][Hkv][D][16], "
                 "bf16 bit patterns; out/lse keyed by 'seq,head'.",
        "generator": "tests/golden/make_exact_cases.py",
        "cases": cases,
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "exact_cases.json")
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
