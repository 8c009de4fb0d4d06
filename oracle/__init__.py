"""CPU oracle for paged decode attention.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers. Nothing here is used by the HIP
library or its Python binding, and nothing here imports them.

Modules:
  sf_oracle.c  fp64 attention over the gathered cache (C, OpenMP), wrapped below
  dense_ref    numpy float64 dense softmax attention on tiny inputs
  exact_ref    high-precision decimal attention for a handful of tokens
  merge_ref    fp64 log-sum-exp merge of partial attention results
  plan_ref     re-derivation of the split-K chunk plan from its stated rule
  append_ref   page allocator, KV append and the growing-cache decode loop
  extend_ref   extend (re-prefill) attention and the new-token store
  cost_ref     throughput cost model and routing
  fp8_ref      FP8 E4M3 encoding and the per-page quantizer of the KV cache
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sf_oracle.c")
_LIB = os.path.join(_HERE, "libsf_oracle.so")
_lib = None
BASE_FLAGS = ["-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared"]
# The CPU-baseline timing build: tuned for the host it runs on, so it is
# built on that host (bench.py does it at run time) and never shipped.
# -ffp-contract=off keeps a * b + c as two roundings, as in the test build.
NATIVE_FLAGS = ["-O3", "-march=native", "-ffp-contract=off", "-std=c11", "-fopenmp", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile sf_oracle.c with the host C compiler (plain -O2, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", *BASE_FLAGS, _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def build_native(out_dir: str) -> str:
    """Compile sf_oracle.c with NATIVE_FLAGS into out_dir (for timing on this
    host only); returns the library path."""
    os.makedirs(out_dir, exist_ok=True)
    path = os.path.join(out_dir, "libsf_oracle_native.so")
    subprocess.run(["gcc", *NATIVE_FLAGS, _SRC, "-o", path, "-lm"], check=True)
    return path


def _declare(L):
    p = ctypes.c_void_p
    i = ctypes.c_int
    L.sf_oracle_decode_attn.argtypes = [i, i, i, i, i, i, i, p, p, p, p, p, ctypes.c_double, p, p, i]
    L.sf_oracle_decode_attn.restype = i
    L.sf_oracle_gather.argtypes = [i, i, i, i, i, p, p, p, i, i, i, p, p]
    L.sf_oracle_gather.restype = i
    L.sf_oracle_max_threads.restype = i
    L.sf_oracle_decode_attn_fp8.argtypes = [i, i, i, i, i, i, i, p, p, p, p, p, p, p, ctypes.c_double, p, p, i]
    L.sf_oracle_decode_attn_fp8.restype = i
    L.sf_oracle_e4m3_value.argtypes = [i]
    L.sf_oracle_e4m3_value.restype = ctypes.c_double
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = _declare(ctypes.CDLL(_LIB))
    return _lib


def load(path: str):
    """A separately built copy of the oracle (build_native)."""
    return _declare(ctypes.CDLL(path))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    assert a.dtype == np.uint16, a.dtype
    return a


def decode_attn(q, k_pool, v_pool, block_table, seq_lens, scale, nthreads: int = 0, using=None):
    """fp64 reference. q [B,Hq,D], k_pool [N,Hkv,D/8,16,8] and v_pool
    [N,Hkv,D,16] are uint16 bf16 bit arrays; returns (out [B,Hq,D] float64,
    lse [B,Hq] float64). using: a library from load() instead of the default."""
    q = _u16(q)
    k_pool = _u16(k_pool)
    v_pool = _u16(v_pool)
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    b, hq, d = q.shape
    n, hkv, groups, p, eight = k_pool.shape
    assert groups * eight == d and eight == 8
    assert v_pool.shape == (n, hkv, d, p) and bt.shape[0] == b and lens.shape == (b,)
    out = np.empty((b, hq, d), dtype=np.float64)
    lse = np.empty((b, hq), dtype=np.float64)
    rc = (using or lib()).sf_oracle_decode_attn(b, hq, hkv, d, p, bt.shape[1], n, _ptr(q), _ptr(k_pool),
                                     _ptr(v_pool), _ptr(bt), _ptr(lens), float(scale),
                                     _ptr(out), _ptr(lse), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle rejected its input (code {rc})")
    return out, lse


def decode_attn_fp8(q, k8, v8, k_scale, v_scale, block_table, seq_lens, scale, nthreads: int = 0):
    """fp64 reference over an fp8 (OCP E4M3) cache with per-(page, KV head)
    scales. q: uint16 bf16 bits [B,Hq,D]; k8, v8: uint8 codes [N,Hkv,16*D]
    in the fp8 tile layouts (sf_oracle.c); k_scale, v_scale float32 [N,Hkv]."""
    q = _u16(q)
    k8 = np.ascontiguousarray(k8, dtype=np.uint8)
    v8 = np.ascontiguousarray(v8, dtype=np.uint8)
    ks = np.ascontiguousarray(k_scale, dtype=np.float32)
    vs = np.ascontiguousarray(v_scale, dtype=np.float32)
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    b, hq, d = q.shape
    n, hkv, tile = k8.shape
    assert tile == 16 * d and v8.shape == (n, hkv, tile) and ks.shape == (n, hkv) and vs.shape == (n, hkv)
    out = np.empty((b, hq, d), dtype=np.float64)
    lse = np.empty((b, hq), dtype=np.float64)
    rc = lib().sf_oracle_decode_attn_fp8(b, hq, hkv, d, 16, bt.shape[1], n, _ptr(q), _ptr(k8), _ptr(v8), _ptr(ks),
                                         _ptr(vs), _ptr(bt), _ptr(lens), float(scale), _ptr(out), _ptr(lse),
                                         int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle rejected its input (code {rc})")
    return out, lse


def e4m3_value(code: int) -> float:
    """The value of an OCP FP8 E4M3 code, from the format definition (C side)."""
    return float(lib().sf_oracle_e4m3_value(int(code)))


def gather(k_pool, v_pool, block_table, seq: int, kvh: int, length: int):
    """Dense [L, D] uint16 copies of one (sequence, KV head)'s cached K and V."""
    k_pool = _u16(k_pool)
    v_pool = _u16(v_pool)
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    n, hkv, groups, p, eight = k_pool.shape
    d = groups * eight
    kd = np.empty((length, d), dtype=np.uint16)
    vd = np.empty((length, d), dtype=np.uint16)
    rc = lib().sf_oracle_gather(hkv, d, p, bt.shape[1], n, _ptr(k_pool), _ptr(v_pool), _ptr(bt),
                                int(seq), int(kvh), int(length), _ptr(kd), _ptr(vd))
    if rc != 0:
        raise ValueError("oracle gather hit an invalid page")
    return kd, vd


def max_threads() -> int:
    return int(lib().sf_oracle_max_threads())
