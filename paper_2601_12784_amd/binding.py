"""ctypes binding of libsf_decode_attn.so (argument marshalling only).

The names mirror the C entry points declared in include/sf_decode_attn.h.
Every step of the computation runs in the HIP library; PyTorch only supplies
device memory and the stream. If the library is missing this module raises:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import torch

PKG = os.path.dirname(os.path.abspath(__file__))
# SF_DECODE_ATTN_LIB selects another build of the same library (the
# sanitized CPU-test copy of build.py --sanitize); default: the in-tree one.
LIB_PATH = os.environ.get("SF_DECODE_ATTN_LIB") or os.path.join(PKG, "libsf_decode_attn.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "sf_decode_attn.h")
PAGE = 16
ITEM_INTS = 8

STATUS = {0: "SF_OK", 1: "SF_ERR_INVALID_ARG", 2: "SF_ERR_UNSUPPORTED", 3: "SF_ERR_CAPACITY",
          4: "SF_ERR_PLAN_MISMATCH", 5: "SF_ERR_HIP"}


class SfError(RuntimeError):
    def __init__(self, where: str, status: int):
        self.status = int(status)
        super().__init__(f"{where}: {STATUS.get(self.status, self.status)} ({status_string(self.status)})")


class sf_attn_desc(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("block_table_stride", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("softmax_scale", ctypes.c_float)]


class sf_plan_opts(ctypes.Structure):
    _fields_ = [("num_cus", ctypes.c_int32), ("chunk_pages", ctypes.c_int32),
                ("workers_per_cu", ctypes.c_int32), ("min_chunk_pages", ctypes.c_int32),
                ("xcd_parity_skew", ctypes.c_int32)]


class sf_plan_info(ctypes.Structure):
    _fields_ = [("num_workers", ctypes.c_int32), ("num_work", ctypes.c_int32),
                ("num_combine", ctypes.c_int32), ("num_partials", ctypes.c_int32),
                ("chunk_pages", ctypes.c_int32), ("workers_per_group", ctypes.c_int32),
                ("work_bytes", ctypes.c_uint64), ("workspace_bytes", ctypes.c_uint64),
                ("desc_key", ctypes.c_uint64)]


class sf_extend_info(ctypes.Structure):
    _fields_ = [("num_items", ctypes.c_int32), ("tokens_per_item", ctypes.c_int32),
                ("num_q_rows", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("work_bytes", ctypes.c_uint64), ("desc_key", ctypes.c_uint64)]


class sf_runner_extras(ctypes.Structure):
    _fields_ = [("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p), ("new_pages_host", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p), ("attn_start", ctypes.c_void_p),
                ("attn_end", ctypes.c_void_p)]


class sf_cost_model(ctypes.Structure):
    _fields_ = [("k1", ctypes.c_double), ("k2", ctypes.c_double), ("k3", ctypes.c_double),
                ("k4", ctypes.c_double), ("k5", ctypes.c_double), ("kv_budget", ctypes.c_double)]


class sf_instance_state(ctypes.Structure):
    _fields_ = [("version", ctypes.c_int32), ("num_running", ctypes.c_int32),
                ("num_waiting", ctypes.c_int32), ("reserved", ctypes.c_int32), ("kv_cache", ctypes.c_double)]


class sf_trajectory(ctypes.Structure):
    _fields_ = [("version", ctypes.c_int32), ("reserved", ctypes.c_int32), ("length", ctypes.c_double)]


_lib = None


def lib():
    """Loads the HIP library (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2601_12784_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    L.sf_decode_attn_plan.argtypes = [P(sf_attn_desc), vp, P(sf_plan_opts), vp, ctypes.c_uint64,
                                      P(sf_plan_info)]
    L.sf_decode_attn.argtypes = [P(sf_attn_desc), P(sf_plan_info), vp, vp, vp, vp, vp, vp, vp, vp,
                                 vp, ctypes.c_uint64, vp]
    L.sf_decode_attn_combine.argtypes = [P(sf_attn_desc), P(sf_plan_info), vp, vp, ctypes.c_uint64,
                                         vp, vp, vp]
    L.sf_decode_attn_scratch.argtypes = [P(sf_attn_desc), P(sf_plan_info), vp, vp, vp, vp, vp, vp, vp, vp]
    L.sf_debug_gather_kv.argtypes = [P(sf_attn_desc), vp, vp, vp, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, vp, vp, vp]
    L.sf_decode_attn_append.argtypes = [P(sf_attn_desc), P(sf_plan_info), vp, vp, vp, vp, vp, vp, vp, vp,
                                        vp, vp, vp, vp, ctypes.c_uint64, vp]
    L.sf_runner_create.argtypes = [P(sf_attn_desc), P(sf_plan_opts), P(vp)]
    L.sf_runner_reserve.argtypes = [vp, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, vp]
    L.sf_runner_reserve.restype = ctypes.c_int
    L.sf_runner_destroy.argtypes = [vp]
    L.sf_runner_destroy.restype = None
    L.sf_runner_step.argtypes = [vp, P(sf_attn_desc), vp, vp, vp, vp, vp, vp, vp, P(sf_runner_extras), vp,
                                 P(sf_plan_info)]
    L.sf_debug_stream_read.argtypes = [vp, ctypes.c_uint64, vp, ctypes.c_int32, vp, vp, vp]
    L.sf_decode_attn_fp8.argtypes = [P(sf_attn_desc), P(sf_plan_info), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                     ctypes.c_uint64, vp]
    L.sf_kv_quantize_fp8.argtypes = [P(sf_attn_desc), vp, vp, vp, vp, ctypes.c_int32, vp, vp, vp, vp, vp]
    L.sf_extend_attn_plan.argtypes = [P(sf_attn_desc), vp, vp, vp, ctypes.c_uint64, P(sf_extend_info)]
    L.sf_extend_attn.argtypes = [P(sf_attn_desc), P(sf_extend_info), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.sf_page_pool_create.argtypes = [ctypes.c_int32, P(vp)]
    L.sf_page_pool_destroy.argtypes = [vp]
    L.sf_page_pool_destroy.restype = None
    L.sf_page_pool_available.argtypes = [vp]
    L.sf_page_pool_available.restype = ctypes.c_int32
    for fn in ("sf_page_pool_claim", "sf_page_pool_release"):
        getattr(L, fn).argtypes = [vp, vp, ctypes.c_int32]
    L.sf_page_pool_alloc.argtypes = [vp, ctypes.c_int32, vp]
    L.sf_page_table_step.argtypes = [vp, vp, ctypes.c_int32, ctypes.c_int32, vp, vp, ctypes.c_int32, vp]
    L.sf_cost_throughput.argtypes = [P(sf_cost_model), P(sf_instance_state)]
    L.sf_cost_marginal_gain.argtypes = [P(sf_cost_model), P(sf_instance_state), ctypes.c_double]
    L.sf_cost_ideal_gain.argtypes = [P(sf_cost_model), ctypes.c_double]
    for fn in ("sf_cost_throughput", "sf_cost_marginal_gain", "sf_cost_ideal_gain"):
        getattr(L, fn).restype = ctypes.c_double
    L.sf_check_block_table.argtypes = [P(sf_attn_desc), vp, vp, P(ctypes.c_int32)]
    L.sf_check_block_table.restype = ctypes.c_int
    L.sf_route.argtypes = [P(sf_cost_model), ctypes.c_double, ctypes.c_int32, vp, ctypes.c_int32, vp,
                           ctypes.c_int32, vp, P(ctypes.c_int32)]
    for fn in ("sf_decode_attn_plan", "sf_decode_attn", "sf_decode_attn_combine", "sf_debug_gather_kv",
               "sf_decode_attn_append", "sf_page_pool_create", "sf_page_pool_claim", "sf_page_pool_alloc",
               "sf_page_pool_release", "sf_page_table_step", "sf_route", "sf_extend_attn_plan",
               "sf_extend_attn", "sf_decode_attn_fp8", "sf_kv_quantize_fp8", "sf_runner_create",
               "sf_runner_step", "sf_debug_stream_read", "sf_decode_attn_scratch"):
        getattr(L, fn).restype = ctypes.c_int
    L.sf_status_string.argtypes = [ctypes.c_int]
    L.sf_status_string.restype = ctypes.c_char_p
    L.sf_version.restype = ctypes.c_int32
    _lib = L
    return L


def header_functions() -> list[str]:
    """Names of the functions include/sf_decode_attn.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sf_[a-z0-9_]+)\s*\(", text)))


# SF_DEBUG_CHECKS=1: before each launch the classes below check every block-
# table entry the launch will read against the pool size (sf_check_block_table),
# on a host copy (DecodeLoopRunner keeps one; the others copy the device table
# back, which synchronizes: a debugging aid, not for timing).
DEBUG_CHECKS = os.environ.get("SF_DEBUG_CHECKS", "") not in ("", "0")


def check_block_table(desc: sf_attn_desc, block_table_host, seq_lens) -> None:
    """Raises SfError (naming the first bad sequence) unless every block-table
    entry a step over seq_lens reads lies in [0, desc.num_pages)."""
    bt = np.ascontiguousarray(block_table_host.cpu().numpy() if isinstance(block_table_host, torch.Tensor)
                              else block_table_host, dtype=np.int32)
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    if bt.shape != (desc.num_seqs, desc.block_table_stride) or lens.shape != (desc.num_seqs,):
        raise ValueError("block table or lengths do not match the descriptor")
    bad = ctypes.c_int32(-1)
    st = lib().sf_check_block_table(ctypes.byref(desc), bt.ctypes.data, lens.ctypes.data, ctypes.byref(bad))
    if st != 0:
        raise SfError(f"sf_check_block_table (sequence {bad.value})", st)


def status_string(status: int) -> str:
    return lib().sf_status_string(int(status)).decode()


def version() -> int:
    return int(lib().sf_version())


def make_desc(num_seqs, num_q_heads, num_kv_heads, head_dim, block_table_stride, num_pages,
              softmax_scale, page_size=PAGE) -> sf_attn_desc:
    return sf_attn_desc(int(num_seqs), int(num_q_heads), int(num_kv_heads), int(head_dim),
                        int(page_size), int(block_table_stride), int(num_pages), float(softmax_scale))


def make_opts(num_cus=0, chunk_pages=0, workers_per_cu=0, min_chunk_pages=0, xcd_parity_skew=0):
    return sf_plan_opts(int(num_cus), int(chunk_pages), int(workers_per_cu), int(min_chunk_pages),
                        int(xcd_parity_skew))


def _addr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(type(x))


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(where, st):
    if st != 0:
        raise SfError(where, st)


def _dev(t: torch.Tensor, name: str, dtype, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on the GPU (got {t.device})")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


# ----------------------------------------------------------------------------
# the C entry points
# ----------------------------------------------------------------------------
def sf_decode_attn_plan(desc: sf_attn_desc, seq_lens, opts: sf_plan_opts | None = None,
                        work_host=None):
    """Plans one decode step on the host. seq_lens: int32 host array/tensor.

    work_host: int32 host buffer (numpy or CPU tensor, pinned for async
    uploads) or None to allocate a numpy buffer of the right size.
    Returns (info, work_host)."""
    if isinstance(seq_lens, torch.Tensor):
        seq_lens = seq_lens.cpu().numpy()
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    if lens.shape != (desc.num_seqs,):
        raise ValueError("seq_lens must have num_seqs entries")
    info = sf_plan_info()
    L = lib()
    op = ctypes.byref(opts) if opts is not None else None
    if work_host is None:
        _check("sf_decode_attn_plan", L.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, op,
                                                            None, 0, ctypes.byref(info)))
        work_host = np.empty(max(1, info.work_bytes // 4), dtype=np.int32)
    cap = work_host.numel() * 4 if isinstance(work_host, torch.Tensor) else work_host.nbytes
    _check("sf_decode_attn_plan", L.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, op,
                                                        _addr(work_host), cap, ctypes.byref(info)))
    return info, work_host


def sf_decode_attn(desc, info, work_host, work_dev, q, k_pool, v_pool, block_table, out, lse=None,
                   workspace=None, stream=None):
    """Enqueues the attention kernel (and the work-list upload if work_host is given)."""
    b, hq, hkv, d = desc.num_seqs, desc.num_q_heads, desc.num_kv_heads, desc.head_dim
    _dev(q, "q", torch.bfloat16, (b, hq, d))
    _dev(k_pool, "k_pool", torch.bfloat16, (desc.num_pages, hkv, d // 8, PAGE, 8))
    _dev(v_pool, "v_pool", torch.bfloat16, (desc.num_pages, hkv, d, PAGE))
    _dev(block_table, "block_table", torch.int32, (b, desc.block_table_stride))
    _dev(out, "out", torch.float32, (b, hq, d))
    _dev(work_dev, "work_dev", torch.int32)
    if work_dev.numel() * 4 < info.work_bytes:
        raise ValueError("work_dev is smaller than the plan")
    if lse is not None:
        _dev(lse, "lse", torch.float32, (b, hq))
    ws_bytes = 0
    if workspace is not None:
        _dev(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    _check("sf_decode_attn", lib().sf_decode_attn(
        ctypes.byref(desc), ctypes.byref(info), _addr(work_host), _addr(work_dev), _addr(q),
        _addr(k_pool), _addr(v_pool), _addr(block_table), _addr(out), _addr(lse),
        _addr(workspace), ws_bytes, _stream(stream)))


def sf_decode_attn_fp8(desc, info, work_host, work_dev, q, k_pool8, v_pool8, k_scale, v_scale, block_table, out,
                       lse=None, workspace=None, stream=None):
    """Enqueues the attention kernel over an fp8 cache (uint8 pools, fp32 scales [N, Hkv])."""
    b, hq, hkv, d = desc.num_seqs, desc.num_q_heads, desc.num_kv_heads, desc.head_dim
    _dev(q, "q", torch.bfloat16, (b, hq, d))
    _dev(k_pool8, "k_pool8", torch.uint8, (desc.num_pages, hkv, PAGE * d))
    _dev(v_pool8, "v_pool8", torch.uint8, (desc.num_pages, hkv, PAGE * d))
    _dev(k_scale, "k_scale", torch.float32, (desc.num_pages, hkv))
    _dev(v_scale, "v_scale", torch.float32, (desc.num_pages, hkv))
    _dev(block_table, "block_table", torch.int32, (b, desc.block_table_stride))
    _dev(out, "out", torch.float32, (b, hq, d))
    _dev(work_dev, "work_dev", torch.int32)
    if work_dev.numel() * 4 < info.work_bytes:
        raise ValueError("work_dev is smaller than the plan")
    if lse is not None:
        _dev(lse, "lse", torch.float32, (b, hq))
    ws_bytes = 0
    if workspace is not None:
        _dev(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    _check("sf_decode_attn_fp8", lib().sf_decode_attn_fp8(
        ctypes.byref(desc), ctypes.byref(info), _addr(work_host), _addr(work_dev), _addr(q), _addr(k_pool8),
        _addr(v_pool8), _addr(k_scale), _addr(v_scale), _addr(block_table), _addr(out), _addr(lse),
        _addr(workspace), ws_bytes, _stream(stream)))


def sf_kv_quantize_fp8(desc, k_pool, v_pool, pages, valid_slots, k_pool8, v_pool8, k_scale, v_scale, stream=None):
    """Quantizes the listed pages (device int32 pages / valid_slots) of bf16 pools into fp8 ones."""
    hkv, d = desc.num_kv_heads, desc.head_dim
    _dev(k_pool, "k_pool", torch.bfloat16, (desc.num_pages, hkv, d // 8, PAGE, 8))
    _dev(v_pool, "v_pool", torch.bfloat16, (desc.num_pages, hkv, d, PAGE))
    _dev(pages, "pages", torch.int32)
    _dev(valid_slots, "valid_slots", torch.int32, tuple(pages.shape))
    _dev(k_pool8, "k_pool8", torch.uint8, (desc.num_pages, hkv, PAGE * d))
    _dev(v_pool8, "v_pool8", torch.uint8, (desc.num_pages, hkv, PAGE * d))
    _dev(k_scale, "k_scale", torch.float32, (desc.num_pages, hkv))
    _dev(v_scale, "v_scale", torch.float32, (desc.num_pages, hkv))
    _check("sf_kv_quantize_fp8", lib().sf_kv_quantize_fp8(
        ctypes.byref(desc), _addr(k_pool), _addr(v_pool), _addr(pages), _addr(valid_slots), int(pages.numel()),
        _addr(k_pool8), _addr(v_pool8), _addr(k_scale), _addr(v_scale), _stream(stream)))


def sf_decode_attn_append(desc, info, work_host, work_dev, q, k_new, v_new, new_pages, k_pool, v_pool,
                          block_table, out, lse, workspace=None, stream=None):
    """Enqueues an appending decode pass: attention over every sequence
    including its newest token (k_new, v_new: bf16 [B, Hkv, D]), then the
    merge of split sequences and the token stores into the pools and the
    block table (so no separate combine call). new_pages: device int32 [B]
    (-1 = no new page) or None."""
    b, hq, hkv, d = desc.num_seqs, desc.num_q_heads, desc.num_kv_heads, desc.head_dim
    _dev(q, "q", torch.bfloat16, (b, hq, d))
    _dev(k_new, "k_new", torch.bfloat16, (b, hkv, d))
    _dev(v_new, "v_new", torch.bfloat16, (b, hkv, d))
    if new_pages is not None:
        _dev(new_pages, "new_pages", torch.int32, (b,))
    _dev(k_pool, "k_pool", torch.bfloat16, (desc.num_pages, hkv, d // 8, PAGE, 8))
    _dev(v_pool, "v_pool", torch.bfloat16, (desc.num_pages, hkv, d, PAGE))
    _dev(block_table, "block_table", torch.int32, (b, desc.block_table_stride))
    _dev(out, "out", torch.float32, (b, hq, d))
    _dev(work_dev, "work_dev", torch.int32)
    if work_dev.numel() * 4 < info.work_bytes:
        raise ValueError("work_dev is smaller than the plan")
    if lse is None:
        raise ValueError("sf_decode_attn_append needs an lse buffer (the merge reads it back)")
    _dev(lse, "lse", torch.float32, (b, hq))
    ws_bytes = 0
    if workspace is not None:
        _dev(workspace, "workspace", workspace.dtype)
        ws_bytes = workspace.numel() * workspace.element_size()
    _check("sf_decode_attn_append", lib().sf_decode_attn_append(
        ctypes.byref(desc), ctypes.byref(info), _addr(work_host), _addr(work_dev), _addr(q), _addr(k_new),
        _addr(v_new), _addr(new_pages), _addr(k_pool), _addr(v_pool), _addr(block_table), _addr(out),
        _addr(lse), _addr(workspace), ws_bytes, _stream(stream)))


def sf_extend_attn_plan(desc: sf_attn_desc, seq_lens, q_lens, work_host=None):
    """Plans extend attention on the host. seq_lens (L_s, new tokens
    included) and q_lens (E_s): int32 host arrays. Returns (info, work_host)."""
    lens = np.ascontiguousarray(np.asarray(seq_lens), dtype=np.int32)
    qls = np.ascontiguousarray(np.asarray(q_lens), dtype=np.int32)
    if lens.shape != (desc.num_seqs,) or qls.shape != (desc.num_seqs,):
        raise ValueError("seq_lens and q_lens must have num_seqs entries")
    info = sf_extend_info()
    L = lib()
    if work_host is None:
        _check("sf_extend_attn_plan", L.sf_extend_attn_plan(ctypes.byref(desc), lens.ctypes.data, qls.ctypes.data,
                                                            None, 0, ctypes.byref(info)))
        work_host = np.empty(max(1, info.work_bytes // 4), dtype=np.int32)
    cap = work_host.numel() * 4 if isinstance(work_host, torch.Tensor) else work_host.nbytes
    _check("sf_extend_attn_plan", L.sf_extend_attn_plan(ctypes.byref(desc), lens.ctypes.data, qls.ctypes.data,
                                                        _addr(work_host), cap, ctypes.byref(info)))
    return info, work_host


def sf_extend_attn(desc, info, work_host, work_dev, q, k_pool, v_pool, block_table, out, lse=None,
                   k_new=None, v_new=None, stream=None):
    """Enqueues extend attention (after the store of k_new / v_new into the
    pools when both are given). q, out: [T, Hq, D]; k_new, v_new: [T, Hkv, D]."""
    t, hq, hkv, d = info.num_q_rows, desc.num_q_heads, desc.num_kv_heads, desc.head_dim
    _dev(q, "q", torch.bfloat16, (t, hq, d))
    _dev(k_pool, "k_pool", torch.bfloat16, (desc.num_pages, hkv, d // 8, PAGE, 8))
    _dev(v_pool, "v_pool", torch.bfloat16, (desc.num_pages, hkv, d, PAGE))
    _dev(block_table, "block_table", torch.int32, (desc.num_seqs, desc.block_table_stride))
    _dev(out, "out", torch.float32, (t, hq, d))
    _dev(work_dev, "work_dev", torch.int32)
    if work_dev.numel() * 4 < info.work_bytes:
        raise ValueError("work_dev is smaller than the plan")
    if lse is not None:
        _dev(lse, "lse", torch.float32, (t, hq))
    if (k_new is None) != (v_new is None):
        raise ValueError("give both k_new and v_new, or neither")
    if k_new is not None:
        _dev(k_new, "k_new", torch.bfloat16, (t, hkv, d))
        _dev(v_new, "v_new", torch.bfloat16, (t, hkv, d))
    _check("sf_extend_attn", lib().sf_extend_attn(
        ctypes.byref(desc), ctypes.byref(info), _addr(work_host), _addr(work_dev), _addr(q), _addr(k_new),
        _addr(v_new), _addr(k_pool), _addr(v_pool), _addr(block_table), _addr(out), _addr(lse),
        _stream(stream)))


class ExtendAttention:
    """Plans and launches extend attention for one batch of re-prefills.

    The work list is planned on the host at each call, written into a pinned
    buffer and uploaded with the launch; everything else runs in the
    library's kernels. Before the pinned buffer is rewritten, the call waits
    for the event recorded after the previous upload, so a queued copy never
    reads a half-written list."""

    def __init__(self, num_q_heads, num_kv_heads, head_dim, device=None):
        self.hq, self.hkv, self.d = int(num_q_heads), int(num_kv_heads), int(head_dim)
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self._work_host = None
        self._work_dev = None
        self._uploaded = None
        self.last_info = None

    def __call__(self, q, k_pool, v_pool, block_table, seq_lens, q_lens, scale, out=None, lse=None,
                 k_new=None, v_new=None, stream=None):
        lens = np.ascontiguousarray(np.asarray(seq_lens), dtype=np.int32)
        qls = np.ascontiguousarray(np.asarray(q_lens), dtype=np.int32)
        desc = make_desc(lens.size, self.hq, self.hkv, self.d, block_table.shape[1], k_pool.shape[0], scale)
        info = sf_extend_info()
        _check("sf_extend_attn_plan", lib().sf_extend_attn_plan(ctypes.byref(desc), lens.ctypes.data,
                                                                qls.ctypes.data, None, 0, ctypes.byref(info)))
        need = max(8, int(info.work_bytes) // 4)
        if self._uploaded is not None:
            self._uploaded.synchronize()
        if self._work_host is None or self._work_host.numel() < need:
            self._work_host = torch.empty(need, dtype=torch.int32, pin_memory=True)
            self._work_dev = torch.empty(need, dtype=torch.int32, device=self.device)
        info, _ = sf_extend_attn_plan(desc, lens, qls, work_host=self._work_host)
        if DEBUG_CHECKS:
            check_block_table(desc, block_table, np.where(qls > 0, lens, 0))
        if out is None:
            out = torch.empty((info.num_q_rows, self.hq, self.d), dtype=torch.float32, device=self.device)
        sf_extend_attn(desc, info, self._work_host, self._work_dev, q, k_pool, v_pool, block_table, out, lse,
                       k_new=k_new, v_new=v_new, stream=stream)
        ev = torch.cuda.Event()
        ev.record(stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.current_stream())
        self._uploaded = ev
        self.last_info = info
        return out


class PagePool:
    """The library's host page allocator (LIFO free list over page ids)."""

    def __init__(self, num_pages: int):
        self._p = ctypes.c_void_p()
        self._L = lib()
        _check("sf_page_pool_create", self._L.sf_page_pool_create(int(num_pages), ctypes.byref(self._p)))
        self.num_pages = int(num_pages)

    def available(self) -> int:
        return int(self._L.sf_page_pool_available(self._p))

    def claim(self, pages) -> None:
        a = np.ascontiguousarray(pages, dtype=np.int32)
        _check("sf_page_pool_claim", self._L.sf_page_pool_claim(self._p, a.ctypes.data, a.size))

    def alloc(self, n: int) -> np.ndarray:
        out = np.empty(max(0, int(n)), dtype=np.int32)
        _check("sf_page_pool_alloc", self._L.sf_page_pool_alloc(self._p, int(n), out.ctypes.data))
        return out

    def release(self, pages) -> None:
        a = np.ascontiguousarray(pages, dtype=np.int32)
        _check("sf_page_pool_release", self._L.sf_page_pool_release(self._p, a.ctypes.data, a.size))

    def __del__(self):
        p = getattr(self, "_p", None)
        if p is not None and p.value:
            self._L.sf_page_pool_destroy(p)
        self._p = None


def cost_throughput(model: sf_cost_model, state: sf_instance_state) -> float:
    return float(lib().sf_cost_throughput(ctypes.byref(model), ctypes.byref(state)))


def cost_marginal_gain(model: sf_cost_model, state: sf_instance_state, length: float) -> float:
    return float(lib().sf_cost_marginal_gain(ctypes.byref(model), ctypes.byref(state), float(length)))


def cost_ideal_gain(model: sf_cost_model, length: float) -> float:
    return float(lib().sf_cost_ideal_gain(ctypes.byref(model), float(length)))


def route(model: sf_cost_model, mu: float, min_initial_version: int, instances, trajectories):
    """sf_route on objects with version/running/waiting/kv (instances) and
    version (None = initial)/length (trajectories). Returns (targets, the
    updated instances as sf_instance_state)."""
    ni, nt = len(instances), len(trajectories)
    inst = (sf_instance_state * max(1, ni))()
    for i, s in enumerate(instances):
        inst[i] = sf_instance_state(int(s.version), int(s.running), int(s.waiting), 0, float(s.kv))
    tr = (sf_trajectory * max(1, nt))()
    for j, t in enumerate(trajectories):
        tr[j] = sf_trajectory(-1 if t.version is None else int(t.version), 0, float(t.length))
    target = np.full(max(1, nt), -1, dtype=np.int32)
    routed = ctypes.c_int32()
    _check("sf_route", lib().sf_route(ctypes.byref(model), float(mu), int(min_initial_version), inst, ni, tr, nt,
                                      target.ctypes.data, ctypes.byref(routed)))
    after = [_InstanceView(inst[i]) for i in range(ni)]
    return target[:nt].tolist(), after


class _InstanceView:
    def __init__(self, s: sf_instance_state):
        self.version, self.running, self.waiting, self.kv = s.version, s.num_running, s.num_waiting, s.kv_cache


def sf_decode_attn_combine(desc, info, work_dev, workspace, out, lse=None, stream=None):
    """Enqueues the log-sum-exp merge of split sequences (no-op if none)."""
    if info.num_combine == 0:
        return
    _dev(out, "out", torch.float32, (desc.num_seqs, desc.num_q_heads, desc.head_dim))
    _dev(work_dev, "work_dev", torch.int32)
    _dev(workspace, "workspace", workspace.dtype)
    if lse is not None:
        _dev(lse, "lse", torch.float32, (desc.num_seqs, desc.num_q_heads))
    _check("sf_decode_attn_combine", lib().sf_decode_attn_combine(
        ctypes.byref(desc), ctypes.byref(info), _addr(work_dev), _addr(workspace),
        workspace.numel() * workspace.element_size(), _addr(out), _addr(lse), _stream(stream)))


SCRATCH_BYTES = 32 << 20   # SF_SCRATCH_BYTES of the header


def sf_decode_attn_scratch(desc, info, work_dev, q, k_pool, v_pool, block_table, out, lse=None, stream=None):
    """sf_decode_attn + sf_decode_attn_combine with the partials in the
    library's own device array (allocates nothing). work_dev: the plan,
    already on the device."""
    b, hq, hkv, d = desc.num_seqs, desc.num_q_heads, desc.num_kv_heads, desc.head_dim
    _dev(q, "q", torch.bfloat16, (b, hq, d))
    _dev(k_pool, "k_pool", torch.bfloat16, (desc.num_pages, hkv, d // 8, PAGE, 8))
    _dev(v_pool, "v_pool", torch.bfloat16, (desc.num_pages, hkv, d, PAGE))
    _dev(block_table, "block_table", torch.int32, (b, desc.block_table_stride))
    _dev(out, "out", torch.float32, (b, hq, d))
    _dev(work_dev, "work_dev", torch.int32)
    if work_dev.numel() * 4 < info.work_bytes:
        raise ValueError("work_dev is smaller than the plan")
    if lse is not None:
        _dev(lse, "lse", torch.float32, (b, hq))
    _check("sf_decode_attn_scratch", lib().sf_decode_attn_scratch(
        ctypes.byref(desc), ctypes.byref(info), _addr(work_dev), _addr(q), _addr(k_pool), _addr(v_pool),
        _addr(block_table), _addr(out), _addr(lse), _stream(stream)))


def kernel_event(ev, stream):
    """The hipEvent_t behind a torch timing event, for an entry point that
    records the kernel's own start or end time into it. torch creates an
    event on its first record, so a fresh one is recorded on `stream` once."""
    if ev.cuda_event == 0:
        ev.record(stream)
    return ev.cuda_event


def sf_debug_stream_read(buf, sink, blocks=16384, stream=None, events=None):
    """Reads every byte of the uint8 device tensor buf once (measurement
    support); sink: a uint8 device tensor of at least 16 bytes. events, if
    given, is a (start, end) pair of torch timing events that take the
    kernel's own start and end times."""
    _dev(buf, "buf", torch.uint8)
    _dev(sink, "sink", torch.uint8)
    if sink.numel() * sink.element_size() < 16:
        raise ValueError("sink must hold at least 16 bytes")
    s = stream or torch.cuda.current_stream(buf.device)
    ev = (None, None) if events is None else (kernel_event(events[0], s), kernel_event(events[1], s))
    _check("sf_debug_stream_read", lib().sf_debug_stream_read(
        _addr(buf), buf.numel() * buf.element_size(), _addr(sink), int(blocks), s.cuda_stream, *ev))


def sf_debug_gather_kv(desc, k_pool, v_pool, block_table, seq, kv_head, length, k_dense, v_dense,
                       stream=None):
    """Dense [length, D] bf16 copies of one (sequence, KV head) via the kernel's translation."""
    d = desc.head_dim
    _dev(k_pool, "k_pool", torch.bfloat16)
    _dev(v_pool, "v_pool", torch.bfloat16)
    _dev(block_table, "block_table", torch.int32)
    _dev(k_dense, "k_dense", torch.bfloat16, (length, d))
    _dev(v_dense, "v_dense", torch.bfloat16, (length, d))
    _check("sf_debug_gather_kv", lib().sf_debug_gather_kv(
        ctypes.byref(desc), _addr(k_pool), _addr(v_pool), _addr(block_table), int(seq),
        int(kv_head), int(length), _addr(k_dense), _addr(v_dense), _stream(stream)))


# ----------------------------------------------------------------------------
# convenience runner: owns the pinned work-list ring and the device buffers
# ----------------------------------------------------------------------------
class DecodeAttention:
    """Plan + attention + combine for successive decode steps, through the
    library's native runner (sf_runner_create / sf_runner_step): one call per
    step plans into the runner's pinned, device-mapped ring and launches the
    kernels, which read that work list in place, on the caller's stream. Tensor checks run once per
    distinct set of tensors (the last 64 sets are remembered)."""

    def __init__(self, num_q_heads, num_kv_heads, head_dim, device=None, num_cus=None,
                 opts: sf_plan_opts | None = None):
        self.hq, self.hkv, self.d = int(num_q_heads), int(num_kv_heads), int(head_dim)
        self.device = torch.device(device or "cuda")
        if num_cus is None:
            num_cus = torch.cuda.get_device_properties(self.device).multi_processor_count
        self.opts = opts if opts is not None else make_opts(num_cus=num_cus)
        if self.opts.num_cus == 0:
            self.opts.num_cus = num_cus
        self.L = lib()
        self._runners = {}
        self._info = sf_plan_info()
        self._extras = sf_runner_extras()
        self._checked = {}
        self._desc_key = None
        self._desc = None
        self.last_info = None
        self._lse = None
        self._host_checked = False   # set by a caller that checked its own host copy

    def _runner(self, chunk_pages):
        o = self.opts
        key = (o.num_cus, int(chunk_pages or 0), o.workers_per_cu, o.min_chunk_pages, o.xcd_parity_skew)
        r = self._runners.get(key)
        if r is None:
            opts = sf_plan_opts(*key)
            shape = make_desc(0, self.hq, self.hkv, self.d, 1, 0, 1.0)
            r = ctypes.c_void_p()
            with torch.cuda.device(self.device):
                _check("sf_runner_create", self.L.sf_runner_create(ctypes.byref(shape), ctypes.byref(opts),
                                                                   ctypes.byref(r)))
            self._runners[key] = r
        return r

    def _check_tensors(self, q, k_pool, v_pool, block_table, out, lse, fp8=None):
        key = (q.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), block_table.data_ptr(),
               out.data_ptr(), None if lse is None else lse.data_ptr(), tuple(q.shape),
               tuple(k_pool.shape), tuple(v_pool.shape), tuple(block_table.shape),
               None if fp8 is None else (fp8[0].data_ptr(), fp8[1].data_ptr()))
        if key in self._checked:
            return
        b, hkv, d = q.shape[0], self.hkv, self.d
        _dev(q, "q", torch.bfloat16, (b, self.hq, d))
        if fp8 is None:
            _dev(k_pool, "k_pool", torch.bfloat16, (k_pool.shape[0], hkv, d // 8, PAGE, 8))
            _dev(v_pool, "v_pool", torch.bfloat16, (k_pool.shape[0], hkv, d, PAGE))
        else:
            _dev(k_pool, "k_pool8", torch.uint8, (k_pool.shape[0], hkv, PAGE * d))
            _dev(v_pool, "v_pool8", torch.uint8, (k_pool.shape[0], hkv, PAGE * d))
            _dev(fp8[0], "k_scale", torch.float32, (k_pool.shape[0], hkv))
            _dev(fp8[1], "v_scale", torch.float32, (k_pool.shape[0], hkv))
        _dev(block_table, "block_table", torch.int32, (b, block_table.shape[1]))
        _dev(out, "out", torch.float32, (b, self.hq, d))
        if lse is not None:
            _dev(lse, "lse", torch.float32, (b, self.hq))
        if len(self._checked) >= 64:      # a few tensor sets in rotation stay checked
            self._checked.clear()
        self._checked[key] = True

    def reserve(self, seq_lens, num_pages, block_table_stride, chunk_pages=None, fp8=False, stream=None):
        """Sizes the native runner's workspace and work-list ring for a step
        over seq_lens (the largest batch to come) ahead of the steps, so no
        step stalls to grow them (sf_runner_reserve)."""
        lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
        desc = make_desc(lens.size, self.hq, self.hkv, self.d, block_table_stride, num_pages, 1.0)
        o = self.opts
        wpc = o.workers_per_cu or (8 if fp8 else 0)
        opts = sf_plan_opts(o.num_cus, int(chunk_pages or 0), wpc, o.min_chunk_pages, o.xcd_parity_skew)
        info = sf_plan_info()
        st = self.L.sf_decode_attn_plan(ctypes.byref(desc), lens.ctypes.data, ctypes.byref(opts), None, 0,
                                        ctypes.byref(info))
        _check("sf_decode_attn_plan", st)
        main = stream or torch.cuda.current_stream(self.device)
        with torch.cuda.device(self.device):
            _check("sf_runner_reserve", self.L.sf_runner_reserve(self._runner(chunk_pages), info.workspace_bytes,
                                                                 info.work_bytes, lens.size, main.cuda_stream))

    def __call__(self, q, k_pool, v_pool, block_table, seq_lens, scale, out=None, lse=None,
                 chunk_pages=None, stream: torch.cuda.Stream | None = None, attn_events=None,
                 append=None, fp8=None):
        """One decode step on `stream` (default: the current stream). attn_events,
        if given, is a (start, end) pair of torch timing events that take the
        attention kernel's own start and end times (none if the step launches
        no attention kernel). append = (k_new, v_new, new_pages) makes it an
        append-then-attend step: k_new, v_new are device bf16 [B, Hkv, D] and
        new_pages a host int32 [B] array (-1 = the token's page is already
        held), uploaded together with the work list. fp8 = (k_scale, v_scale)
        makes k_pool / v_pool an fp8 cache (uint8 E4M3 codes [N, Hkv, 16*D],
        fp32 scales [N, Hkv]); it cannot be combined with append."""
        if fp8 is not None and append is not None:
            raise ValueError("the fp8 cache has no appending step")
        b = q.shape[0]
        main = stream or torch.cuda.current_stream(self.device)
        if out is None:
            out = torch.empty((b, self.hq, self.d), dtype=torch.float32, device=self.device)
        self._check_tensors(q, k_pool, v_pool, block_table, out, lse, fp8)
        dkey = (b, block_table.shape[1], k_pool.shape[0], float(scale))
        if dkey != self._desc_key:
            self._desc = make_desc(b, self.hq, self.hkv, self.d, block_table.shape[1], k_pool.shape[0], scale)
            self._desc_key = dkey
        if isinstance(seq_lens, torch.Tensor):
            seq_lens = seq_lens.cpu().numpy()
        lens = seq_lens if (isinstance(seq_lens, np.ndarray) and seq_lens.dtype == np.int32
                            and seq_lens.flags.c_contiguous) else np.ascontiguousarray(seq_lens, np.int32)
        if lens.shape != (b,):
            raise ValueError("seq_lens must have one entry per sequence")
        ex = self._extras
        ex.k_new = ex.v_new = ex.new_pages_host = ex.k_scale = ex.v_scale = ex.attn_start = ex.attn_end = None
        pages = None
        if append is not None:
            k_new, v_new, new_pages = append
            _dev(k_new, "k_new", torch.bfloat16, (b, self.hkv, self.d))
            _dev(v_new, "v_new", torch.bfloat16, (b, self.hkv, self.d))
            pages = np.ascontiguousarray(new_pages, dtype=np.int32)
            if pages.shape != (b,):
                raise ValueError("new_pages must have one entry per sequence")
            ex.k_new, ex.v_new, ex.new_pages_host = k_new.data_ptr(), v_new.data_ptr(), pages.ctypes.data
            if lse is None:  # the merge reads lse back: keep one of our own
                if self._lse is None or self._lse.numel() < b * self.hq:
                    self._lse = torch.empty(b * self.hq * 5 // 4 + 64, dtype=torch.float32, device=self.device)
                lse = self._lse[: b * self.hq].view(b, self.hq)
        if fp8 is not None:
            ex.k_scale, ex.v_scale = fp8[0].data_ptr(), fp8[1].data_ptr()
        if DEBUG_CHECKS and not self._host_checked:
            # an appending step reads the pool for its L - 1 cached tokens only
            # (the newest token's page may still be -1: the step writes it)
            check_block_table(self._desc, block_table, lens - 1 if append is not None else lens)
            if pages is not None and np.any((pages < -1) | (pages >= k_pool.shape[0])):
                raise ValueError("new_pages holds a page id outside the pool")
        self._host_checked = False
        if attn_events is not None:
            ex.attn_start = kernel_event(attn_events[0], main)
            ex.attn_end = kernel_event(attn_events[1], main)
        info = self._info
        _check("sf_runner_step", self.L.sf_runner_step(
            self._runner(chunk_pages), ctypes.byref(self._desc), lens.ctypes.data, q.data_ptr(), k_pool.data_ptr(),
            v_pool.data_ptr(), block_table.data_ptr(), out.data_ptr(), None if lse is None else lse.data_ptr(),
            ctypes.byref(ex), main.cuda_stream, ctypes.byref(info)))
        self.last_info = sf_plan_info.from_buffer_copy(info)
        return out

    def __del__(self):
        L = getattr(self, "L", None)
        for r in getattr(self, "_runners", {}).values():
            if L is not None and r.value:
                L.sf_runner_destroy(r)
        self._runners = {}


class PageTable:
    """Host bookkeeping of a growing paged cache: the page pool and a host copy
    of the block table.

    Each decode step generates one token per running trajectory (App. B.1).
    advance(lens) moves to the next step's lengths (0 for a sequence that has
    left) and
      1. returns to the pool every page of the sequences that have left since
         the previous step (ascending sequence order, each in block-table order);
      2. if appending, takes one page for every newest token that opens a page
         (index L - 1 a multiple of 16), in ascending sequence order, and
         records it in the host block table.
    It returns the int32 [B] new-page array the append kernel takes (-1 where
    the token lands in a page the sequence already holds).
    """

    def __init__(self, num_pages, bt_host, lens0):
        self.bt = np.array(bt_host, dtype=np.int32, order="C", copy=True)
        lens0 = np.asarray(lens0, dtype=np.int64)
        self.pool = PagePool(num_pages)
        npg = (lens0 + PAGE - 1) // PAGE
        held = [self.bt[s, : npg[s]] for s in range(lens0.size)]
        self.pool.claim(np.concatenate(held) if held else np.zeros(0, np.int32))
        self.prev = np.ascontiguousarray(lens0, dtype=np.int32)
        self.new_pages = np.empty(lens0.size, dtype=np.int32)

    def advance(self, lens, appending=True) -> np.ndarray:
        """The library's sf_page_table_step on the host table; returns new_pages."""
        lens = np.ascontiguousarray(lens, dtype=np.int32)
        if lens.shape != self.prev.shape:
            raise ValueError("lens must have one entry per sequence")
        _check("sf_page_table_step", self.pool._L.sf_page_table_step(
            self.pool._p, self.bt.ctypes.data, self.bt.shape[1], lens.size, self.prev.ctypes.data,
            lens.ctypes.data, int(bool(appending)), self.new_pages.ctypes.data))
        self.prev = lens
        return self.new_pages


class DecodeLoopRunner:
    """Multi-step decode over a growing paged cache: per step, PageTable
    bookkeeping on the host, then append-then-attend and the merge of split
    sequences on the GPU. The first step (the prompt) only attends.
    block_table is the device table the kernels read and extend."""

    def __init__(self, num_q_heads, num_kv_heads, head_dim, k_pool, v_pool, block_table, bt_host, lens0,
                 scale, device=None, num_cus=None, attn=None):
        """attn: an existing DecodeAttention of the same head geometry to reuse
        (its native runner keeps its pinned ring and workspace across loops)."""
        if attn is not None and (attn.hq, attn.hkv, attn.d) != (int(num_q_heads), int(num_kv_heads), int(head_dim)):
            raise ValueError("attn was made for another head geometry")
        self.attn = attn or DecodeAttention(num_q_heads, num_kv_heads, head_dim, device=device, num_cus=num_cus)
        self.k_pool, self.v_pool, self.block_table, self.scale = k_pool, v_pool, block_table, float(scale)
        self.table = PageTable(k_pool.shape[0], bt_host, lens0)
        self.steps = 0

    @property
    def bt_host(self):
        return self.table.bt

    @property
    def pool(self):
        return self.table.pool

    def step(self, q, lens, k_new=None, v_new=None, out=None, lse=None, stream=None, attn_events=None):
        lens = np.asarray(lens, dtype=np.int64)
        appending = self.steps > 0
        if appending and (k_new is None or v_new is None):
            raise ValueError("every step after the first appends a token: pass k_new and v_new")
        new_pages = self.table.advance(lens, appending)
        if DEBUG_CHECKS:
            desc = make_desc(lens.size, self.attn.hq, self.attn.hkv, self.attn.d, self.table.bt.shape[1],
                             self.k_pool.shape[0], self.scale)
            check_block_table(desc, self.table.bt, lens)
            self.attn._host_checked = True
        append = (k_new, v_new, new_pages) if appending else None
        out = self.attn(q, self.k_pool, self.v_pool, self.block_table, lens.astype(np.int32), self.scale,
                        out=out, lse=lse, stream=stream, attn_events=attn_events, append=append)
        self.steps += 1
        return out
