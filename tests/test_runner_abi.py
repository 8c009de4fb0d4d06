"""The native runner's C ABI on the CPU: struct sizes shared with the ctypes
binding, and the argument checks that return before any device call."""
import ctypes

import pytest

from paper_2601_12784_amd import binding as B


def test_struct_sizes_match_the_header():
    assert ctypes.sizeof(B.sf_runner_extras) == 56
    assert ctypes.sizeof(B.sf_extend_info) == 32
    assert ctypes.sizeof(B.sf_plan_info) == 48


def test_runner_rejects_bad_arguments_without_a_device():
    L = B.lib()
    r = ctypes.c_void_p()
    assert L.sf_runner_create(None, None, ctypes.byref(r)) == 1
    bad = B.make_desc(0, 6, 4, 128, 1, 0, 1.0)              # Hq % Hkv != 0
    assert L.sf_runner_create(ctypes.byref(bad), None, ctypes.byref(r)) == 1
    odd = B.make_desc(0, 4, 1, 96, 1, 0, 1.0)               # head_dim 96 is not built
    assert L.sf_runner_create(ctypes.byref(odd), None, ctypes.byref(r)) == 2
    opts = B.sf_plan_opts(0, 0, 0, 0, -251)                  # parity skew below -250
    good = B.make_desc(0, 4, 1, 128, 1, 0, 1.0)
    assert L.sf_runner_create(ctypes.byref(good), ctypes.byref(opts), ctypes.byref(r)) == 1
    desc = B.make_desc(1, 4, 1, 128, 1, 1, 1.0)
    assert L.sf_runner_step(None, ctypes.byref(desc), None, None, None, None, None, None, None, None, None,
                            None) == 1
    assert L.sf_runner_reserve(None, 0, 0, 0, None) == 1
    L.sf_runner_destroy(None)                                # a NULL runner is a no-op


@pytest.mark.skipif(B.torch.cuda.is_available(), reason="only meaningful without a GPU")
def test_runner_create_reports_the_missing_device():
    L = B.lib()
    r = ctypes.c_void_p()
    good = B.make_desc(0, 4, 1, 128, 1, 0, 1.0)
    assert L.sf_runner_create(ctypes.byref(good), None, ctypes.byref(r)) in (0, 5)
    if r.value:
        L.sf_runner_destroy(r)
