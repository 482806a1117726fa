"""The C-ABI library on the CPU: it loads, exports every symbol include/sj.h
declares, and its host-side argument handling works without a GPU."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sj.h")
LIB = os.path.join(ROOT, "paper_2006_12608_amd", "libsj.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sj_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("sj_create", "sj_join_ip", "sj_join_l2", "sj_count", "sj_destroy"):
        assert want in names


def test_library_exports_every_declared_symbol():
    assert os.path.exists(LIB), "libsj.so not built"
    lib = ctypes.CDLL(LIB)
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (sj_\w+)", out))
    assert set(declared_functions()) <= exported


def test_binding_exposes_the_c_names():
    import paper_2006_12608_amd as sj
    for name in declared_functions():
        assert hasattr(sj, name), name


def test_null_context_and_arguments_are_rejected():
    import paper_2006_12608_amd as sj
    st, n = sj.sj_join_ip(None, sj.SJ_F16, None, 0, None, 0, 0, 0.0, None, 0)
    assert st == sj.SJ_E_INVAL and n == 0
    assert "context" in sj.sj_last_error()
    st, n = sj.sj_join_l2(None, sj.SJ_I8, None, 0, None, 0, 0, 0.0, None, 0)
    assert st == sj.SJ_E_INVAL
    st, n = sj.sj_count(None, sj.SJ_IP, sj.SJ_BF16, None, 0, None, 0, 0, 0.0)
    assert st == sj.SJ_E_INVAL
    sj.sj_destroy(None)     # NULL-safe
    st = sj.lib.sj_join_ip(None, 1, None, 0, None, 0, 0, 0.0, None, 0, None, 0)
    assert st == sj.SJ_E_INVAL


def test_stats_reject_null():
    import paper_2006_12608_amd as sj
    assert sj.lib.sj_get_stats(None, None) == sj.SJ_E_INVAL


def test_create_without_gpu_fails_cleanly():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    import paper_2006_12608_amd as sj
    h = ctypes.c_void_p()
    st = sj.lib.sj_create(ctypes.byref(h), 0, None)
    assert st in (sj.SJ_E_HIP, sj.SJ_E_INVAL)
    assert h.value is None
    assert sj.sj_last_error()
