"""The C-ABI library loads and exports every function include/tre.h
declares (no compute calls: this runs without a GPU)."""
import ctypes
import os
import re

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tre.h")
LIB = os.path.join(ROOT, "paper_2609_29160_amd", "libtre.so")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tre_[a-z_]+)\s*\(", src)))


def _lib():
    if not os.path.exists(LIB):
        from paper_2609_29160_amd.build import build_library
        build_library()
    return ctypes.CDLL(LIB)


def test_library_exports_every_declared_function():
    L = _lib()
    names = _declared()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), f"{n} declared in tre.h but not exported"


def test_binding_covers_the_header():
    from paper_2609_29160_amd import tre
    assert sorted(tre.EXPORTS) == _declared()


def test_struct_layouts():
    from paper_2609_29160_amd import tre
    assert tre.PROFILE_DTYPE.itemsize == 56
    assert tre.SCENARIO_DTYPE.itemsize == 24
    assert tre.MOVE_DTYPE.itemsize == 8
    assert ctypes.sizeof(tre._TraceCfg) == 40
    assert ctypes.sizeof(tre._CtlOut) == 40
    assert ctypes.sizeof(tre._TssOut) == 56
    assert ctypes.sizeof(tre._Actuation) == 32
    assert tre.SLO_DTYPE.itemsize == 40 and tre.FIT_DTYPE.itemsize == 32
    assert tre.REQ_LATENCY_DTYPE.itemsize == 24
    assert tre.SERVICE_DTYPE.itemsize == 8 and tre.LOOP_STATS_DTYPE.itemsize == 32
    assert ctypes.sizeof(tre._LoopRequests) == 6 * 8 + 9 * 4 + 4  # padded to 8


def test_error_message_without_gpu_call():
    L = _lib()
    L.tre_last_error.restype = ctypes.c_char_p
    L.tre_events_info.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    assert L.tre_events_info(None, None) == 1
    assert b"NULL" in L.tre_last_error()
