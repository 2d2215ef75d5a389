"""The C-ABI library builds, loads and exports every entry point that
include/mfsgd.h declares (no compute call: this runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mfsgd.h")
LIB = os.path.join(ROOT, "paper_1610_05838_amd", "libmfsgd.so")


def declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|int64_t|const char\s*\*)\s*(mfsgd_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def libpath():
    if not os.path.exists(LIB):
        from paper_1610_05838_amd import _build
        _build.build()
    return LIB


def test_header_declares_the_boundary():
    names = declared()
    for must in ("mfsgd_init", "mfsgd_epoch", "mfsgd_rmse", "mfsgd_plan", "mfsgd_get_factors",
                 "mfsgd_set_factors", "mfsgd_finalize", "mfsgd_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol(libpath):
    lib = ctypes.CDLL(libpath)
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_exports_are_c_symbols(libpath):
    """extern "C": the exported names are not C++-mangled."""
    out = os.popen(f"nm -D --defined-only {libpath}").read()
    for n in declared():
        assert re.search(rf"\b{n}\b", out), n


def test_options_without_gpu(libpath):
    """Option handling is pure host logic."""
    lib = ctypes.CDLL(libpath)
    lib.mfsgd_set_option.argtypes = [ctypes.c_char_p, ctypes.c_int64]
    lib.mfsgd_get_option.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64)]
    lib.mfsgd_last_error.restype = ctypes.c_char_p
    v = ctypes.c_int64()
    assert lib.mfsgd_get_option(b"batch_f", ctypes.byref(v)) == 0 and v.value == 256
    assert lib.mfsgd_set_option(b"batch_f", 100) == -1  # not a multiple of 64
    assert b"multiple of 64" in lib.mfsgd_last_error()
    assert lib.mfsgd_set_option(b"depth", 3) == -1
    assert lib.mfsgd_set_option(b"no_such_key", 1) == -1
    assert lib.mfsgd_set_option(b"depth", 8) == 0
    assert lib.mfsgd_get_option(b"depth", ctypes.byref(v)) == 0 and v.value == 8
    assert lib.mfsgd_set_option(b"depth", 4) == 0
    assert lib.mfsgd_get_option(b"table_grid", ctypes.byref(v)) == 0 and v.value == 256
    assert lib.mfsgd_set_option(b"table_grid", 1025) == -1 and lib.mfsgd_set_option(b"table_grid", 0) == -1
    assert lib.mfsgd_get_option(b"table_workers", ctypes.byref(v)) == 0 and v.value == 0
    assert lib.mfsgd_set_option(b"table_workers", -1) == -1
    assert lib.mfsgd_get_option(b"half_waves", ctypes.byref(v)) == 0 and v.value == 1
    assert lib.mfsgd_set_option(b"half_waves", 3) == -1
    assert lib.mfsgd_get_option(b"table_blocks", ctypes.byref(v)) == -4  # read-only, needs init
    lib.mfsgd_get_epoch.restype = ctypes.c_int64
    assert lib.mfsgd_get_epoch() == -1  # not initialised


def test_read_only_keys_without_gpu(libpath):
    """Every read-only key the header lists is known to the library: before
    mfsgd_init reading one is a state error (not an unknown key), and none can
    be set."""
    src = open(HEADER).read()
    block = src[src.index("Read-only keys"):src.index("int mfsgd_set_option")]
    keys = sorted(set(re.findall(r'"([a-z_0-9]+)"', block)))
    assert {"resident_waves", "xcds", "blocked_pairs", "half_workers", "teams_grid"} <= set(keys)
    lib = ctypes.CDLL(libpath)
    lib.mfsgd_set_option.argtypes = [ctypes.c_char_p, ctypes.c_int64]
    lib.mfsgd_get_option.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64)]
    v = ctypes.c_int64()
    read_only = []
    for k in keys:
        rc = lib.mfsgd_get_option(k.encode(), ctypes.byref(v))
        if rc == 0:  # a settable option that the text mentions
            continue
        assert rc == -4, k                                   # MFSGD_ESTATE, not MFSGD_EINVAL
        assert lib.mfsgd_set_option(k.encode(), 1) == -1, k  # MFSGD_EINVAL
        read_only.append(k)
    assert {"resident_waves", "xcds", "xcd_round_robin", "cus", "partitioned", "hogwild_form", "hogwild_atomic",
            "half_workers", "blocked_pairs", "table_blocks", "blocked_per_cu", "teams_grid"} <= set(read_only)
