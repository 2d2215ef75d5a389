"""Thin ctypes binding of ``libmfsgd.so`` (C ABI in ``include/mfsgd.h``).

Argument marshalling only: every step of the computation runs in the HIP
kernels of the library.  Device arrays are torch tensors on the current GPU;
streams are torch streams (default: ``torch.cuda.current_stream()``).

Samples are int32 tensors of shape (nnz, 3) whose columns hold u, v and the
bit pattern of the float32 rating r -- exactly the packed 12-byte records the
library reads.  ``samples_to_device`` builds one from a numpy structured array.

The library is loaded on first use.  If it has not been built the binding
raises ``ImportError``: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch  # loads the HIP runtime that the library then shares (same SONAME)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmfsgd.so")

OK, EINVAL, ENOMEM, EHIP, ESTATE, ETIMEOUT, ENUMERIC = 0, -1, -2, -3, -4, -5, -6
BATCH_HOGWILD, WAVEFRONT, WAVEFRONT_DET, GLOBAL_TABLE = 0, 1, 2, 3
FP32, FP16 = 0, 1
DBG_VISITS, DBG_TRACE, DBG_PLAN_STARTS, DBG_PLAN_ORDER, DBG_TEAM_MAP, DBG_TEAM_SIZES = 1, 2, 3, 4, 5, 6
DBG_TABLE_STARTS, DBG_TABLE_ORDER, DBG_PRIORITY = 7, 8, 9

SCHEMES = {"hogwild": BATCH_HOGWILD, "wavefront": WAVEFRONT, "wavefront_det": WAVEFRONT_DET,
           "table": GLOBAL_TABLE}

SAMPLE_DTYPE = np.dtype([("u", "<i4"), ("v", "<i4"), ("r", "<f4")])


class MfsgdError(RuntimeError):
    def __init__(self, code: int, fn: str, msg: str):
        super().__init__(f"{fn} failed with status {code}: {msg}")
        self.code = code


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "(hipcc for gfx950); there is no CPU fallback")
        L = C.CDLL(LIB_PATH)
        i32, i64, u64, f32, vp = C.c_int32, C.c_int64, C.c_uint64, C.c_float, C.c_void_p
        sig = {
            "mfsgd_set_option": ([C.c_char_p, i64], C.c_int),
            "mfsgd_get_option": ([C.c_char_p, C.POINTER(i64)], C.c_int),
            "mfsgd_reset_options": ([], C.c_int),
            "mfsgd_init": ([i64, i64, i32, u64], C.c_int),
            "mfsgd_plan": ([vp, i64, i32, vp], C.c_int),
            "mfsgd_epoch": ([vp, i64, f32, f32, f32, i32, vp], C.c_int),
            "mfsgd_epoch_staged": ([vp, i64, f32, f32, f32, vp], C.c_int),
            "mfsgd_rmse": ([vp, i64, C.POINTER(C.c_double), vp], C.c_int),
            "mfsgd_rmse_noalloc": ([vp, i64, vp, vp], C.c_int),
            "mfsgd_check_samples": ([vp, i64, vp], C.c_int),
            "mfsgd_sync": ([vp], C.c_int),
            "mfsgd_get_factors": ([vp, vp, vp], C.c_int),
            "mfsgd_set_factors": ([vp, vp, vp], C.c_int),
            "mfsgd_set_epoch": ([i64], C.c_int),
            "mfsgd_get_epoch": ([], i64),
            "mfsgd_debug_read": ([i32, vp, i64, vp], C.c_int),
            "mfsgd_finalize": ([], C.c_int),
            "mfsgd_last_error": ([], C.c_char_p),
            "mfsgd_version": ([], C.c_char_p),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(rc: int, fn: str) -> int:
    if rc != OK:
        raise MfsgdError(rc, fn, lib().mfsgd_last_error().decode())
    return rc


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _samples_ptr(t: torch.Tensor):
    if t.dtype != torch.int32 or t.dim() != 2 or t.shape[1] != 3 or not t.is_contiguous() or not t.is_cuda:
        raise TypeError("samples must be a contiguous int32 cuda tensor of shape (nnz, 3)")
    return C.c_void_p(t.data_ptr() if t.numel() else 0), t.shape[0]


def samples_to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    """numpy structured (u, v, r) records -> int32 (nnz, 3) device tensor."""
    a = np.ascontiguousarray(a)
    assert a.dtype == SAMPLE_DTYPE
    t = torch.from_numpy(a.view(np.int32).reshape(-1, 3).copy())
    return t.to(device)


def version() -> str:
    return lib().mfsgd_version().decode()


def set_option(key: str, value: int) -> None:
    _check(lib().mfsgd_set_option(key.encode(), int(value)), "mfsgd_set_option")


def get_option(key: str) -> int:
    v = C.c_int64()
    _check(lib().mfsgd_get_option(key.encode(), C.byref(v)), "mfsgd_get_option")
    return v.value


def reset_options() -> None:
    """Every option back to its default."""
    _check(lib().mfsgd_reset_options(), "mfsgd_reset_options")


def init(m: int, n: int, k: int, seed: int) -> None:
    _check(lib().mfsgd_init(m, n, k, seed), "mfsgd_init")


def plan(samples: torch.Tensor, s: int, stream=None) -> None:
    p, nnz = _samples_ptr(samples)
    _check(lib().mfsgd_plan(p, nnz, s, _stream(stream)), "mfsgd_plan")


def epoch(samples: torch.Tensor, lr: float, lambda_p: float, lambda_q: float, scheme="hogwild",
          stream=None) -> None:
    p, nnz = _samples_ptr(samples)
    sc = SCHEMES[scheme] if isinstance(scheme, str) else int(scheme)
    _check(lib().mfsgd_epoch(p, nnz, lr, lambda_p, lambda_q, sc, _stream(stream)), "mfsgd_epoch")


def epoch_staged(samples, lr: float, lambda_p: float, lambda_q: float, stream=None) -> None:
    """mfsgd_epoch_staged on host samples: a numpy (u, v, r) record array or
    an int32 (nnz, 3) CPU tensor (pinned or not).  A pinned array must stay
    alive and unchanged until the work on `stream` completes."""
    if isinstance(samples, np.ndarray):
        if samples.dtype != SAMPLE_DTYPE or not samples.flags["C_CONTIGUOUS"]:
            raise TypeError("samples must be a C-contiguous array of (u, v, r) records")
        p, nnz = C.c_void_p(samples.ctypes.data if samples.size else 0), samples.shape[0]
    else:
        t = samples
        if t.dtype != torch.int32 or t.dim() != 2 or t.shape[1] != 3 or not t.is_contiguous() or t.is_cuda:
            raise TypeError("samples must be a contiguous int32 CPU tensor of shape (nnz, 3)")
        p, nnz = C.c_void_p(t.data_ptr() if t.numel() else 0), t.shape[0]
    _check(lib().mfsgd_epoch_staged(p, nnz, lr, lambda_p, lambda_q, _stream(stream)), "mfsgd_epoch_staged")


def rmse(test: torch.Tensor, stream=None) -> float:
    p, n = _samples_ptr(test)
    out = C.c_double()
    _check(lib().mfsgd_rmse(p, n, C.byref(out), _stream(stream)), "mfsgd_rmse")
    return out.value


def rmse_noalloc(test: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """Enqueue the test RMSE into out[0] (a float64 device tensor) without
    allocating or waiting (mfsgd_rmse_noalloc)."""
    if out.dtype != torch.float64 or not out.is_cuda or out.numel() < 1:
        raise ValueError("out must be a float64 device tensor with at least one element")
    p, n = _samples_ptr(test)
    _check(lib().mfsgd_rmse_noalloc(p, n, C.c_void_p(out.data_ptr()), _stream(stream)), "mfsgd_rmse_noalloc")


def check_samples(samples: torch.Tensor, stream=None) -> None:
    p, nnz = _samples_ptr(samples)
    _check(lib().mfsgd_check_samples(p, nnz, _stream(stream)), "mfsgd_check_samples")


def sync(stream=None) -> None:
    _check(lib().mfsgd_sync(_stream(stream)), "mfsgd_sync")


def _storage_dtype():
    return torch.float16 if get_option("dtype") == FP16 else torch.float32


def get_factors(m: int, n: int, k: int, dtype=None, device="cuda", stream=None):
    """(P, Q) copies, shapes (m, k) and (n, k), storage dtype of the model."""
    dtype = dtype or _storage_dtype()
    P = torch.empty((m, k), dtype=dtype, device=device)
    Q = torch.empty((n, k), dtype=dtype, device=device)
    _check(lib().mfsgd_get_factors(C.c_void_p(P.data_ptr()), C.c_void_p(Q.data_ptr()), _stream(stream)),
           "mfsgd_get_factors")
    return P, Q


def set_factors(P: torch.Tensor, Q: torch.Tensor, stream=None) -> None:
    P = P.contiguous()
    Q = Q.contiguous()
    _check(lib().mfsgd_set_factors(C.c_void_p(P.data_ptr()), C.c_void_p(Q.data_ptr()), _stream(stream)),
           "mfsgd_set_factors")


def set_epoch(t: int) -> None:
    _check(lib().mfsgd_set_epoch(t), "mfsgd_set_epoch")


def get_epoch() -> int:
    return lib().mfsgd_get_epoch()


def debug_visits(nnz: int, stream=None) -> torch.Tensor:
    out = torch.empty(nnz, dtype=torch.int32, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_VISITS, C.c_void_p(out.data_ptr()), nnz, _stream(stream)), "mfsgd_debug_read")
    return out


def debug_trace(count: int, stream=None) -> torch.Tensor:
    out = torch.empty(count, dtype=torch.int32, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_TRACE, C.c_void_p(out.data_ptr()), count, _stream(stream)),
           "mfsgd_debug_read")
    return out


def debug_plan_starts(s: int, stream=None) -> torch.Tensor:
    out = torch.empty(s * s + 1, dtype=torch.int64, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_PLAN_STARTS, C.c_void_p(out.data_ptr()), s * s + 1, _stream(stream)),
           "mfsgd_debug_read")
    return out


def debug_plan_order(nnz: int, stream=None) -> torch.Tensor:
    out = torch.empty(max(nnz, 1), dtype=torch.int64, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_PLAN_ORDER, C.c_void_p(out.data_ptr()), nnz, _stream(stream)),
           "mfsgd_debug_read")
    return out[:nnz]


def debug_table_starts(s: int, stream=None) -> torch.Tensor:
    out = torch.empty(s * s + 1, dtype=torch.int64, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_TABLE_STARTS, C.c_void_p(out.data_ptr()), s * s + 1, _stream(stream)),
           "mfsgd_debug_read")
    return out


def debug_table_order(nnz: int, stream=None) -> torch.Tensor:
    out = torch.empty(max(nnz, 1), dtype=torch.int64, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_TABLE_ORDER, C.c_void_p(out.data_ptr()), nnz, _stream(stream)),
           "mfsgd_debug_read")
    return out[:nnz]


def debug_team_layout(s: int, stream=None):
    """(map, sizes) of the last block-scheduled epoch: per (XCD x, arrival
    slot j) at x * (len(map) / xcds) + j -- or per workgroup for one-wavefront
    teams -- team << 16 | member (-1 idle), per team its workgroup count."""
    grid = get_option("teams_grid")
    tmap = torch.empty(max(grid, 1), dtype=torch.int32, device="cuda")
    sizes = torch.empty(s, dtype=torch.int32, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_TEAM_MAP, C.c_void_p(tmap.data_ptr()), grid, _stream(stream)),
           "mfsgd_debug_read")
    _check(lib().mfsgd_debug_read(DBG_TEAM_SIZES, C.c_void_p(sizes.data_ptr()), s, _stream(stream)),
           "mfsgd_debug_read")
    return tmap[:grid], sizes


def debug_priority(s: int, stream=None):
    """Critical-path weight of every (team, wave) block of the last pooled
    block-scheduled epoch: uint32 tensor of s*s, entry t*s + w."""
    out = torch.empty(s * s, dtype=torch.int32, device="cuda")
    _check(lib().mfsgd_debug_read(DBG_PRIORITY, C.c_void_p(out.data_ptr()), s * s, _stream(stream)),
           "mfsgd_debug_read")
    return out


def finalize() -> None:
    _check(lib().mfsgd_finalize(), "mfsgd_finalize")
