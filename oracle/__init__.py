"""CPU oracle for SGD matrix factorisation (arXiv 1610.05838) -- TEST INFRASTRUCTURE.

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``mfsgd_oracle.c`` (plain C,
binary64 arithmetic) through ctypes and shares no code with the GPU library.

Arrays are numpy arrays:
  samples : structured array with fields u (int32), v (int32), r (float32)
  P, Qt   : float32 or float16 arrays of shape (m, k) and (n, k)
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mfsgd_oracle.c")
LIB = os.path.join(HERE, "libmfsgd_oracle.so")

SAMPLE_DTYPE = np.dtype([("u", "<i4"), ("v", "<i4"), ("r", "<f4")])
F32, F16 = 0, 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no FMA contraction, OpenMP for the
    timing-only Hogwild! variant)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
             "-shared", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        i32, i64, u64, f32, f64, vp = C.c_int32, C.c_int64, C.c_uint64, C.c_float, C.c_double, C.c_void_p
        L.orc_half_to_double.argtypes = [C.c_uint16]
        L.orc_half_to_double.restype = f64
        L.orc_double_to_half.argtypes = [f64]
        L.orc_double_to_half.restype = C.c_uint16
        L.orc_splitmix64.argtypes = [u64, u64]
        L.orc_splitmix64.restype = u64
        L.orc_init_factors.argtypes = [i64, i64, i32, u64, C.c_int, vp, vp]
        L.orc_init_factors.restype = None
        L.orc_init_rows.argtypes = [i64, i32, u64, C.c_int, C.c_int, vp, i64, vp]
        L.orc_init_rows.restype = None
        L.orc_sgd_step.argtypes = [vp, vp, i32, f64, f64, f64, f64]
        L.orc_sgd_step.restype = None
        L.orc_epoch_serial.argtypes = [i32, C.c_int, vp, vp, vp, i64, f32, f32, f32]
        L.orc_epoch_serial.restype = C.c_int
        L.orc_hogwild_batch_owner.argtypes = [i64, i32, i64, vp]
        L.orc_hogwild_batch_owner.restype = None
        L.orc_row_block.argtypes = [i64, i64, i32]
        L.orc_row_block.restype = i32
        L.orc_col_block.argtypes = [i64, i64, i32]
        L.orc_col_block.restype = i32
        L.orc_fisher_yates.argtypes = [u64, i32, vp]
        L.orc_fisher_yates.restype = None
        L.orc_wavefront_sigma.argtypes = [u64, i64, i32, vp]
        L.orc_wavefront_sigma.restype = C.c_int
        L.orc_balanced_bounds.argtypes = [vp, i64, i64, C.c_int, i32, vp]
        L.orc_balanced_bounds.restype = C.c_int
        L.orc_bounded_block.argtypes = [i64, vp, i32]
        L.orc_bounded_block.restype = i32
        L.orc_block_order.argtypes = [vp, i64, i64, i64, i32, vp, vp, vp, vp]
        L.orc_block_order.restype = C.c_int
        L.orc_epoch_wavefront.argtypes = [i64, i64, i32, C.c_int, vp, vp, vp, i64, f32, f32, f32, i32, u64,
                                          i64, C.c_int]
        L.orc_epoch_wavefront.restype = C.c_int
        L.orc_table_order.argtypes = [u64, i64, vp, i64, vp]
        L.orc_table_order.restype = C.c_int
        L.orc_epoch_table.argtypes = [i64, i64, i32, C.c_int, vp, vp, vp, i64, f32, f32, f32, i32, u64, i64]
        L.orc_epoch_table.restype = C.c_int
        L.orc_rmse.argtypes = [i32, C.c_int, vp, vp, vp, i64]
        L.orc_rmse.restype = f64
        L.orc_sq_errors.argtypes = [i32, C.c_int, vp, vp, vp, i64, vp]
        L.orc_sq_errors.restype = None
        L.orc_objective.argtypes = [i32, C.c_int, vp, vp, vp, i64, f64, f64]
        L.orc_objective.restype = f64
        L.orc_epoch_hogwild_omp.argtypes = [i32, C.c_int, vp, vp, vp, i64, f32, f32, f32, i32, i32]
        L.orc_epoch_hogwild_omp.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float16:
        return F16
    raise TypeError(f"feature storage must be float32 or float16, got {a.dtype}")


def _samples(S) -> np.ndarray:
    S = np.ascontiguousarray(S)
    if S.dtype != SAMPLE_DTYPE:
        raise TypeError("samples must use oracle.SAMPLE_DTYPE")
    return S


# --- scalar helpers ---------------------------------------------------------------------------
def half_to_double(bits: int) -> float:
    return lib().orc_half_to_double(bits)


def double_to_half(x: float) -> int:
    return lib().orc_double_to_half(x)


def splitmix64(state0: int, i: int) -> int:
    return lib().orc_splitmix64(state0, i)


def sgd_step(p, q, r: float, lr: float, lambda_p: float, lambda_q: float):
    """One update in binary64 on copies of p and q; returns (p', q')."""
    p = np.array(p, dtype=np.float64)
    q = np.array(q, dtype=np.float64)
    lib().orc_sgd_step(_ptr(p), _ptr(q), len(p), r, lr, lambda_p, lambda_q)
    return p, q


# --- array routines ---------------------------------------------------------------------------
def init_factors(m: int, n: int, k: int, seed: int, dtype=np.float32):
    P = np.empty((m, k), dtype=dtype)
    Qt = np.empty((n, k), dtype=dtype)
    lib().orc_init_factors(m, n, k, seed, _dtype_code(P), _ptr(P), _ptr(Qt))
    return P, Qt


def init_rows(N: int, k: int, seed: int, which: int, rows, dtype=np.float32):
    """Initial values of the given rows of P (which=0) or Q^T (which=1)."""
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((len(rows), k), dtype=dtype)
    lib().orc_init_rows(N, k, seed, _dtype_code(out), which, _ptr(rows), len(rows), _ptr(out))
    return out


def epoch_serial(P, Qt, S, lr, lambda_p, lambda_q):
    """In place: one epoch of serial SGD in array order."""
    S = _samples(S)
    rc = lib().orc_epoch_serial(P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt), _ptr(S), len(S), lr, lambda_p,
                                lambda_q)
    if rc:
        raise MemoryError("oracle epoch failed")


def epoch_wavefront(P, Qt, S, lr, lambda_p, lambda_q, s, seed, t, balanced=False):
    """In place: one deterministic wavefront-update epoch (serial-equivalent order).
    balanced: cut the grid by sample counts (balanced_bounds) instead of equal index ranges."""
    S = _samples(S)
    rc = lib().orc_epoch_wavefront(P.shape[0], Qt.shape[0], P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt),
                                   _ptr(S), len(S), lr, lambda_p, lambda_q, s, seed, t, int(bool(balanced)))
    if rc:
        raise MemoryError("oracle wavefront epoch failed")


def table_order(seed: int, t: int, blocks) -> np.ndarray:
    """Order in which a single worker takes the given blocks (ids ascending:
    the non-empty blocks) from the global scheduling table in epoch t."""
    blocks = np.ascontiguousarray(blocks, dtype=np.int64)
    out = np.empty(max(len(blocks), 1), dtype=np.int64)
    if lib().orc_table_order(seed, t, _ptr(blocks), len(blocks), _ptr(out)):
        raise MemoryError
    return out[:len(blocks)]


def epoch_table(P, Qt, S, lr, lambda_p, lambda_q, s, seed, t):
    """In place: one global-table epoch with a single worker (the non-empty
    blocks of the equal-range s x s grid in table_order, array order inside
    a block)."""
    S = _samples(S)
    rc = lib().orc_epoch_table(P.shape[0], Qt.shape[0], P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt), _ptr(S),
                               len(S), lr, lambda_p, lambda_q, s, seed, t)
    if rc:
        raise MemoryError("oracle global-table epoch failed")


def epoch_hogwild_omp(P, Qt, S, lr, lambda_p, lambda_q, f=256, nthreads=0) -> int:
    """Timing-only racy variant; returns the thread count used."""
    S = _samples(S)
    return lib().orc_epoch_hogwild_omp(P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt), _ptr(S), len(S), lr,
                                       lambda_p, lambda_q, f, nthreads)


def hogwild_batch_owner(nnz: int, f: int, W: int) -> np.ndarray:
    nb = (nnz + f - 1) // f
    out = np.empty(max(nb, 1), dtype=np.int64)
    lib().orc_hogwild_batch_owner(nnz, f, W, _ptr(out))
    return out[:nb]


def fisher_yates(stream: int, s: int) -> np.ndarray:
    a = np.empty(s, dtype=np.int32)
    lib().orc_fisher_yates(stream, s, _ptr(a))
    return a


def wavefront_sigma(seed: int, t: int, s: int) -> np.ndarray:
    """sigma[i, w] = column block of worker i in wave w of epoch t."""
    sig = np.empty((s, s), dtype=np.int32)
    if lib().orc_wavefront_sigma(seed, t, s, _ptr(sig)):
        raise MemoryError
    return sig


def row_block(u, m, s):
    return lib().orc_row_block(u, m, s)


def col_block(v, n, s):
    return lib().orc_col_block(v, n, s)


def balanced_bounds(S, N, which, s) -> np.ndarray:
    """First index of each of the s consecutive ranges (which: 0 users, 1 items)
    whose largest sample count is minimal; bounds[s] = N."""
    S = _samples(S)
    b = np.empty(s + 1, dtype=np.int64)
    if lib().orc_balanced_bounds(_ptr(S), len(S), N, which, s, _ptr(b)):
        raise MemoryError
    return b


def bounded_block(i, bounds, s) -> int:
    b = np.ascontiguousarray(bounds, dtype=np.int64)
    return lib().orc_bounded_block(i, _ptr(b), s)


def block_order(S, m, n, s, balanced=False):
    S = _samples(S)
    order = np.empty(max(len(S), 1), dtype=np.int64)
    start = np.empty(s * s + 1, dtype=np.int64)
    rb = balanced_bounds(S, m, 0, s) if balanced else None
    cb = balanced_bounds(S, n, 1, s) if balanced else None
    if lib().orc_block_order(_ptr(S), len(S), m, n, s, None if rb is None else _ptr(rb),
                             None if cb is None else _ptr(cb), _ptr(order), _ptr(start)):
        raise MemoryError
    return order[:len(S)], start


def block_starts(S, m, n, s, balanced=False) -> np.ndarray:
    """start[b] = first position of block b in the stable bucketing (the
    `start` of block_order, without the order array)."""
    S = _samples(S)
    start = np.empty(s * s + 1, dtype=np.int64)
    rb = balanced_bounds(S, m, 0, s) if balanced else None
    cb = balanced_bounds(S, n, 1, s) if balanced else None
    if lib().orc_block_order(_ptr(S), len(S), m, n, s, None if rb is None else _ptr(rb),
                             None if cb is None else _ptr(cb), None, _ptr(start)):
        raise MemoryError
    return start


def rmse(P, Qt, T) -> float:
    T = _samples(T)
    return lib().orc_rmse(P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt), _ptr(T), len(T))


def sq_errors(P, Qt, T) -> np.ndarray:
    T = _samples(T)
    out = np.empty(max(len(T), 1), dtype=np.float64)
    lib().orc_sq_errors(P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt), _ptr(T), len(T), _ptr(out))
    return out[:len(T)]


def objective(P, Qt, S, lambda_p, lambda_q) -> float:
    S = _samples(S)
    return lib().orc_objective(P.shape[1], _dtype_code(P), _ptr(P), _ptr(Qt), _ptr(S), len(S), lambda_p,
                               lambda_q)
