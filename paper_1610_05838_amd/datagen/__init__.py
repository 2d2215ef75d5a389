"""Seeded synthetic workloads with the shapes of the paper's data sets.

The paper trains on Netflix, Yahoo!Music and Hugewiki (section 5.1, Table 2).
Those are not available, so each workload here is a planted low-rank model with
the same m, n, k, train/test sizes and a comparable index skew:

  tiny       m=1,000  n=500  k=32, 50,000 distinct uniform cells, 1% held out,
             r = p*.q* + N(0, 0.1)
  netflix    m=480,189 n=17,770 k=128, 99,072,112 train + 1,408,395 test,
             Zipf(1.0) users and items, r = clamp(round(3.6 + p*.q* + N(0,0.3)), 1, 5)
  yahoo      m=1,000,990 n=624,961 k=128, 252,800,275 + 4,003,960, Zipf(0.8),
             r = clamp(round(100 Phi(p*.q* + N(0,0.25))), 0, 100) / 20
  hugewiki   m=50,082,603 n=39,780 k=128, 3,069,000,000 + 31,000,000,
             Zipf(1.0) users, uniform items, r = N(0,1) + p*.q* with a
             planted rank of 16 (a rank-128 planted user model alone would
             take 25.6 GB of host memory)

p*, q* entries are N(0, 1/sqrt(rank)) (second parameter = variance, so p*.q*
has unit variance); the planted rank is k unless the workload sets "rank".  The training hyper-parameters of each workload ride along in
the returned dict.  This module makes inputs only; it performs no SGD.
"""
from __future__ import annotations

import ctypes as C
import functools
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mfgen.c")
LIB = os.path.join(HERE, "libmfgen.so")

SAMPLE_DTYPE = np.dtype([("u", "<i4"), ("v", "<i4"), ("r", "<f4")])

ADDITIVE, STARS, PERCENTILE, REAL = 0, 1, 2, 3
SEED_BASE = 0x1610058300


class _Table(C.Structure):
    _fields_ = [("cdf", C.c_void_p), ("perm", C.c_void_p), ("guide", C.c_void_p), ("guide_bits", C.c_int)]


class _Spec(C.Structure):
    _fields_ = [("m", C.c_int64), ("n", C.c_int64), ("k", C.c_int32), ("model", C.c_int32),
                ("seed", C.c_uint64), ("noise_var", C.c_double), ("mean", C.c_double)]


# Workload registry.  "draw" is "distinct" (uniform cells without replacement) or
# "independent" (i.i.d. pairs from the index distributions).
WORKLOADS = {
    "tiny": dict(m=1000, n=500, k=32, ntrain=49_500, ntest=500, draw="distinct", zipf_u=0.0, zipf_v=0.0,
                 model=ADDITIVE, noise_var=0.1, mean=0.0, seed=SEED_BASE + 1, dtype="fp32", lr=0.01,
                 lam=0.05, decay=1.0, epochs=5),
    "netflix": dict(m=480_189, n=17_770, k=128, ntrain=99_072_112, ntest=1_408_395, draw="independent",
                    zipf_u=1.0, zipf_v=1.0, model=STARS, noise_var=0.3, mean=3.6, seed=SEED_BASE + 2,
                    dtype="fp32", lr=0.003, lam=0.05, decay=0.99, epochs=20),
    "netflix_fp16": dict(m=480_189, n=17_770, k=128, ntrain=99_072_112, ntest=1_408_395, draw="independent",
                         zipf_u=1.0, zipf_v=1.0, model=STARS, noise_var=0.3, mean=3.6, seed=SEED_BASE + 2,
                         dtype="fp16", lr=0.003, lam=0.05, decay=0.99, epochs=20, grid_s=32),
    "yahoo": dict(m=1_000_990, n=624_961, k=128, ntrain=252_800_275, ntest=4_003_960, draw="independent",
                  zipf_u=0.8, zipf_v=0.8, model=PERCENTILE, noise_var=0.25, mean=0.0, seed=SEED_BASE + 4,
                  dtype="fp32", lr=0.001, lam=0.02, decay=1.0, epochs=20),
    "hugewiki": dict(m=50_082_603, n=39_780, k=128, ntrain=3_069_000_000, ntest=31_000_000,
                     draw="independent", zipf_u=1.0, zipf_v=0.0, model=REAL, noise_var=1.0, mean=0.0,
                     seed=SEED_BASE + 5, dtype="fp16", lr=0.01, lam=0.01, decay=1.0, epochs=10, grid_s=64,
                     rank=16),
}


def build(force: bool = True) -> str:
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, SRC,
                               "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        vp = C.c_void_p
        L.gen_planted.argtypes = [C.POINTER(_Spec), vp, vp]
        L.gen_planted.restype = None
        L.gen_zipf_table.argtypes = [C.c_int64, C.c_double, C.c_uint64, C.c_int, vp, vp]
        L.gen_zipf_table.restype = None
        L.gen_zipf_guide.argtypes = [C.c_int64, vp, C.c_int, vp]
        L.gen_zipf_guide.restype = None
        L.gen_pick_batch.argtypes = [vp, C.c_int64, C.c_int64, C.POINTER(_Table), vp]
        L.gen_pick_batch.restype = None
        L.gen_draw.argtypes = [C.POINTER(_Spec), vp, vp, C.POINTER(_Table), C.POINTER(_Table), C.c_int64, C.c_int64,
                               vp]
        L.gen_draw.restype = None
        L.gen_distinct.argtypes = [C.POINTER(_Spec), vp, vp, C.c_int64, vp]
        L.gen_distinct.restype = C.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _rank(w) -> int:
    return w.get("rank", w["k"])


def _spec(w) -> _Spec:
    return _Spec(w["m"], w["n"], _rank(w), w["model"], w["seed"], w["noise_var"], w["mean"])


def workload(name: str, **overrides) -> dict:
    """The workload description (sizes, distributions, hyper-parameters)."""
    w = dict(WORKLOADS[name])
    w.update(overrides)
    w["name"] = name
    return w


@functools.lru_cache(maxsize=4)
def _planted(m, n, k, model, seed, noise_var, mean):
    sp = _Spec(m, n, k, model, seed, noise_var, mean)
    Ps = np.empty((m, k), dtype=np.float32)
    Qs = np.empty((n, k), dtype=np.float32)
    lib().gen_planted(C.byref(sp), _p(Ps), _p(Qs))
    return Ps, Qs


@functools.lru_cache(maxsize=8)
def zipf_table(N: int, a: float, seed: int, which: int):
    cdf = np.empty(N, dtype=np.float64)
    perm = np.empty(N, dtype=np.int32)
    lib().gen_zipf_table(N, a, seed, which, _p(cdf), _p(perm))
    return cdf, perm


def guide_bits(N: int) -> int:
    return max(10, min(24, int(N).bit_length() + 2))


@functools.lru_cache(maxsize=8)
def zipf_guide(N: int, a: float, seed: int, which: int):
    cdf, _ = zipf_table(N, a, seed, which)
    bits = guide_bits(N)
    guide = np.empty((1 << bits) + 1, dtype=np.int64)
    lib().gen_zipf_guide(N, _p(cdf), bits, _p(guide))
    return guide, bits


def _table(N: int, a: float, seed: int, which: int, guided: bool):
    """ctypes table of one index distribution (and the arrays it points at)."""
    if a <= 0:
        return _Table(None, None, None, 0), ()
    cdf, perm = zipf_table(N, a, seed, which)
    guide, bits = zipf_guide(N, a, seed, which) if guided else (None, 0)
    return _Table(_p(cdf), _p(perm), _p(guide), bits), (cdf, perm, guide)


def pick(x: np.ndarray, N: int, a: float, seed: int, which: int, guided: bool = True) -> np.ndarray:
    """Indices picked for explicit uniforms x in [0, 1)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    t, keep = _table(N, a, seed, which, guided)
    out = np.empty(max(len(x), 1), dtype=np.int64)
    lib().gen_pick_batch(_p(x), len(x), N, C.byref(t), _p(out))
    return out[:len(x)]


def planted(w: dict):
    return _planted(w["m"], w["n"], _rank(w), w["model"], w["seed"], w["noise_var"], w["mean"])


def draw(w: dict, c0: int, count: int, out: np.ndarray | None = None, guided: bool = True) -> np.ndarray:
    """Samples for counters c0 .. c0+count-1 of an "independent" workload.
    guided=False searches the Zipf tables without their guide (same result)."""
    assert w["draw"] == "independent"
    Ps, Qs = planted(w)
    tu, keep_u = _table(w["m"], w["zipf_u"], w["seed"], 0, guided)
    tv, keep_v = _table(w["n"], w["zipf_v"], w["seed"], 1, guided)
    if out is None:
        out = np.empty(count, dtype=SAMPLE_DTYPE)
    assert out.dtype == SAMPLE_DTYPE and out.flags["C_CONTIGUOUS"] and len(out) >= count
    lib().gen_draw(C.byref(_spec(w)), _p(Ps), _p(Qs), C.byref(tu), C.byref(tv), c0, count, _p(out))
    return out


def make(w: dict):
    """(train, test) sample arrays of a workload.  Train samples are counters
    0..ntrain-1 and test samples ntrain..ntrain+ntest-1 of the same process; for
    "distinct" workloads the first ntrain cells are train, the rest test."""
    if w["draw"] == "distinct":
        total = w["ntrain"] + w["ntest"]
        Ps, Qs = planted(w)
        out = np.empty(total, dtype=SAMPLE_DTYPE)
        if lib().gen_distinct(C.byref(_spec(w)), _p(Ps), _p(Qs), total, _p(out)):
            raise ValueError("more distinct cells requested than the grid holds")
        return out[:w["ntrain"]].copy(), out[w["ntrain"]:].copy()
    train = draw(w, 0, w["ntrain"])
    test = draw(w, w["ntrain"], w["ntest"])
    return train, test


def lr_at(w: dict, t: int) -> float:
    """Learning rate of epoch t (0-based): lr * decay^t."""
    return float(w["lr"] * (w["decay"] ** t))


def draw_to_device(w: dict, c0: int, count: int, device="cuda", chunk: int = 1 << 25, progress=None):
    """The samples of counters c0 .. c0+count-1 as an int32 (count, 3) torch
    tensor on `device`, generated chunk by chunk through a pinned host buffer
    (so a multi-GB sample array never has to exist in host memory)."""
    import torch

    out = torch.empty((count, 3), dtype=torch.int32, device=device)
    if count == 0:
        return out
    n0 = min(chunk, count)
    bufs = [torch.empty((n0, 3), dtype=torch.int32).pin_memory() for _ in range(2)]
    done = [None, None]
    stream = torch.cuda.current_stream(device)
    for i, off in enumerate(range(0, count, chunk)):
        n = min(chunk, count - off)
        b = i & 1
        if done[b] is not None:
            done[b].synchronize()  # the copy that last read this buffer has finished
        host = bufs[b][:n]
        draw(w, c0 + off, n, out=host.numpy().view(SAMPLE_DTYPE).reshape(-1))
        out[off:off + n].copy_(host, non_blocking=True)
        done[b] = torch.cuda.Event()
        done[b].record(stream)
        if progress:
            progress(off + n, count)
    torch.cuda.synchronize(device)
    return out
