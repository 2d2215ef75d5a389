"""mfsgd_rmse_noalloc (the entry point for callers that cannot allocate)
against mfsgd_rmse through the C ABI: the same value on two calls in a row,
the second on a smaller test set, both after training, and 0 for an empty
test set."""
import ctypes

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


def test_rmse_noalloc_equals_rmse():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1610_05838_amd import mfsgd as M
    L = M.lib()
    rng = np.random.default_rng(2024)
    m, n, k, seed = 3000, 1700, 128, 41
    S = np.zeros(200_000, dtype=oracle.SAMPLE_DTYPE)
    S["u"], S["v"], S["r"] = rng.integers(0, m, len(S)), rng.integers(0, n, len(S)), rng.uniform(1, 5, len(S))
    T1 = np.zeros(50_001, dtype=oracle.SAMPLE_DTYPE)
    T1["u"], T1["v"], T1["r"] = rng.integers(0, m, len(T1)), rng.integers(0, n, len(T1)), rng.uniform(1, 5, len(T1))
    T2 = np.ascontiguousarray(T1[:777])
    for dtype in (0, 1):
        M.reset_options()
        M.set_option("dtype", dtype)
        M.init(m, n, k, seed)
        M.epoch(M.samples_to_device(S), 0.01, 0.05, 0.05, "hogwild")
        out = torch.full((1,), -1.0, dtype=torch.float64, device="cuda")
        stream = torch.cuda.current_stream()
        for T in (T1, T2):
            dT = M.samples_to_device(T)
            rc = L.mfsgd_rmse_noalloc(ctypes.c_void_p(dT.data_ptr()), len(T), ctypes.c_void_p(out.data_ptr()),
                                      ctypes.c_void_p(stream.cuda_stream))
            assert rc == 0, L.mfsgd_last_error()
            torch.cuda.synchronize()
            got = float(out.item())
            want = M.rmse(dT)
            print(f"dtype {dtype} ntest {len(T)}: noalloc {got!r} rmse {want!r}")
            assert got == want
        rc = L.mfsgd_rmse_noalloc(ctypes.c_void_p(dT.data_ptr()), 0, ctypes.c_void_p(out.data_ptr()),
                                  ctypes.c_void_p(stream.cuda_stream))
        assert rc == 0
        torch.cuda.synchronize()
        assert float(out.item()) == 0.0
        assert L.mfsgd_rmse_noalloc(ctypes.c_void_p(dT.data_ptr()), 10, None, ctypes.c_void_p(stream.cuda_stream)) == -1
    M.finalize()
