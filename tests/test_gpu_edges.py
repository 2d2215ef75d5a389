"""Degenerate shapes through the C ABI against the oracle: a 1 x 1 model
(every sample updates the same two rows, so every in-flight window forwards),
and grids with more row or column blocks than users or items (empty blocks
in every wave).  Single-worker batch-Hogwild!, the deterministic
wavefront-update and the one-worker global table all match the oracle's order
within max-abs 1e-4 (binary32) / 2e-2 (binary16)."""
import numpy as np
import pytest

import oracle
from test_gpu_parity import TOL, factors, maxabs, rand_samples, setup

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def M():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1610_05838_amd import mfsgd
    mfsgd.lib()
    yield mfsgd
    mfsgd.finalize()


SHAPES = [(1, 1), (3, 2), (2, 7), (13, 1)]


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("m,n", SHAPES)
def test_degenerate_shapes(M, m, n, dtype):
    rng = np.random.default_rng(m * 31 + n)
    S = rand_samples(rng, m, n, 777, lo=-1.0, hi=1.0)
    k, seed, lr, lam, s = 32, 4321 + m, 0.01, 0.02, 8
    dS = M.samples_to_device(S)

    setup(M, m, n, k, seed, dtype, workers=1, partition=0)
    M.epoch(dS, lr, lam, lam, "hogwild")
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    oracle.epoch_serial(Po, Qo, S, lr, lam, lam)
    P, Q = factors(M, m, n, k, dtype)
    assert maxabs(P, Po) <= TOL[dtype] and maxabs(Q, Qo) <= TOL[dtype]

    setup(M, m, n, k, seed, dtype, balance=0)
    M.plan(dS, s)
    M.epoch(dS, lr, lam, lam, "wavefront_det")
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    oracle.epoch_wavefront(Po, Qo, S, lr, lam, lam, s, seed, 0, balanced=False)
    P, Q = factors(M, m, n, k, dtype)
    assert maxabs(P, Po) <= TOL[dtype] and maxabs(Q, Qo) <= TOL[dtype]

    setup(M, m, n, k, seed, dtype, table_grid=s, table_workers=1)
    M.epoch(dS, lr, lam, lam, "table")
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    oracle.epoch_table(Po, Qo, S, lr, lam, lam, s, seed, 0)
    P, Q = factors(M, m, n, k, dtype)
    assert maxabs(P, Po) <= TOL[dtype] and maxabs(Q, Qo) <= TOL[dtype]
    assert M.get_option("table_blocks") == len({(u * s // m) * s + v * s // n for u, v in zip(S["u"], S["v"])})


@pytest.mark.parametrize("m,n", SHAPES)
def test_degenerate_shapes_many_workers_cover_every_sample(M, m, n):
    """Every schedule with many workers still uses each sample exactly once."""
    rng = np.random.default_rng(7 * m + n)
    S = rand_samples(rng, m, n, 5000)
    dS = M.samples_to_device(S)
    setup(M, m, n, 32, 5, debug=1, partition=0, workers=64)
    M.epoch(dS, 0.001, 0.0, 0.0, "hogwild")
    assert bool((M.debug_visits(len(S)) == 1).all().item())
    M.plan(dS, 8)
    for scheme in ("wavefront", "wavefront_det"):
        M.epoch(dS, 0.001, 0.0, 0.0, scheme)
        assert bool((M.debug_visits(len(S)) == 1).all().item())
    setup(M, m, n, 32, 5, debug=1, table_grid=8, table_workers=16)
    M.epoch(dS, 0.001, 0.0, 0.0, "table")
    assert bool((M.debug_visits(len(S)) == 1).all().item())
