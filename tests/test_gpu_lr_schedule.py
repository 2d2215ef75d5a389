"""The evaluation section's learning-rate schedule on the GPU path against
the oracle (section 5.1: the rate of epoch t is s_t = alpha / (1 + beta *
t^1.5), with alpha, beta and lambda from Table 3).  The schedule is host-side:
the caller passes s_t as the epoch's lr.  A small model runs five epochs
with one batch-Hogwild! worker (the serial order) and with the deterministic
wavefront-update schedule, and the factors are compared with the oracle's
after every epoch under the same per-epoch rates: max-abs 1e-4 (binary32),
2e-2 (binary16)."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

TOL = {np.float32: 1e-4, np.float16: 2e-2}


@pytest.fixture(scope="module")
def M():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1610_05838_amd import mfsgd
    mfsgd.lib()
    yield mfsgd
    mfsgd.finalize()


def s_t(alpha, beta, t):
    return alpha / (1.0 + beta * t ** 1.5)


@pytest.mark.parametrize("mode", ["one_worker", "wavefront_det"])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("row", ["Netflix", "Yahoo!Music"])
def test_paper_schedule_matches_oracle(M, gen, row, dtype, mode):
    import converge
    lam, alpha, beta = converge.PAPER_PARAMS[{"Netflix": "netflix", "Yahoo!Music": "yahoo"}[row]]
    rng = np.random.default_rng(1610 + len(row) + (dtype == np.float16) + 7 * (mode == "one_worker"))
    m, n, k, seed, s = 300, 200, 64, 97, 4
    S = np.zeros(40_000, dtype=oracle.SAMPLE_DTYPE)
    S["u"], S["v"] = rng.integers(0, m, len(S)), rng.integers(0, n, len(S))
    S["r"] = rng.uniform(1.0, 5.0, len(S)).astype(np.float32)
    M.reset_options()
    M.set_option("dtype", 1 if dtype == np.float16 else 0)
    M.set_option("balance", 1)
    if mode == "one_worker":
        M.set_option("partition", 0)
        M.set_option("workers", 1)
    M.init(m, n, k, seed)
    dS = M.samples_to_device(S)
    if mode == "wavefront_det":
        M.plan(dS, s)
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    worst = []
    for t in range(5):
        lr = s_t(alpha, beta, t)
        assert converge.lr_schedule({"name": "netflix" if row == "Netflix" else "yahoo"}, "paper")[0](t) == lr
        if mode == "one_worker":
            M.epoch(dS, lr, lam, lam, "hogwild")
            oracle.epoch_serial(Po, Qo, S, lr, lam, lam)
        else:
            M.epoch(dS, lr, lam, lam, "wavefront_det")
            oracle.epoch_wavefront(Po, Qo, S, lr, lam, lam, s, seed, t, balanced=True)
        P, Q = M.get_factors(m, n, k)
        P, Q = P.cpu().numpy().astype(dtype), Q.cpu().numpy().astype(dtype)
        err = max(float(np.abs(P.astype(np.float64) - Po).max()), float(np.abs(Q.astype(np.float64) - Qo).max()))
        worst.append(err)
        assert err <= TOL[dtype], (t, lr, err)
    print(f"{row} {np.dtype(dtype).name} {mode}: rates {[round(s_t(alpha, beta, t), 5) for t in range(5)]}, "
          f"max-abs per epoch {['%.2e' % x for x in worst]}")
