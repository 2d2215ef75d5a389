"""Full-size checks on the Netflix-shaped workload the benchmark times
(m=480,189, n=17,770, k=128, 99,072,112 training and 1,408,395 test ratings,
binary32).  The serial oracle needs minutes per epoch at this size, so these
are properties that hold at any size plus outputs the oracle computes one by
one (the test RMSE of the trained factors)."""
import numpy as np
import pytest

import oracle

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


@pytest.fixture(scope="module")
def netflix(M, gen):
    w = gen.workload("netflix")
    S, T = gen.make(w)
    return w, S, T, M.samples_to_device(S), M.samples_to_device(T)


def reset(M, **opts):
    o = dict(dtype=0, batch_f=256, workers=0, depth=2, team_waves=0, partition=2, hogwild_grid=0, balance=1,
             sync_every=0, sync_l1=0, spin_limit=1 << 24, skip_stores=2, debug=0, wave_launch=0, half_waves=1, table_grid=256,
             table_workers=0)
    o.update(opts)
    M.reset_options()
    for k, v in o.items():
        M.set_option(k, v)


def test_default_hogwild_visits_every_sample(M, netflix):
    """The default batch-Hogwild! (one XCD, batches claimed in order) on the
    full Netflix shape: every sample is used exactly once.  Its convergence
    against the serial oracle is test_gpu_trajectory's."""
    import torch
    w, S, T, dS, dT = netflix
    reset(M, depth=0, debug=1)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    assert M.get_option("hogwild_form") == 4  # the top item holds 9.6 % of the samples: one XCD
    v = M.debug_visits(len(S))
    assert bool(torch.all(v == 1)), "a sample was skipped or used twice"


def test_one_address_space_form_visits_every_sample(M, netflix):
    """The one-address-space form over all XCDs (option partition = 0, not the
    default: its per-XCD copies of the hot rows trail the serial order by more
    than the Hogwild! tolerance on this shape): every sample used exactly once
    and batch b run by worker b mod W."""
    import torch
    w, S, T, dS, dT = netflix
    reset(M, partition=0, debug=3)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    assert M.get_option("partitioned") == 0
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    assert bool(torch.all(M.debug_visits(len(S)) == 1)), "a sample was skipped or used twice"
    f = 256
    nb = (len(S) + f - 1) // f
    W = min(M.get_option("resident_waves"), nb)
    tr = M.debug_trace(nb).cpu().numpy()
    assert np.array_equal(tr, np.arange(nb) % W)


def test_rmse_kernel_matches_oracle_on_trained_factors(M, netflix):
    w, S, T, dS, dT = netflix
    reset(M)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    P, Q = M.get_factors(w["m"], w["n"], w["k"])
    P, Q = P.cpu().numpy(), Q.cpu().numpy()
    assert M.rmse(dT) == pytest.approx(oracle.rmse(P, Q, T), rel=1e-6)
    sub = T[:: 97]
    assert M.rmse(M.samples_to_device(sub)) == pytest.approx(float(np.sqrt(oracle.sq_errors(P, Q, sub).mean())),
                                                             rel=1e-6)


def test_partitioned_form_at_full_size(M, netflix):
    import torch
    w, S, T, dS, dT = netflix
    reset(M, partition=1, debug=3)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    x = M.get_option("xcds")
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    assert bool(torch.all(M.debug_visits(len(S)) == 1))
    tr = M.debug_trace(x * x).cpu().numpy().reshape(x, x)
    assert np.array_equal(tr, oracle.wavefront_sigma(w["seed"], 0, x))


def test_global_table_at_full_size_replays_serially(M, netflix):
    """The global scheduling table at its bench setting (a 256 x 256 grid, 128
    workers): every sample used once, and the factors equal the oracle's
    serial update of the blocks in the order the trace records (blocks held at
    once share no row and no column), within max-abs 1e-4; the test RMSE
    kernel agrees with the oracle's on the result."""
    import torch
    w, S, T, dS, dT = netflix
    reset(M, table_grid=256, table_workers=128, debug=3)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "table")
    assert bool(torch.all(M.debug_visits(len(S)) == 1))
    B = M.get_option("table_blocks")
    tr = M.debug_trace(3 * B).cpu().numpy().reshape(-1, 3)
    order, start = oracle.block_order(S, w["m"], w["n"], 256)
    assert B == int(np.count_nonzero(np.diff(start)))
    seq = np.concatenate([order[start[b]:start[b + 1]] for b in tr[:, 0]])
    del order
    Po, Qo = oracle.init_factors(w["m"], w["n"], w["k"], w["seed"], np.float32)
    oracle.epoch_serial(Po, Qo, S[seq], w["lr"], w["lam"], w["lam"])
    P, Q = M.get_factors(w["m"], w["n"], w["k"])
    P, Q = P.cpu().numpy(), Q.cpu().numpy()
    assert float(np.abs(P - Po).max()) <= 1e-4 and float(np.abs(Q - Qo).max()) <= 1e-4
    assert M.rmse(dT) == pytest.approx(oracle.rmse(Po, Qo, T), rel=1e-5)


def test_deterministic_wavefront_at_full_size_matches_oracle(M, netflix):
    """Deterministic wavefront-update on the full Netflix shape (32 x 32 grid cut
    by sample counts, one wavefront per worker): every factor entry within
    max-abs 1e-4 of the oracle's serial-equivalent wave order after one epoch."""
    w, S, T, dS, dT = netflix
    s = 32
    reset(M, balance=1)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    M.plan(dS, s)
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "wavefront_det")
    P, Q = M.get_factors(w["m"], w["n"], w["k"])
    P, Q = P.cpu().numpy(), Q.cpu().numpy()
    Po, Qo = oracle.init_factors(w["m"], w["n"], w["k"], w["seed"], np.float32)
    oracle.epoch_wavefront(Po, Qo, S, w["lr"], w["lam"], w["lam"], s, w["seed"], 0, balanced=True)
    print(f"full-size deterministic wavefront: max-abs P {np.abs(P - Po).max():.3g} Q {np.abs(Q - Qo).max():.3g}")
    assert float(np.abs(P - Po).max()) <= 1e-4 and float(np.abs(Q - Qo).max()) <= 1e-4
    assert M.rmse(dT) == pytest.approx(oracle.rmse(Po, Qo, T), rel=1e-5)


def test_half_wavefront_workers_at_full_size(M, netflix):
    """The Netflix shape trained at k = 32 (same samples): one address space
    with two workers per wavefront (every resident slot: 2 x resident
    wavefronts) uses every sample once with batch b on worker b mod W and
    trains; the XCD-partitioned form with paired claims uses every sample
    once in the oracle's column orders."""
    import torch
    w, S, T, dS, dT = netflix
    f = 256
    nb = (len(S) + f - 1) // f
    reset(M, partition=0, debug=3)
    M.init(w["m"], w["n"], 32, w["seed"])
    assert M.get_option("half_workers") == 1
    r0 = M.rmse(dT)
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    assert bool(torch.all(M.debug_visits(len(S)) == 1))
    W = min(2 * M.get_option("resident_waves"), nb)
    assert np.array_equal(M.debug_trace(nb).cpu().numpy(), oracle.hogwild_batch_owner(len(S), f, W))
    M.set_option("debug", 0)
    hist = [r0, M.rmse(dT)]
    for t in range(1, 3):
        M.epoch(dS, w["lr"] * w["decay"] ** t, w["lam"], w["lam"], "hogwild")
        hist.append(M.rmse(dT))
    print("k = 32 half-wavefront test rmse by epoch", hist)
    assert all(b < a for a, b in zip(hist, hist[1:]))
    reset(M, partition=1, debug=3)
    M.init(w["m"], w["n"], 32, w["seed"])
    assert M.get_option("partitioned") == 1
    x = M.get_option("xcds")
    M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    assert bool(torch.all(M.debug_visits(len(S)) == 1))
    tr = M.debug_trace(3 * x * x).cpu().numpy()
    assert np.array_equal(tr[:x * x].reshape(x, x), oracle.wavefront_sigma(w["seed"], 0, x))
