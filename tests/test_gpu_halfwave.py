"""Two batch-Hogwild! workers per wavefront at k <= 32 (option half_waves).

A row of 32 values fills half of a 64-lane wavefront, so the one-address-space
batch-Hogwild! kernel runs one worker per half.  Checks, through the C ABI:

* a lone worker computes the same bits as the one-worker-per-wavefront kernel
  (its 32-lane dot product adds the same terms in the same order) and matches
  the serial oracle (section 3.2.2 with W = 1 is the serial order);
* W workers whose batches touch disjoint rows and columns (batch b uses only
  the rows of group b mod W) do not interact, so the result is the serial
  oracle's whatever the interleaving, bit-identical to the one-per-wavefront
  kernel; odd W leaves the upper half of the last wavefront idle, and ragged
  sizes end a half's sequence mid-chunk or mid-batch;
* the schedule: batch b is run by worker b mod W, every sample exactly once.
Tolerances as in the other parity tests: max-abs 1e-4 (binary32) and 2e-2
(binary16) against the binary64 oracle.
"""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

TOL = {np.float32: 1e-4, np.float16: 2e-2}
DEFAULTS = dict(dtype=0, batch_f=256, workers=0, depth=2, team_waves=0, partition=0, hogwild_grid=0, balance=1,
                sync_every=0, sync_l1=0, spin_limit=1 << 24, skip_stores=2, debug=0,
                wave_launch=0, half_waves=1, table_grid=256, table_workers=0)


@pytest.fixture(scope="module")
def M():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1610_05838_amd import mfsgd
    mfsgd.lib()
    yield mfsgd
    mfsgd.finalize()


def run(M, S, m, n, k, seed, dtype, epochs=1, **opts):
    o = dict(DEFAULTS)
    o["dtype"] = 1 if dtype == np.float16 else 0
    o.update(opts)
    M.reset_options()
    for key, val in o.items():
        M.set_option(key, val)
    M.init(m, n, k, seed)
    dS = M.samples_to_device(S)
    for _ in range(epochs):
        M.epoch(dS, 0.01, 0.05, 0.04, "hogwild")
    P, Q = M.get_factors(m, n, k)
    return P.cpu().numpy().astype(dtype), Q.cpu().numpy().astype(dtype)


def serial(S, m, n, k, seed, dtype, epochs=1):
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    for _ in range(epochs):
        oracle.epoch_serial(Po, Qo, S, 0.01, 0.05, 0.04)
    return Po, Qo


def maxabs(a, b):
    return float(np.max(np.abs(a.astype(np.float64) - b.astype(np.float64)))) if a.size else 0.0


def bits(a):
    return a.view(np.uint32 if a.dtype == np.float32 else np.uint16)


def grouped_samples(rng, W, f, nnz, mu, nv):
    """Batch b of f consecutive samples draws its user from [g mu, (g+1) mu)
    and its item from [g nv, (g+1) nv), g = b mod W: the workers of
    batch-Hogwild! with W workers then share no row and no column."""
    a = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
    g = (np.arange(nnz) // f) % W
    a["u"] = g * mu + rng.integers(0, mu, nnz)
    a["v"] = g * nv + rng.integers(0, nv, nnz)
    a["r"] = rng.uniform(1.0, 5.0, nnz).astype(np.float32)
    return a, W * mu, W * nv


@pytest.mark.parametrize("depth", [1, 2, 4, 8])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("k", [1, 20, 32])
def test_lone_worker_same_bits_as_full_wavefront(M, depth, dtype, k):
    rng = np.random.default_rng(100 * depth + k)
    for m, n, nnz in ((7, 5, 2001), (400, 300, 6037)):  # 7 x 5: consecutive samples share rows all the time
        S = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
        S["u"] = rng.integers(0, m, nnz)
        S["v"] = rng.integers(0, n, nnz)
        S["r"] = rng.uniform(1.0, 5.0, nnz).astype(np.float32)
        seed = 5 + k
        Ph, Qh = run(M, S, m, n, k, seed, dtype, workers=1, depth=depth, half_waves=1)
        Pf, Qf = run(M, S, m, n, k, seed, dtype, workers=1, depth=depth, half_waves=0)
        assert np.array_equal(bits(Ph), bits(Pf)) and np.array_equal(bits(Qh), bits(Qf)), (m, n)
        Po, Qo = serial(S, m, n, k, seed, dtype)
        assert maxabs(Ph, Po) <= TOL[dtype] and maxabs(Qh, Qo) <= TOL[dtype], (m, n)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("W,f,nnz", [
    (2, 256, 20 * 256),            # both halves of one wavefront, whole batches
    (2, 64, 37 * 64 + 45),         # ragged: the array ends inside the upper half's batch
    (3, 256, 11 * 256 + 200),      # odd: the second wavefront's upper half idles
    (5, 128, 23 * 128 + 17),       # last batch partial and owned by a lower half
    (8, 64, 8 * 64 * 3 + 64 + 31), # the last wavefronts run one batch fewer
])
def test_disjoint_workers_equal_serial(M, dtype, W, f, nnz):
    rng = np.random.default_rng(W * 7919 + nnz)
    S, m, n = grouped_samples(rng, W, f, nnz, 6, 4)
    k, seed = 32, 41 + W
    for depth in (1, 2, 8):
        Ph, Qh = run(M, S, m, n, k, seed, dtype, epochs=2, workers=W, batch_f=f, depth=depth, half_waves=1)
        Pf, Qf = run(M, S, m, n, k, seed, dtype, epochs=2, workers=W, batch_f=f, depth=depth, half_waves=0)
        assert np.array_equal(bits(Ph), bits(Pf)) and np.array_equal(bits(Qh), bits(Qf)), depth
        Po, Qo = serial(S, m, n, k, seed, dtype, epochs=2)
        assert maxabs(Ph, Po) <= TOL[dtype] and maxabs(Qh, Qo) <= TOL[dtype], depth


@pytest.mark.parametrize("k", [16, 32])
@pytest.mark.parametrize("W", [1, 2, 7, 1000, 0])
def test_schedule_and_coverage(M, k, W):
    rng = np.random.default_rng(W + k)
    m, n, nnz, seed, f = 3000, 2000, 300_017, 9, 256
    S = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
    S["u"] = rng.integers(0, m, nnz)
    S["v"] = rng.integers(0, n, nnz)
    S["r"] = rng.uniform(1.0, 5.0, nnz).astype(np.float32)
    M.reset_options()
    for key, val in dict(DEFAULTS, debug=3, workers=W).items():
        M.set_option(key, val)
    M.init(m, n, k, seed)
    M.epoch(M.samples_to_device(S), 0.001, 0.05, 0.05, "hogwild")
    assert np.all(M.debug_visits(nnz).cpu().numpy() == 1)
    nb = (nnz + f - 1) // f
    trace = M.debug_trace(nb).cpu().numpy()
    if W == 0:  # the default: two workers per resident wavefront, fewer if batches run out
        Wd = min(2 * M.get_option("resident_waves"), nb)
        assert np.array_equal(trace, oracle.hogwild_batch_owner(nnz, f, Wd))
    else:
        assert np.array_equal(trace, oracle.hogwild_batch_owner(nnz, f, min(W, nb)))


@pytest.mark.parametrize("nnz", [1, 5, 31, 32, 33, 255, 257])
def test_tiny_arrays(M, nnz):
    rng = np.random.default_rng(nnz)
    m, n, k, seed = 9, 6, 32, 3
    S = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
    S["u"] = rng.integers(0, m, nnz)
    S["v"] = rng.integers(0, n, nnz)
    S["r"] = rng.uniform(1.0, 5.0, nnz).astype(np.float32)
    for W in (1, 2, 3):
        P, Q = run(M, S, m, n, k, seed, np.float32, workers=W, batch_f=64)
        if W == 1 or nnz <= 64:  # a single batch: one worker runs everything
            Po, Qo = serial(S, m, n, k, seed, np.float32)
            assert maxabs(P, Po) <= 1e-4 and maxabs(Q, Qo) <= 1e-4, W


def test_two_workers_rmse_gap(M, gen):
    """Both halves of one wavefront as two batch-Hogwild! workers that do
    share rows (the tiny workload's model and density on a 4000 x 2000 grid):
    after five epochs the test RMSE is within the binary32 Hogwild! tolerance
    of the serial oracle's (workers far below min(m, n), the condition under
    which Hogwild! behaves like serial SGD)."""
    w = gen.workload("tiny", m=4000, n=2000, ntrain=49_500 * 16, ntest=500 * 16, seed=gen.SEED_BASE + 11)
    S, T = gen.make(w)
    m, n, k, seed = w["m"], w["n"], w["k"], w["seed"]
    assert k <= 32
    M.reset_options()
    for key, val in dict(DEFAULTS, workers=2).items():
        M.set_option(key, val)
    M.init(m, n, k, seed)
    dS, dT = M.samples_to_device(S), M.samples_to_device(T)
    for _ in range(5):
        M.epoch(dS, w["lr"], w["lam"], w["lam"], "hogwild")
    got = M.rmse(dT)
    Po, Qo = oracle.init_factors(m, n, k, seed, np.float32)
    for _ in range(5):
        oracle.epoch_serial(Po, Qo, S, w["lr"], w["lam"], w["lam"])
    want = oracle.rmse(Po, Qo, T)
    print(f"two half-wavefront workers rmse {got:.6f} oracle {want:.6f}")
    assert abs(got - want) <= 1e-3


# ---------------------------------------------------------------------------- block-scheduled kernel
def disjoint_block_samples(rng, s, f, G, gu, gv):
    """An s x s grid (equal index ranges) in which batch j of block (t, c)
    draws its users from sub-range c G + j of row block t and its items from
    sub-range j of column block c.  Every user then belongs to one batch, and
    an item's batches lie in different blocks of its column, which the
    column tickets order: batches that may run at the same time (those of one
    block, and those of a team's consecutive blocks) touch disjoint rows, so
    any run of the schedule equals the serial update in the schedule's block
    order.  Blocks hold 0..G batches of f samples, the last one ragged; the
    array lists the blocks in random order, each block's samples in batch
    order."""
    m, n = s * s * G * gu, s * G * gv
    parts = []
    for t in range(s):
        for c in range(s):
            nb = int(rng.integers(0, G + 1))
            for j in range(nb):
                cnt = f if j < nb - 1 else int(rng.integers(1, f + 1))
                a = np.zeros(cnt, dtype=oracle.SAMPLE_DTYPE)
                a["u"] = (t * s + c) * G * gu + j * gu + rng.integers(0, gu, cnt)
                a["v"] = c * G * gv + j * gv + rng.integers(0, gv, cnt)
                a["r"] = rng.uniform(1.0, 5.0, cnt).astype(np.float32)
                parts.append((t * s + c, j, a))
    order = rng.permutation(s * s)
    rank = np.empty(s * s, dtype=np.int64)
    rank[order] = np.arange(s * s)
    parts.sort(key=lambda p: (rank[p[0]], p[1]))
    return np.concatenate([p[2] for p in parts]), m, n


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("s,skip", [(4, 0), (8, 0), (8, 2), (16, 0)])
def test_block_scheduled_pairs_equal_schedule_order(M, dtype, s, skip):
    """Partitioned batch-Hogwild! at k = 32: pooled wavefronts claim two
    batches at a time and run one per half (also where skipped stores would
    be chosen); on blocks whose concurrently runnable batches commute the
    result is the oracle's update in the wavefront block order (section
    3.2.3), and the same bits as one batch per wavefront."""
    scheme = "hogwild"
    rng = np.random.default_rng(s * 31 + skip)
    f = 64
    G, gu, gv = 6, 3, 2
    S, m, n = disjoint_block_samples(rng, s, f, G, gu, gv)
    k, seed = 32, 123 + s
    opts = dict(batch_f=f, balance=0, partition=1, hogwild_grid=s, skip_stores=skip)
    res = {}
    for half in (1, 0):
        o = dict(DEFAULTS, dtype=1 if dtype == np.float16 else 0, half_waves=half, **opts)
        M.reset_options()
        for key, val in o.items():
            M.set_option(key, val)
        M.init(m, n, k, seed)
        dS = M.samples_to_device(S)
        if scheme == "wavefront":
            M.plan(dS, s)
        else:
            assert M.get_option("partitioned") == 1
        for _ in range(2):
            M.epoch(dS, 0.01, 0.05, 0.04, scheme)
        P, Q = M.get_factors(m, n, k)
        res[half] = (P.cpu().numpy().astype(dtype), Q.cpu().numpy().astype(dtype))
    (Ph, Qh), (Pf, Qf) = res[1], res[0]
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    for t in range(2):
        oracle.epoch_wavefront(Po, Qo, S, 0.01, 0.05, 0.04, s, seed, t, balanced=False)
    for half, (P, Q) in res.items():
        # name the rows (and their blocks) that left the schedule's result
        dP = np.abs(P.astype(np.float64) - Po).max(axis=1)
        dQ = np.abs(Q.astype(np.float64) - Qo).max(axis=1)
        badP, badQ = np.nonzero(dP > TOL[dtype])[0], np.nonzero(dQ > TOL[dtype])[0]
        where = (f"half_waves={half}: P rows {badP[:8].tolist()} (blocks {(badP[:8] // (G * gu)).tolist()}), "
                 f"Q rows {badQ[:8].tolist()} (column blocks {(badQ[:8] // (G * gv)).tolist()}), "
                 f"max {dP.max():.3g} / {dQ.max():.3g}")
        print(where)
        assert badP.size == 0 and badQ.size == 0, where
    assert np.array_equal(bits(Ph), bits(Pf)) and np.array_equal(bits(Qh), bits(Qf))


@pytest.mark.parametrize("dtype,k", [(np.float32, 64), (np.float32, 128), (np.float16, 128), (np.float16, 256)])
@pytest.mark.parametrize("scheme,skip", [("hogwild", 0), ("hogwild", 1), ("wavefront", 0), ("wavefront", 1)])
def test_block_scheduled_wide_pairs_equal_schedule_order(M, dtype, k, scheme, skip):
    """Two batches per claim at rows wider than 32 values (option
    half_waves = 2: each lane of a half holds k/32 values, 8 to 16 bytes),
    with and without skipped stores, under the partitioned batch-Hogwild! and
    wavefront-update schedules: on blocks whose concurrently runnable batches
    commute the result is the oracle's update in the wavefront block order
    (section 3.2.3) within the usual bounds, and a second run gives the same
    bits."""
    rng = np.random.default_rng(77 + skip + (scheme == "wavefront"))
    s, f = 8, 64
    G, gu, gv = 6, 3, 2
    S, m, n = disjoint_block_samples(rng, s, f, G, gu, gv)
    seed = 31
    opts = dict(batch_f=f, balance=0, partition=1, hogwild_grid=s, skip_stores=skip, half_waves=2)
    runs = []
    for rep in range(2):
        o = dict(DEFAULTS, dtype=1 if dtype == np.float16 else 0, **opts)
        M.reset_options()
        for key, val in o.items():
            M.set_option(key, val)
        M.init(m, n, k, seed)
        dS = M.samples_to_device(S)
        if scheme == "wavefront":
            M.plan(dS, s)
        for _ in range(2):
            M.epoch(dS, 0.01, 0.05, 0.04, scheme)
        runs.append(tuple(x.cpu().numpy().astype(dtype) for x in M.get_factors(m, n, k)))
    Po, Qo = oracle.init_factors(m, n, k, seed, dtype)
    for t in range(2):
        oracle.epoch_wavefront(Po, Qo, S, 0.01, 0.05, 0.04, s, seed, t, balanced=False)
    P, Q = runs[0]
    assert maxabs(P, Po) <= TOL[dtype] and maxabs(Q, Qo) <= TOL[dtype]
    assert np.array_equal(bits(runs[1][0]), bits(P)) and np.array_equal(bits(runs[1][1]), bits(Q))


@pytest.mark.parametrize("half", [1, 0])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("s", [8, 16])
def test_block_scheduled_runs_repeat_bit_for_bit(M, dtype, s, half):
    """Column hand-over under load: blocks of at most a few batches, so the
    next block in a column is claimed the moment its ticket moves and its
    first batch reads the rows the previous block wrote on another XCD.  On
    data whose concurrently runnable batches commute, every run of the
    schedule is the same computation, so repeated runs agree bit for bit
    (a ticket seen before the releasing XCD's L2 write-back has finished
    shows up as a lost update in some column's first batch)."""
    rng = np.random.default_rng(1000 + s)
    f = 64
    S, m, n = disjoint_block_samples(rng, s, f, 3, 3, 2)
    k, seed = 32, 7 + s
    first = None
    for rep in range(6):
        o = dict(DEFAULTS, dtype=1 if dtype == np.float16 else 0, half_waves=half, batch_f=f, balance=0,
                 partition=1, hogwild_grid=s, skip_stores=0)
        M.reset_options()
        for key, val in o.items():
            M.set_option(key, val)
        M.init(m, n, k, seed)
        dS = M.samples_to_device(S)
        for _ in range(3):
            M.epoch(dS, 0.01, 0.05, 0.04, "hogwild")
        P, Q = (x.cpu().numpy().astype(dtype) for x in M.get_factors(m, n, k))
        if first is None:
            first = (P, Q)
            continue
        rows_p = np.nonzero(np.any(bits(P) != bits(first[0]), axis=1))[0]
        rows_q = np.nonzero(np.any(bits(Q) != bits(first[1]), axis=1))[0]
        assert rows_p.size == 0 and rows_q.size == 0, \
            f"run {rep}: P rows {rows_p[:8].tolist()}, Q rows {rows_q[:8].tolist()} differ from run 0"


@pytest.mark.parametrize("scheme,s,opts", [
    ("hogwild", 8, {"partition": 1}), ("hogwild", 16, {"partition": 1, "hogwild_grid": 16}),
    ("wavefront", 32, {}),
])
def test_block_scheduled_pairs_coverage_and_handover(M, gen, scheme, s, opts):
    """Race check with two batches per claim (partitioned batch-Hogwild! at
    k = 32, pooled teams, Zipf blocks; wavefront-update, which keeps one batch
    per claim, alongside): every sample once, the oracle's column orders, and
    in every column each wave's block claimed only after the previous wave's
    block completed (claim and completion stamps of one event counter)."""
    w = gen.workload("netflix", m=30_000, n=4_000, ntrain=800_000, ntest=0)
    S = gen.draw(w, 0, w["ntrain"])
    M.reset_options()
    for key, val in dict(DEFAULTS, **{"partition": 2, "debug": 3, "skip_stores": 0, **opts}).items():
        M.set_option(key, val)
    M.init(w["m"], w["n"], 32, w["seed"])
    dS = M.samples_to_device(S)
    if scheme != "hogwild":
        M.plan(dS, s)
    for t in range(2):
        M.epoch(dS, 0.002, 0.01, 0.01, scheme)
        assert bool((M.debug_visits(len(S)) == 1).all().item())
        tr = M.debug_trace(3 * s * s).cpu().numpy()
        assert np.array_equal(tr[:s * s].reshape(s, s), oracle.wavefront_sigma(w["seed"], t, s))
        cols = tr[:s * s].reshape(s, s)
        st = tr[s * s:3 * s * s].view(np.uint32).reshape(s, s, 2).astype(np.int64)
        assert np.all(st[:, :, 0] < st[:, :, 1])
        team_of = np.empty((s, s), dtype=np.int64)
        for tm in range(s):
            team_of[cols[tm], np.arange(s)] = tm
        for c in range(s):
            prev, nxt = team_of[c, :-1], team_of[c, 1:]
            assert np.all(st[nxt, np.arange(1, s), 0] > st[prev, np.arange(s - 1), 1]), c


# ---------------------------------------------------------------------------- wider rows (half_waves = 2)
@pytest.mark.parametrize("depth", [1, 2, 8])
@pytest.mark.parametrize("dtype,k", [(np.float32, 50), (np.float32, 128), (np.float16, 64), (np.float16, 128),
                                     (np.float16, 256)])
def test_wide_rows_lone_worker_equals_serial(M, depth, dtype, k):
    """half_waves = 2: two workers per wavefront at wider rows (KP/32 values
    per lane); one worker equals the serial oracle within the storage
    tolerance (its lane sums run in another order than one worker per
    wavefront, so bits may differ)."""
    rng = np.random.default_rng(7 * depth + k)
    for m, n, nnz in ((7, 5, 2001), (400, 300, 6037)):
        S = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
        S["u"] = rng.integers(0, m, nnz)
        S["v"] = rng.integers(0, n, nnz)
        S["r"] = rng.uniform(1.0, 5.0, nnz).astype(np.float32)
        seed = 11 + k
        P, Q = run(M, S, m, n, k, seed, dtype, workers=1, depth=depth, half_waves=2)
        Po, Qo = serial(S, m, n, k, seed, dtype)
        assert maxabs(P, Po) <= TOL[dtype] and maxabs(Q, Qo) <= TOL[dtype], (m, n)


@pytest.mark.parametrize("dtype,k", [(np.float32, 128), (np.float16, 128), (np.float16, 256)])
@pytest.mark.parametrize("W,f,nnz", [(2, 64, 37 * 64 + 45), (3, 256, 11 * 256 + 200), (8, 64, 8 * 64 * 3 + 64 + 31)])
def test_wide_rows_disjoint_workers_equal_serial(M, dtype, k, W, f, nnz):
    rng = np.random.default_rng(W * 31 + k)
    S, m, n = grouped_samples(rng, W, f, nnz, 6, 4)
    seed = 5 + W
    for depth in (1, 2):
        P, Q = run(M, S, m, n, k, seed, dtype, epochs=2, workers=W, batch_f=f, depth=depth, half_waves=2)
        Po, Qo = serial(S, m, n, k, seed, dtype, epochs=2)
        assert maxabs(P, Po) <= TOL[dtype] and maxabs(Q, Qo) <= TOL[dtype], depth


@pytest.mark.parametrize("dtype", [0, 1])
def test_wide_rows_schedule_and_coverage(M, dtype):
    rng = np.random.default_rng(dtype)
    m, n, nnz, seed, f = 3000, 2000, 300_017, 9, 256
    S = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
    S["u"] = rng.integers(0, m, nnz)
    S["v"] = rng.integers(0, n, nnz)
    S["r"] = rng.uniform(1.0, 5.0, nnz).astype(np.float32)
    for W in (7, 0):
        M.reset_options()
        for key, val in dict(DEFAULTS, dtype=dtype, debug=3, workers=W, half_waves=2).items():
            M.set_option(key, val)
        M.init(m, n, 128, seed)
        M.epoch(M.samples_to_device(S), 0.001, 0.05, 0.05, "hogwild")
        assert np.all(M.debug_visits(nnz).cpu().numpy() == 1)
        nb = (nnz + f - 1) // f
        Wd = W if W else min(2 * M.get_option("resident_waves"), nb)
        assert np.array_equal(M.debug_trace(nb).cpu().numpy(), oracle.hogwild_batch_owner(nnz, f, Wd))


def test_blocked_pairs_choice(M):
    """Read-only key blocked_pairs: -1 before a block-scheduled epoch (a
    one-address-space epoch leaves it there).  Pooled wavefront-update at
    k = 128 claims two batches per wavefront when no column block of the plan
    holds more than twice its mean share (uniform items) and one where a hot
    item's column block does; half_waves = 0 turns it off and 2 on; teams of
    one wavefront (the deterministic scheme) keep one batch; block-scheduled
    batch-Hogwild! pairs its claims at k = 32."""
    rng = np.random.default_rng(5)
    m, n, nnz, s = 3000, 2000, 200_000, 8
    uni = np.zeros(nnz, dtype=oracle.SAMPLE_DTYPE)
    uni["u"] = rng.integers(0, m, nnz)
    uni["v"] = rng.integers(0, n, nnz)
    uni["r"] = rng.standard_normal(nnz)
    hot = uni.copy()
    hot["v"][::2] = 7  # one item with half of the samples: its column block holds four times its share

    def last(S, k, scheme, **opts):
        M.reset_options()
        for key, val in dict(DEFAULTS, **opts).items():
            M.set_option(key, val)
        M.init(m, n, k, 3)
        assert M.get_option("blocked_pairs") == -1
        dS = M.samples_to_device(S)
        if scheme != "hogwild":
            M.plan(dS, s)
        M.epoch(dS, 0.01, 0.05, 0.04, scheme)
        return M.get_option("blocked_pairs")

    assert last(uni, 128, "wavefront") == 1
    assert last(hot, 128, "wavefront") == 0
    assert last(uni, 128, "wavefront", half_waves=0) == 0
    assert last(hot, 128, "wavefront", half_waves=2) == 1
    assert last(uni, 128, "wavefront_det") == 0
    assert last(uni, 32, "hogwild", partition=1, hogwild_grid=8) == 1
    assert last(uni, 128, "hogwild") == -1


def test_half_workers_choice(M):
    """Read-only key half_workers: two workers per wavefront at k <= 32 by
    default; at every width of at most 16 bytes per lane with half_waves = 2;
    never with 0."""
    cases = [(1, 0, 32, 1), (1, 1, 32, 1), (1, 0, 64, 0), (1, 0, 128, 0), (1, 1, 64, 0), (1, 1, 128, 0),
             (1, 1, 256, 0), (2, 0, 128, 1), (2, 0, 256, 0), (2, 1, 256, 1), (2, 1, 512, 0), (0, 0, 32, 0),
             (0, 1, 128, 0)]
    for half, dtype, k, want in cases:
        M.reset_options()
        for key, val in dict(DEFAULTS, dtype=dtype, half_waves=half).items():
            M.set_option(key, val)
        M.init(50, 40, k, 1)
        assert M.get_option("half_workers") == want, (half, dtype, k)
