"""Pins of the CPU oracle against facts that do not come from the oracle itself:
hand-worked examples, published test vectors, closed forms, invariants,
library routines for special cases and brute force on tiny inputs."""
import itertools
import json
import math
import os

import numpy as np
import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def samples(rows, orc):
    a = np.zeros(len(rows), dtype=orc.SAMPLE_DTYPE)
    for i, (u, v, r) in enumerate(rows):
        a[i] = (u, v, r)
    return a


# ---------------------------------------------------------------------------- single update
def test_k1_worked_example(orc):
    g = gold("k1_update.json")
    p, q = orc.sgd_step([g["p"]], [g["q"]], g["r"], g["lr"], g["lambda_p"], g["lambda_q"])
    assert p[0] == g["p_new"] and q[0] == g["q_new"]
    assert q[0] != g["q_new_if_q_used_updated_p"]


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_k1_worked_example_in_storage(orc, dtype):
    """The same update applied through an epoch over one sample, for each storage type
    (all values are exact in binary16)."""
    g = gold("k1_update.json")
    P = np.array([[g["p"]]], dtype=dtype)
    Q = np.array([[g["q"]]], dtype=dtype)
    orc.epoch_serial(P, Q, samples([(0, 0, g["r"])], orc), g["lr"], g["lambda_p"], g["lambda_q"])
    assert float(P[0, 0]) == g["p_new"] and float(Q[0, 0]) == g["q_new"]


def test_k2_worked_example(orc):
    g = gold("k2_update.json")
    p, q = orc.sgd_step(g["p"], g["q"], g["r"], g["lr"], g["lambda_p"], g["lambda_q"])
    assert list(p) == g["p_new"] and list(q) == g["q_new"]


def test_update_is_half_gradient_step(orc):
    """(p' - p)/lr equals minus half the gradient of the per-sample cost
    (r - p.q)^2 + lp |p|^2 + lq |q|^2, measured by central differences."""
    rng = np.random.default_rng(7)
    k = 6
    p0, q0 = rng.normal(size=k), rng.normal(size=k)
    r, lr, lp, lq = 1.7, 1e-3, 0.3, 0.11

    def cost(p, q):
        return (r - p @ q) ** 2 + lp * (p @ p) + lq * (q @ q)

    p1, q1 = orc.sgd_step(p0, q0, r, lr, lp, lq)
    h = 1e-6
    for j in range(k):
        e = np.zeros(k)
        e[j] = h
        gp = (cost(p0 + e, q0) - cost(p0 - e, q0)) / (2 * h)
        gq = (cost(p0, q0 + e) - cost(p0, q0 - e)) / (2 * h)
        assert (p1[j] - p0[j]) / lr == pytest.approx(-0.5 * gp, rel=1e-7, abs=1e-8)
        assert (q1[j] - q0[j]) / lr == pytest.approx(-0.5 * gq, rel=1e-7, abs=1e-8)


def test_transpose_symmetry(orc):
    """Swapping the roles of users and items (u<->v, P<->Q, lp<->lq) gives the
    mirrored result bit for bit: both vectors are updated from their old values."""
    rng = np.random.default_rng(3)
    m, n, k = 7, 5, 8
    P = rng.uniform(0, 0.4, (m, k)).astype(np.float32)
    Q = rng.uniform(0, 0.4, (n, k)).astype(np.float32)
    S = samples([(rng.integers(m), rng.integers(n), rng.normal() + 1) for _ in range(60)], orc)
    St = S.copy()
    St["u"], St["v"] = S["v"], S["u"]
    P1, Q1 = P.copy(), Q.copy()
    orc.epoch_serial(P1, Q1, S, 0.05, 0.02, 0.07)
    P2, Q2 = Q.copy(), P.copy()
    orc.epoch_serial(P2, Q2, St, 0.05, 0.07, 0.02)
    assert np.array_equal(P1, Q2) and np.array_equal(Q1, P2)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_lr_zero_is_identity(orc, dtype):
    rng = np.random.default_rng(1)
    m, n, k = 20, 15, 16
    P, Q = orc.init_factors(m, n, k, 99, dtype)
    S = samples([(rng.integers(m), rng.integers(n), rng.normal()) for _ in range(300)], orc)
    P1, Q1 = P.copy(), Q.copy()
    orc.epoch_serial(P1, Q1, S, 0.0, 0.05, 0.05)
    assert np.array_equal(P1, P) and np.array_equal(Q1, Q)
    P2, Q2 = P.copy(), Q.copy()
    orc.epoch_wavefront(P2, Q2, S, 0.0, 0.05, 0.05, 4, 99, 0)
    assert np.array_equal(P2, P) and np.array_equal(Q2, Q)


def test_zero_error_no_regularisation_is_identity(orc):
    P = np.array([[0.5, 0.25]], dtype=np.float32)
    Q = np.array([[2.0, 4.0]], dtype=np.float32)
    orc.epoch_serial(P, Q, samples([(0, 0, 2.0)], orc), 0.3, 0.0, 0.0)  # p.q = 2 exactly
    assert P.tolist() == [[0.5, 0.25]] and Q.tolist() == [[2.0, 4.0]]


def test_repeated_sample_fits_rating(orc):
    P = np.array([[0.1, 0.2, 0.3]], dtype=np.float64).astype(np.float32)
    Q = np.array([[0.3, 0.1, 0.2]], dtype=np.float32)
    S = samples([(0, 0, 2.5)] * 2000, orc)
    orc.epoch_serial(P, Q, S, 0.05, 0.0, 0.0)
    assert float(P[0].astype(np.float64) @ Q[0].astype(np.float64)) == pytest.approx(2.5, abs=1e-5)


def test_zero_padding_invariant(orc):
    """Padding k=100 with 28 zero columns: the first 100 columns evolve bit for bit
    as at k=100 and the padding stays exactly zero."""
    rng = np.random.default_rng(5)
    m, n = 30, 20
    P = rng.uniform(0, 0.1, (m, 100)).astype(np.float32)
    Q = rng.uniform(0, 0.1, (n, 100)).astype(np.float32)
    S = samples([(rng.integers(m), rng.integers(n), rng.uniform(1, 5)) for _ in range(500)], orc)
    Pp = np.zeros((m, 128), np.float32)
    Qp = np.zeros((n, 128), np.float32)
    Pp[:, :100], Qp[:, :100] = P, Q
    orc.epoch_serial(P, Q, S, 0.01, 0.05, 0.05)
    orc.epoch_serial(Pp, Qp, S, 0.01, 0.05, 0.05)
    assert np.array_equal(Pp[:, :100], P) and np.array_equal(Qp[:, :100], Q)
    assert not Pp[:, 100:].any() and not Qp[:, 100:].any()


def test_planted_noiseless_training_rmse_goes_to_zero(orc):
    """On an exactly rank-k rating matrix (every cell observed), serial SGD with
    no regularisation drives the training RMSE towards 0."""
    rng = np.random.default_rng(11)
    m, n, k = 40, 30, 3
    Ps, Qs = rng.normal(0, 0.7, (m, k)), rng.normal(0, 0.7, (n, k))
    cells = [(u, v) for u in range(m) for v in range(n)]
    rng.shuffle(cells)
    S = samples([(u, v, float(Ps[u] @ Qs[v])) for u, v in cells], orc)
    P = rng.uniform(0, 0.5, (m, k)).astype(np.float32)
    Q = rng.uniform(0, 0.5, (n, k)).astype(np.float32)
    hist = [orc.rmse(P, Q, S)]
    for _ in range(300):
        orc.epoch_serial(P, Q, S, 0.05, 0.0, 0.0)
        hist.append(orc.rmse(P, Q, S))
    assert hist[-1] < 0.01 * hist[0] and hist[-1] < 5e-3
    assert hist[5] < hist[0] and hist[-1] <= hist[5]


# ---------------------------------------------------------------------------- RMSE
def test_rmse_hand_example(orc):
    g = gold("rmse_hand.json")
    P = np.array(g["P"], np.float32)
    Q = np.array(g["Qt"], np.float32)
    S = samples(g["samples"], orc)
    assert orc.sq_errors(P, Q, S).tolist() == g["sq_errors"]
    assert orc.rmse(P, Q, S) == math.sqrt(g["rmse_squared"])


def test_rmse_special_cases(orc):
    rng = np.random.default_rng(2)
    S = samples([(rng.integers(5), rng.integers(4), rng.normal()) for _ in range(50)], orc)
    P0 = np.zeros((5, 8), np.float32)
    Q = rng.uniform(size=(4, 8)).astype(np.float32)
    # P = 0: every prediction is 0, so RMSE = sqrt(mean r^2)
    r = S["r"].astype(np.float64)
    assert orc.rmse(P0, Q, S) == pytest.approx(math.sqrt(float(np.mean(r * r))), rel=1e-15)
    assert orc.rmse(P0, Q, S[:0]) == 0.0
    # ratings that are exactly the predictions (dyadic values): RMSE 0
    P = np.full((5, 8), 0.5, np.float32)
    Q = np.full((4, 8), 0.25, np.float32)
    S2 = S.copy()
    S2["r"] = 1.0
    assert orc.rmse(P, Q, S2) == 0.0


# ---------------------------------------------------------------------------- binary16
def test_half_round_trip_exhaustive(orc):
    for b in range(65536):
        x = orc.half_to_double(b)
        if math.isnan(x):
            assert (b & 0x7c00) == 0x7c00 and (b & 0x3ff)
            continue
        assert orc.double_to_half(x) == b


def test_half_ties_to_even(orc):
    assert orc.double_to_half(1 + 2 ** -11) == 0x3C00  # tie between 1 and 1+2^-10 -> even (1)
    assert orc.double_to_half(1 + 3 * 2 ** -11) == 0x3C02  # tie -> 1 + 2^-9 (even)
    assert orc.double_to_half(65504.0) == 0x7BFF
    assert orc.double_to_half(65519.99) == 0x7BFF
    assert orc.double_to_half(65520.0) == 0x7C00
    assert orc.double_to_half(2 ** -25) == 0x0000  # tie between 0 and the smallest subnormal
    assert orc.double_to_half(3 * 2 ** -25) == 0x0002
    assert orc.double_to_half(-0.0) == 0x8000


def test_half_matches_numpy_conversion(orc):
    """numpy converts binary64 to binary16 with a single round-to-nearest-even."""
    rng = np.random.default_rng(0)
    xs = np.concatenate([rng.normal(0, 1, 20000), rng.normal(0, 1e-5, 5000), rng.normal(0, 3e4, 5000),
                         rng.uniform(0, 0.2, 20000)])
    with np.errstate(over="ignore"):
        ref = xs.astype(np.float16).view(np.uint16)
    got = np.array([orc.double_to_half(float(x)) for x in xs], dtype=np.uint16)
    assert np.array_equal(got, ref)


# ---------------------------------------------------------------------------- SplitMix64 / init
def test_splitmix64_published_vectors(orc):
    for vec in gold("splitmix64.json")["vectors"]:
        for i, o in enumerate(vec["outputs"]):
            assert orc.splitmix64(vec["seed"], i) == int(o, 0)


@pytest.mark.parametrize("k", [1, 32, 100, 128])
def test_init_range_and_moments(orc, k):
    P, Q = orc.init_factors(2000, 300, k, 12345, np.float32)
    hi = 1.0 / math.sqrt(k)
    for A in (P, Q):
        assert A.min() >= 0.0 and A.max() < hi
        assert float(A.mean()) == pytest.approx(0.5 * hi, rel=0.02)
        assert float(A.var()) == pytest.approx(hi * hi / 12, rel=0.05)
    assert not np.array_equal(P[:300], Q)  # distinct streams


def test_init_deterministic_and_half_consistent(orc):
    P1, Q1 = orc.init_factors(50, 40, 16, 7, np.float32)
    P2, Q2 = orc.init_factors(50, 40, 16, 7, np.float32)
    P3, _ = orc.init_factors(50, 40, 16, 8, np.float32)
    assert np.array_equal(P1, P2) and np.array_equal(Q1, Q2) and not np.array_equal(P1, P3)
    Ph, Qh = orc.init_factors(50, 40, 16, 7, np.float16)
    # binary16 init is the binary64 value rounded once; it lies within half a binary16 ulp
    # of the binary32 rounding of the same value
    ulp = np.spacing(Ph.astype(np.float16)).astype(np.float64)
    assert np.all(np.abs(Ph.astype(np.float64) - P1.astype(np.float64)) <= 0.5 * ulp + 1e-9)


# ---------------------------------------------------------------------------- schedules
def test_fisher_yates_is_uniform(orc):
    """All 3! orders appear with equal frequency over many streams (a Sattolo-style
    off-by-one would produce only the 2 cyclic permutations)."""
    counts = {}
    N = 60000
    for st in range(N):
        key = tuple(orc.fisher_yates(orc.splitmix64(424242, st), 3))
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 6
    for c in counts.values():
        assert abs(c - N / 6) < 5 * math.sqrt(N / 6)


@pytest.mark.parametrize("s", [1, 2, 5, 32, 64])
def test_sigma_is_latin_square(orc, s):
    for t in range(3):
        sig = orc.wavefront_sigma(2024, t, s)
        for i in range(s):
            assert sorted(sig[i]) == list(range(s))  # each worker visits every column once
            assert sorted(sig[:, i]) == list(range(s))  # in each wave, workers use distinct columns
    if s > 2:
        assert not np.array_equal(orc.wavefront_sigma(2024, 0, s), orc.wavefront_sigma(2024, 1, s))


def test_block_mapping(orc):
    m, n, s = 480189, 17770, 32
    assert orc.row_block(0, m, s) == 0 and orc.row_block(m - 1, m, s) == s - 1
    assert orc.col_block(0, n, s) == 0 and orc.col_block(n - 1, n, s) == s - 1
    # sizes of row blocks differ by at most one
    rows = np.bincount([orc.row_block(u, 1000, 7) for u in range(1000)])
    assert rows.max() - rows.min() <= 1 and rows.sum() == 1000


def test_block_order_is_stable_bucketing(orc):
    rng = np.random.default_rng(4)
    m, n, s = 53, 41, 4
    S = samples([(rng.integers(m), rng.integers(n), float(i)) for i in range(700)], orc)
    order, start = orc.block_order(S, m, n, s)
    assert sorted(order.tolist()) == list(range(700))
    for b in range(s * s):
        idx = order[start[b]:start[b + 1]]
        assert np.all(np.diff(idx) > 0)  # array order kept inside a block
        for i in idx:
            assert orc.row_block(S[i]["u"], m, s) * s + orc.col_block(S[i]["v"], n, s) == b


def _wavefront_sequence(orc, S, m, n, s, seed, t, reverse_workers=False, balanced=False):
    order, start = orc.block_order(S, m, n, s, balanced)
    sig = orc.wavefront_sigma(seed, t, s)
    seq = []
    for w in range(s):
        workers = range(s - 1, -1, -1) if reverse_workers else range(s)
        for i in workers:
            b = i * s + sig[i, w]
            seq.extend(order[start[b]:start[b + 1]].tolist())
    return np.array(seq, dtype=np.int64)


@pytest.mark.parametrize("balanced", [False, True])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_wavefront_blocks_commute(orc, dtype, balanced):
    """Blocks of one wave share no row and no column (independent samples,
    section 2.3), so the wavefront epoch equals a serial epoch over its schedule
    with the workers of every wave taken in either order."""
    rng = np.random.default_rng(9)
    m, n, k, s, seed = 64, 48, 8, 4, 77
    S = samples([(rng.integers(m), rng.integers(n), rng.uniform(1, 5)) for _ in range(3000)], orc)
    P, Q = orc.init_factors(m, n, k, seed, dtype)
    Pw, Qw = P.copy(), Q.copy()
    orc.epoch_wavefront(Pw, Qw, S, 0.02, 0.05, 0.05, s, seed, 3, balanced)
    for rev in (False, True):
        seq = _wavefront_sequence(orc, S, m, n, s, seed, 3, rev, balanced)
        assert sorted(seq.tolist()) == list(range(len(S)))
        Ps, Qs = P.copy(), Q.copy()
        orc.epoch_serial(Ps, Qs, S[seq], 0.02, 0.05, 0.05)
        assert np.array_equal(Ps, Pw) and np.array_equal(Qs, Qw)


def test_wavefront_single_block_is_serial(orc):
    rng = np.random.default_rng(12)
    S = samples([(rng.integers(20), rng.integers(10), rng.normal()) for _ in range(400)], orc)
    P, Q = orc.init_factors(20, 10, 4, 5, np.float32)
    P1, Q1, P2, Q2 = P.copy(), Q.copy(), P.copy(), Q.copy()
    orc.epoch_wavefront(P1, Q1, S, 0.05, 0.01, 0.02, 1, 5, 0)
    orc.epoch_serial(P2, Q2, S, 0.05, 0.01, 0.02)
    assert np.array_equal(P1, P2) and np.array_equal(Q1, Q2)


def test_two_by_two_blocking_feasible_orders(orc):
    """Brute force over the 24 orders of a 2 x 2 grid run by 2 workers: an order is
    feasible when each pair issued together is independent (no shared row or
    column).  Exactly 8 are, and every wavefront schedule is one of them."""
    g = gold("blocking_2x2.json")
    blocks = [(0, 0), (0, 1), (1, 0), (1, 1)]

    def indep(a, b):
        return a[0] != b[0] and a[1] != b[1]

    feasible = {o for o in itertools.permutations(blocks) if indep(o[0], o[1]) and indep(o[2], o[3])}
    assert len(list(itertools.permutations(blocks))) == g["orders"]
    assert len(feasible) == g["feasible"]
    seen = set()
    for t in range(40):
        sig = orc.wavefront_sigma(31337, t, 2)
        for w0 in (0, 1):  # the two workers of a wave may be issued in either order
            for w1 in (0, 1):
                o = ((w0, sig[w0, 0]), (1 - w0, sig[1 - w0, 0]), (w1, sig[w1, 1]), (1 - w1, sig[1 - w1, 1]))
                assert o in feasible
                seen.add(o)
    assert seen == feasible


def test_hogwild_single_worker_is_serial_order(orc):
    own = orc.hogwild_batch_owner(1000, 256, 1)
    assert own.tolist() == [0, 0, 0, 0]
    own = orc.hogwild_batch_owner(1025, 256, 3)
    assert own.tolist() == [0, 1, 2, 0, 1]


def _range_loads(counts, bounds):
    return [int(sum(counts[bounds[k]:bounds[k + 1]])) for k in range(len(bounds) - 1)]


def test_balanced_bounds_are_optimal(orc):
    """Brute force over every way of cutting a short index range into s consecutive
    (possibly empty) ranges: the oracle's cut reaches the smallest possible
    largest-range load, its ranges cover 0..N in order, and each index lands in
    its range."""
    rng = np.random.default_rng(21)
    for trial in range(40):
        N = int(rng.integers(1, 9))
        s = int(rng.integers(1, 5))
        nnz = int(rng.integers(0, 40))
        u = np.minimum(rng.zipf(1.5, nnz) - 1, N - 1) if nnz else np.zeros(0, int)
        S = samples([(int(x), 0, 1.0) for x in u], orc)
        counts = np.bincount(S["u"], minlength=N) if nnz else np.zeros(N, int)
        b = orc.balanced_bounds(S, N, 0, s).tolist()
        assert b[0] == 0 and b[-1] == N and all(x <= y for x, y in zip(b, b[1:]))
        best = min(max(_range_loads(counts, [0, *cuts, N]))
                   for cuts in itertools.combinations_with_replacement(range(N + 1), s - 1))
        assert max(_range_loads(counts, b)) == best
        for i in range(N):
            k = orc.bounded_block(i, b, s)
            assert b[k] <= i < b[k + 1]


def test_balanced_blocks_even_out_skew(orc, gen):
    """Netflix-shaped skew: equal index ranges leave a block row 1.5x heavier than
    the mean; the optimal contiguous cut brings it close to the mean."""
    w = gen.workload("netflix", ntrain=400_000, ntest=0)
    S = gen.draw(w, 0, w["ntrain"])
    s = 8
    for which, N, col in ((0, w["m"], "u"), (1, w["n"], "v")):
        counts = np.bincount(S[col], minlength=N)
        b = orc.balanced_bounds(S, N, which, s)
        loads = _range_loads(counts, b)
        assert sum(loads) == len(S)
        assert max(loads) / (len(S) / s) < 1.15  # users reach 1.01, items 1.12 (contiguous optimum)
        uniform = [int(np.sum(((S[col].astype(np.int64) * s) // N) == k)) for k in range(s)]
        assert max(uniform) / (len(S) / s) > 1.3


def test_balanced_wavefront_single_block_is_serial(orc):
    rng = np.random.default_rng(13)
    S = samples([(rng.integers(20), rng.integers(10), rng.normal()) for _ in range(400)], orc)
    P, Q = orc.init_factors(20, 10, 4, 5, np.float32)
    P1, Q1, P2, Q2 = P.copy(), Q.copy(), P.copy(), Q.copy()
    orc.epoch_wavefront(P1, Q1, S, 0.05, 0.01, 0.02, 1, 5, 0, True)
    orc.epoch_serial(P2, Q2, S, 0.05, 0.01, 0.02)
    assert np.array_equal(P1, P2) and np.array_equal(Q1, Q2)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_init_rows_equal_full_init(orc, dtype):
    P, Q = orc.init_factors(300, 70, 24, 31, dtype)
    rows = np.array([0, 299, 17, 17, 150])
    assert np.array_equal(orc.init_rows(300, 24, 31, 0, rows, dtype), P[rows])
    assert np.array_equal(orc.init_rows(70, 24, 31, 1, [69, 0, 5], dtype), Q[[69, 0, 5]])


# ---------------------------------------------------------------------------- global scheduling table
def test_table_order_is_a_permutation(orc):
    rng = np.random.default_rng(21)
    for nb in (0, 1, 2, 7, 100, 4096):
        blocks = np.sort(rng.choice(1 << 20, size=nb, replace=False))
        for t in (0, 5):
            o = orc.table_order(99, t, blocks)
            assert sorted(o.tolist()) == blocks.tolist()


def test_table_order_is_uniform(orc):
    """All 4! orders of four blocks appear equally often over the epochs (a draw
    over the full list instead of the blocks left, or a taken block not replaced
    by the list's last entry, repeats blocks or skews the orders)."""
    counts = {}
    N = 48000
    for t in range(N):
        key = tuple(orc.table_order(5150, t, [3, 9, 10, 17]).tolist())
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 24
    for c in counts.values():
        assert abs(c - N / 24) < 5 * math.sqrt(N / 24)


def test_table_order_keyed_by_seed_and_epoch(orc):
    b = np.arange(50) * 3
    a0 = orc.table_order(1, 0, b)
    assert np.array_equal(a0, orc.table_order(1, 0, b))
    assert not np.array_equal(a0, orc.table_order(1, 1, b))
    assert not np.array_equal(a0, orc.table_order(2, 0, b))
    assert not np.array_equal(a0, b)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_table_single_block_is_serial(orc, dtype):
    rng = np.random.default_rng(13)
    S = samples([(rng.integers(20), rng.integers(10), rng.normal()) for _ in range(400)], orc)
    P, Q = orc.init_factors(20, 10, 4, 5, dtype)
    P1, Q1, P2, Q2 = P.copy(), Q.copy(), P.copy(), Q.copy()
    orc.epoch_table(P1, Q1, S, 0.05, 0.01, 0.02, 1, 5, 3)
    orc.epoch_serial(P2, Q2, S, 0.05, 0.01, 0.02)
    assert np.array_equal(P1, P2) and np.array_equal(Q1, Q2)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_table_diagonal_blocks_commute(orc, dtype):
    """Samples only in the diagonal blocks (i, i): such blocks share no row and no
    column (independent samples, section 2.3), so in whatever order the table
    hands them out the epoch equals the serial epoch in array order."""
    rng = np.random.default_rng(14)
    m, n, k, s = 60, 45, 6, 5
    rows = []
    for x in range(2500):
        u = int(rng.integers(m))
        i = u * s // m
        lo, hi = -(-i * n // s), -(-(i + 1) * n // s)
        rows.append((u, int(rng.integers(lo, hi)), rng.uniform(1, 5)))
    S = samples(rows, orc)
    assert all(orc.row_block(x["u"], m, s) == orc.col_block(x["v"], n, s) for x in S)
    P, Q = orc.init_factors(m, n, k, 8, dtype)
    Ps, Qs = P.copy(), Q.copy()
    orc.epoch_serial(Ps, Qs, S, 0.03, 0.05, 0.04)
    for t in range(4):
        Pt, Qt = P.copy(), Q.copy()
        orc.epoch_table(Pt, Qt, S, 0.03, 0.05, 0.04, s, 8, t)
        assert np.array_equal(Pt, Ps) and np.array_equal(Qt, Qs)


def test_table_epoch_is_serial_over_its_schedule(orc):
    """Blocks in the table's order, each block's samples in array order (the
    stable bucketing pinned above), every sample exactly once."""
    rng = np.random.default_rng(15)
    m, n, k, s, seed, t = 70, 33, 5, 6, 41, 2
    S = samples([(rng.integers(m), rng.integers(n), rng.uniform(1, 5)) for _ in range(1500)], orc)
    order, start = orc.block_order(S, m, n, s)
    nonempty = [b for b in range(s * s) if start[b + 1] > start[b]]
    seq = np.concatenate([order[start[b]:start[b + 1]] for b in orc.table_order(seed, t, nonempty)])
    assert sorted(seq.tolist()) == list(range(len(S)))
    P, Q = orc.init_factors(m, n, k, seed, np.float32)
    P1, Q1, P2, Q2 = P.copy(), Q.copy(), P.copy(), Q.copy()
    orc.epoch_table(P1, Q1, S, 0.02, 0.05, 0.05, s, seed, t)
    orc.epoch_serial(P2, Q2, S[seq], 0.02, 0.05, 0.05)
    assert np.array_equal(P1, P2) and np.array_equal(Q1, Q2)
    P3, Q3 = P.copy(), Q.copy()
    orc.epoch_serial(P3, Q3, S, 0.02, 0.05, 0.05)
    assert not np.array_equal(P1, P3)  # the block order does change the result


def test_table_lr_zero_is_identity(orc):
    rng = np.random.default_rng(16)
    S = samples([(rng.integers(30), rng.integers(30), rng.normal()) for _ in range(600)], orc)
    P, Q = orc.init_factors(30, 30, 8, 2, np.float16)
    P1, Q1 = P.copy(), Q.copy()
    orc.epoch_table(P1, Q1, S, 0.0, 0.05, 0.05, 4, 2, 0)
    assert np.array_equal(P1, P) and np.array_equal(Q1, Q)


# ---------------------------------------------------------------------------- section 2.2 objective
def test_objective_hand_example(orc):
    g = gold("objective_hand.json")
    P = np.array(g["P"], dtype=np.float32)
    Q = np.array(g["Qt"], dtype=np.float32)
    S = samples(g["samples"], orc)
    assert orc.objective(P, Q, S, g["lambda_p"], g["lambda_q"]) == g["objective"]
    # one term per sample
    for row, term in zip(g["samples"], g["terms"]):
        assert orc.objective(P, Q, samples([row], orc), g["lambda_p"], g["lambda_q"]) == term


def test_objective_without_regularisation_is_sum_of_squared_errors(orc):
    """With lambda = 0 the cost is N * RMSE^2 over the same samples (ties the
    objective to the RMSE routine, written separately)."""
    rng = np.random.default_rng(11)
    m, n, k, N = 40, 30, 8, 500
    P = rng.normal(size=(m, k)).astype(np.float32)
    Q = rng.normal(size=(n, k)).astype(np.float32)
    S = np.zeros(N, dtype=orc.SAMPLE_DTYPE)
    S["u"], S["v"], S["r"] = rng.integers(0, m, N), rng.integers(0, n, N), rng.normal(size=N)
    obj = orc.objective(P, Q, S, 0.0, 0.0)
    assert obj == pytest.approx(N * orc.rmse(P, Q, S) ** 2, rel=1e-12)
    # the regularisers add lambda |row|^2 once per sample that uses the row
    lp, lq = 0.3, 0.7
    reg = sum(lp * float(np.dot(P[u].astype(np.float64), P[u])) + lq * float(np.dot(Q[v].astype(np.float64), Q[v]))
              for u, v in zip(S["u"], S["v"]))
    assert orc.objective(P, Q, S, lp, lq) == pytest.approx(obj + reg, rel=1e-12)


def test_update_descends_the_objective(orc):
    """A single-sample epoch moves (p, q) along minus half the gradient of that
    sample's cost, so for a small rate the objective drops by lr/2 times the
    squared gradient norm, up to a second-order term of relative size ~lr."""
    rng = np.random.default_rng(5)
    k = 8
    P = rng.normal(size=(1, k)).astype(np.float32)
    Q = rng.normal(size=(1, k)).astype(np.float32)
    r, lp, lq, lr = 0.9, 0.2, 0.4, 1e-3
    S = samples([(0, 0, r)], orc)
    p, q = P[0].astype(np.float64), Q[0].astype(np.float64)
    e = r - p @ q
    gp = -2 * e * q + 2 * lp * p
    gq = -2 * e * p + 2 * lq * q
    f0 = orc.objective(P, Q, S, lp, lq)
    orc.epoch_serial(P, Q, S, lr, lp, lq)
    f1 = orc.objective(P, Q, S, lp, lq)
    assert f0 - f1 == pytest.approx(0.5 * lr * (gp @ gp + gq @ gq), rel=2e-2)


# ---------------------------------------------------------------------------- OpenMP Hogwild! timing variant
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_openmp_hogwild_one_thread_is_serial(orc, dtype):
    """With one thread the batches are claimed in order, so the timing variant
    is the serial epoch bit for bit (ragged last batch included)."""
    rng = np.random.default_rng(3)
    m, n, k, N, f = 60, 45, 16, 3 * 256 + 77, 256
    P0, Q0 = orc.init_factors(m, n, k, 99, dtype)
    S = np.zeros(N, dtype=orc.SAMPLE_DTYPE)
    S["u"], S["v"], S["r"] = rng.integers(0, m, N), rng.integers(0, n, N), rng.normal(size=N)
    Pa, Qa, Pb, Qb = P0.copy(), Q0.copy(), P0.copy(), Q0.copy()
    orc.epoch_serial(Pa, Qa, S, 0.05, 0.02, 0.03)
    used = orc.epoch_hogwild_omp(Pb, Qb, S, 0.05, 0.02, 0.03, f=f, nthreads=1)
    assert used == 1
    assert np.array_equal(Pa.view(np.uint8), Pb.view(np.uint8)) and np.array_equal(Qa.view(np.uint8), Qb.view(np.uint8))


@pytest.mark.parametrize("f", [16, 64])
def test_openmp_hogwild_disjoint_batches_equal_serial(orc, f):
    """Several threads on batches whose rows are disjoint: every batch commutes
    with every other, so the result is the serial epoch bit for bit whatever
    the interleaving.  A batch run twice, a sample skipped or a batch bound
    off by one would change some row."""
    rng = np.random.default_rng(17)
    nb, k, ru, rv = 97, 8, 3, 2          # rows per batch: ru users, rv items
    N = nb * f - f // 2                  # ragged last batch
    m, n = nb * ru, nb * rv
    S = np.zeros(N, dtype=orc.SAMPLE_DTYPE)
    b = np.arange(N) // f
    S["u"] = b * ru + rng.integers(0, ru, N)
    S["v"] = b * rv + rng.integers(0, rv, N)
    S["r"] = rng.normal(size=N)
    P0, Q0 = orc.init_factors(m, n, k, 5, np.float32)
    Pa, Qa, Pb, Qb = P0.copy(), Q0.copy(), P0.copy(), Q0.copy()
    orc.epoch_serial(Pa, Qa, S, 0.1, 0.05, 0.05)
    used = orc.epoch_hogwild_omp(Pb, Qb, S, 0.1, 0.05, 0.05, f=f, nthreads=4)
    assert used == 4
    assert np.array_equal(Pa, Pb) and np.array_equal(Qa, Qb)
    # every row moved (no batch was skipped)
    assert (Pb != P0).any(axis=1).all() and (Qb != Q0).any(axis=1).all()


@pytest.mark.parametrize("balanced", [False, True])
def test_block_starts_equal_block_order_starts(orc, balanced):
    rng = np.random.default_rng(23)
    m, n, N, s = 300, 170, 20_000, 7
    S = np.zeros(N, dtype=orc.SAMPLE_DTYPE)
    S["u"] = (rng.zipf(1.6, N) - 1) % m
    S["v"] = rng.integers(0, n, N)
    order, start = orc.block_order(S, m, n, s, balanced=balanced)
    assert np.array_equal(orc.block_starts(S, m, n, s, balanced=balanced), start)
