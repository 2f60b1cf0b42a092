"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Each test checks the oracle against a published value, a hand-worked fixture,
a closed form, an exact invariant or brute force on a tiny input, chosen so
that a plausible slip (a dropped term, a wrong sign or index, a transposed
operand, an off-by-one in the schedule) fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workloads import gaussian_mixture, epoch_orders

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def sched(lr, sigma, lr1=None, sigma1=None, lr_decay=oracle.LINEAR,
          sigma_decay=oracle.EXPONENTIAL):
    return oracle.schedule(lr, lr if lr1 is None else lr1, sigma,
                           sigma if sigma1 is None else sigma1, lr_decay,
                           sigma_decay)


# --------------------------------------------------------------- generator
def test_splitmix64_published_check_values():
    g = _gold("splitmix64_seed0.json")
    out = oracle.splitmix64(g["seed"], len(g["outputs_hex"]))
    assert [f"{int(v):016x}" for v in out] == g["outputs_hex"]


def test_init_uniform_is_top_24_bits_on_grid():
    g = _gold("splitmix64_seed0.json")
    W = oracle.init_uniform(0, 1, 3)
    want = [int(h, 16) >> 40 for h in g["outputs_hex"]]
    assert (W.ravel() * 2**24).tolist() == [float(v) for v in want]
    big = oracle.init_uniform(7, 100, 1000)
    assert big.min() >= 0.0 and big.max() < 1.0
    assert np.all(big * 2**24 == np.floor(big * 2**24))
    assert np.all(big.astype(np.float32).astype(np.float64) == big)
    assert abs(big.mean() - 0.5) < 5e-3
    # element i of the map is output i of the stream: row-major (u, j)
    assert np.array_equal(oracle.init_uniform(7, 10, 100).ravel(), big.ravel()[:1000])


def test_shuffle_is_uniform_permutation():
    for n in (1, 2, 5, 1000):
        p = oracle.shuffle(3, 11, n)
        assert sorted(p.tolist()) == list(range(n))
    counts = {}
    for e in range(6000):
        key = tuple(oracle.shuffle(1, e, 3).tolist())
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 6
    assert all(abs(c - 1000) < 150 for c in counts.values())
    assert not np.array_equal(oracle.shuffle(0, 0, 50), oracle.shuffle(0, 1, 50))


# --------------------------------------------------------------- schedule
def test_schedule_endpoints_and_midpoints():
    s = sched(0.5, 10.0, lr1=0.01, sigma1=1.0)
    T = 101
    assert oracle.schedule_at(0, T, s) == (0.5, 10.0)
    assert oracle.schedule_at(T - 1, T, s) == (0.01, 1.0)
    lr, sg = oracle.schedule_at(50, T, s)
    assert lr == pytest.approx(0.255, rel=1e-15)          # arithmetic mean
    assert sg == pytest.approx(math.sqrt(10.0), rel=1e-15)  # geometric mean
    lr, sg = oracle.schedule_at(25, T, s)
    assert lr == pytest.approx(0.5 - 0.49 / 4, rel=1e-15)
    assert sg == pytest.approx(10.0 ** 0.75, rel=1e-15)
    # a single-step schedule sits at its start
    assert oracle.schedule_at(0, 1, s) == (0.5, 10.0)
    # exponential learning rate and linear radius are also available
    s2 = sched(0.5, 10.0, lr1=0.005, sigma1=2.0, lr_decay=oracle.EXPONENTIAL,
               sigma_decay=oracle.LINEAR)
    lr, sg = oracle.schedule_at(1, 3, s2)
    assert lr == pytest.approx(0.05, rel=1e-15) and sg == pytest.approx(6.0, rel=1e-15)
    # equal endpoints are constant, also for an infinite radius
    s3 = sched(0.25, math.inf)
    assert oracle.schedule_at(7, 10, s3) == (0.25, math.inf)


# --------------------------------------------------------------- lattice
def test_lattice_positions_and_neighbour_counts():
    assert oracle.position(oracle.RECT, 7, 0) == (0.0, 0.0)
    assert oracle.position(oracle.RECT, 7, 9) == (1.0, 2.0)
    y, x = oracle.position(oracle.HEX, 7, 9)
    assert x == 2.5 and y == pytest.approx(math.sqrt(3) / 2)
    assert oracle.position(oracle.HEX, 7, 14) == (pytest.approx(math.sqrt(3)), 0.0)
    for topo, want in ((oracle.RECT, 4), (oracle.HEX, 6)):
        rows, cols = 7, 7
        c = 3 * cols + 3
        cy, cx = oracle.position(topo, cols, c)
        near = 0
        for u in range(rows * cols):
            if u == c:
                continue
            y, x = oracle.position(topo, cols, u)
            if math.hypot(y - cy, x - cx) <= 1 + 1e-9:
                near += 1
        assert near == want


def test_gaussian_neighbourhood_values():
    rows, cols = 5, 5
    c = 12  # centre (2, 2)
    sigma = 1 / math.sqrt(2)  # so that h = lr * e^{-g}
    h = oracle.neighbourhood(rows, cols, oracle.RECT, c, 1.0, sigma)
    assert h[c] == 1.0
    assert h[13] == pytest.approx(0.36787944117144233, rel=1e-14)   # e^-1
    assert h[18] == pytest.approx(0.1353352832366127, rel=1e-14)    # e^-2
    assert h[14] == pytest.approx(0.01831563888873418, rel=1e-13)   # e^-4
    h2 = oracle.neighbourhood(rows, cols, oracle.RECT, c, 0.25, sigma)
    assert h2[c] == 0.25 and h2[13] == pytest.approx(0.25 / math.e, rel=1e-14)
    # symmetry h(u; c) = h(c; u)
    for a in range(25):
        ha = oracle.neighbourhood(rows, cols, oracle.HEX, a, 0.3, 1.7)
        for b in range(25):
            hb = oracle.neighbourhood(rows, cols, oracle.HEX, b, 0.3, 1.7)
            assert ha[b] == hb[a]
    # radius 0: Kronecker delta; infinite radius: lr everywhere
    z = oracle.neighbourhood(rows, cols, oracle.RECT, 7, 0.4, 0.0)
    assert z[7] == 0.4 and np.count_nonzero(z) == 1
    assert np.all(oracle.neighbourhood(rows, cols, oracle.RECT, 7, 0.4, math.inf) == 0.4)


# --------------------------------------------------------------- competition
def test_tiny_map_hand_worked():
    g = _gold("tiny_map_2x2.json")
    W = np.array(g["W"], dtype=np.float64)
    x = np.array([g["x"]], dtype=np.float32)
    D = oracle.distances(W, x[0])
    assert D.tolist() == g["squared_distances"]
    ev = oracle.evaluate(W, g["rows"], g["cols"], x)
    assert ev["c1"][0] == g["bmu"] and ev["c2"][0] == g["second_bmu"]
    assert ev["qe"] == g["qe"] and ev["te"] == g["te"]


def test_bmu_brute_force_tiny_maps():
    rng = np.random.default_rng(5)
    for rows, cols, d in ((2, 2, 1), (3, 3, 4), (2, 5, 3), (1, 7, 2)):
        W = rng.integers(-4, 5, size=(rows * cols, d)).astype(np.float64) / 4
        X = (rng.integers(-8, 9, size=(40, d)) / 8).astype(np.float32)
        ev = oracle.evaluate(W, rows, cols, X)
        for i in range(X.shape[0]):
            D = [sum((float(X[i, j]) - W[u, j]) ** 2 for j in range(d))
                 for u in range(rows * cols)]
            best = min(range(len(D)), key=lambda u: (D[u], u))
            second = min((u for u in range(len(D)) if u != best),
                         key=lambda u: (D[u], u))
            assert ev["c1"][i] == best and ev["c2"][i] == second
            assert ev["d1"][i] == D[best] and ev["d2"][i] == D[second]


def test_exact_ties_break_to_lowest_index():
    W = np.array([[0.5, 0.5], [1.0, 0.0], [0.5, 0.5], [1.0, 0.0]])
    X = np.array([[0.5, 0.5], [1.0, 0.0], [0.75, 0.25]], dtype=np.float32)
    ev = oracle.evaluate(W, 2, 2, X)
    assert ev["c1"].tolist() == [0, 1, 0]
    assert ev["c2"].tolist() == [2, 3, 1]
    # the training step takes the same winner
    s = sched(1.0, 0.0)
    W1, tr = oracle.train(W, 2, 2, X[2:3], np.array([0]), s, trace=True)
    assert tr.tolist() == [0]
    assert W1[0].tolist() == [0.75, 0.25] and W1[2].tolist() == [0.5, 0.5]


def test_line_map_nearest_point_and_topographic_error():
    N = 9
    W = np.arange(N, dtype=np.float64)[:, None]
    X = np.array([[3.25], [0.0], [8.75], [-2.0], [5.5]], dtype=np.float32)
    ev = oracle.evaluate(W, 1, N, X)
    assert ev["c1"].tolist() == [3, 0, 8, 0, 5]
    assert ev["c2"].tolist() == [4, 1, 7, 1, 6]    # 5.5: tie 5 / 6 -> 5 first
    assert ev["te"] == 0.0
    assert ev["qe"] == pytest.approx((0.25 + 0 + 0.75 + 2 + 0.5) / 5, rel=1e-15)
    # swap prototypes 2 and 6: samples near 2 and 6 now have far second BMUs
    Ws = W.copy()
    Ws[[2, 6]] = Ws[[6, 2]]
    X2 = np.array([[2.25], [6.25], [4.0], [0.25]], dtype=np.float32)
    ev2 = oracle.evaluate(Ws, 1, N, X2)
    # 2.25 -> unit 6 (value 2), second unit 3 (value 3): |6-3| = 3 > 1
    # 6.25 -> unit 2 (value 6), second unit 7 (value 7): |2-7| = 5 > 1
    # 4.00 -> unit 4, second unit 3 (tie 3 / 5): adjacent
    # 0.25 -> unit 0, second unit 1: adjacent
    assert ev2["c1"].tolist() == [6, 2, 4, 0]
    assert ev2["c2"].tolist() == [3, 7, 3, 1]
    assert ev2["te"] == 0.5


def test_qe_zero_when_every_sample_is_a_prototype():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((12, 7)).astype(np.float32)
    ev = oracle.evaluate(X.astype(np.float64), 3, 4, X)
    assert ev["qe"] == 0.0
    assert ev["c1"].tolist() == list(range(12))


def test_single_unit_map_has_no_topographic_error():
    X = np.ones((3, 2), dtype=np.float32)
    ev = oracle.evaluate(np.zeros((1, 2)), 1, 1, X)
    assert ev["te"] == 0.0 and ev["c2"].tolist() == [-1, -1, -1]
    assert ev["qe"] == pytest.approx(math.sqrt(2), rel=1e-15)


# --------------------------------------------------------------- adaptation
def test_radius_zero_moves_only_the_bmu_by_lr_times_difference():
    rng = np.random.default_rng(7)
    W = (rng.integers(0, 64, size=(12, 5)) / 64).astype(np.float64)
    X = (rng.integers(0, 64, size=(1, 5)) / 64).astype(np.float32)
    s = sched(0.25, 0.0)
    W1, tr = oracle.train(W, 3, 4, X, np.array([0]), s, trace=True)
    c = tr[0]
    assert c == int(np.argmin(((X[0].astype(np.float64) - W) ** 2).sum(1)))
    others = np.arange(12) != c
    assert np.array_equal(W1[others], W[others])
    assert np.array_equal(W1[c], W[c] + 0.25 * (X[0] - W[c]))


def test_unit_learning_rate_radius_zero_copies_the_sample_exactly():
    rng = np.random.default_rng(8)
    W = rng.random((20, 33)).astype(np.float32).astype(np.float64)
    X = rng.standard_normal((4, 33)).astype(np.float32)
    s = sched(1.0, 0.0)
    W1, tr = oracle.train(W, 4, 5, X, np.array([2]), s, trace=True)
    assert np.array_equal(W1[tr[0]], X[2].astype(np.float64))


def test_infinite_radius_contracts_pairwise_differences():
    rng = np.random.default_rng(9)
    W = rng.random((6, 10))
    X = rng.random((1, 10)).astype(np.float32)
    lr = 0.375
    W1, _ = oracle.train(W, 2, 3, X, np.array([0]), sched(lr, math.inf))
    for a in range(6):
        for b in range(6):
            np.testing.assert_allclose(W1[a] - W1[b], (1 - lr) * (W[a] - W[b]),
                                       rtol=0, atol=1e-15)
    # and every prototype moved toward the sample by the same fraction
    np.testing.assert_allclose(W1 - X[0], (1 - lr) * (W - X[0]), rtol=0, atol=1e-15)


def test_single_unit_map_is_an_exponential_moving_average():
    # w_T = (1 - a)^T w_0 + sum_k a (1 - a)^(T-1-k) x_k, exact in rationals
    a = Fraction(1, 4)
    xs = [Fraction(k, 16) for k in (3, -5, 11, 0, 7, 15, -16, 2, 9, 1)]
    X = np.array([[float(v), float(-v)] for v in xs], dtype=np.float32)
    w0 = Fraction(5, 8)
    W0 = np.array([[float(w0), float(-w0)]])
    T = len(xs)
    want = (1 - a) ** T * w0 + sum(a * (1 - a) ** (T - 1 - k) * xs[k] for k in range(T))
    W1, tr = oracle.train(W0, 1, 1, X, np.arange(T), sched(0.25, 3.0))
    assert W1[0, 0] == float(want) and W1[0, 1] == -float(want)


def test_translation_invariance():
    rng = np.random.default_rng(10)
    X = (rng.integers(0, 256, size=(30, 6)) / 256).astype(np.float32)
    W = rng.integers(0, 256, size=(16, 6)) / 256
    shift = np.array([4.0, -2.0, 8.0, 1.0, -16.0, 0.5])
    order = np.tile(np.arange(30), 2).astype(np.int32)
    s = oracle.schedule(0.5, 0.25, 2.0, 0.5)
    W1, t1 = oracle.train(W, 4, 4, X, order, s, trace=True)
    W2, t2 = oracle.train(W + shift, 4, 4, (X + shift).astype(np.float32), order, s,
                          trace=True)
    assert np.array_equal(t1, t2)
    np.testing.assert_allclose(W2 - shift, W1, rtol=0, atol=1e-12)


# --------------------------------------------------------------- trajectory
def test_thread_count_and_resume_do_not_change_bits():
    X = gaussian_mixture(64, 24, 4, 0.1, seed=3)
    W0 = oracle.init_uniform(1, 25, 24)
    order = epoch_orders(64, 5, seed=2)
    s = oracle.schedule(0.5, 0.01, 3.0, 0.5)
    Wa, ta = oracle.train(W0, 5, 5, X, order, s, nthreads=1, trace=True)
    Wb, tb = oracle.train(W0, 5, 5, X, order, s, nthreads=4, trace=True)
    assert np.array_equal(Wa, Wb) and np.array_equal(ta, tb)
    T = order.shape[0]
    Wc, _ = oracle.train(W0, 5, 5, X, order[:128], s, step0=0, total_steps=T)
    Wc, _ = oracle.train(Wc, 5, 5, X, order[128:], s, step0=128, total_steps=T)
    assert np.array_equal(Wa, Wc)


def test_quantization_error_non_increasing_on_separated_mixture():
    X = gaussian_mixture(400, 16, 4, 0.02, seed=11)
    W = oracle.init_uniform(0, 36, 16)
    s = oracle.schedule(0.5, 0.01, 3.0, 0.5)
    epochs = 6
    T = epochs * 400
    qes = [oracle.evaluate(W, 6, 6, X)["qe"]]
    for e in range(epochs):
        order = epoch_orders(400, 1, seed=1, first_epoch=e)
        W, _ = oracle.train(W, 6, 6, X, order, s, step0=e * 400, total_steps=T)
        qes.append(oracle.evaluate(W, 6, 6, X)["qe"])
    assert all(b <= a + 1e-12 for a, b in zip(qes, qes[1:])), qes
    assert qes[-1] < 0.1 * qes[0]


# ------------------------------------------------- near-tie coin trainings
def test_near_tie_training_without_ties_is_the_plain_training():
    """With tie_rel = 0 only exact ties are coin candidates; on data with
    none, every seed reproduces the plain training bit for bit."""
    X = gaussian_mixture(64, 24, 4, 0.1, seed=3)
    W0 = oracle.init_uniform(1, 25, 24)
    order = epoch_orders(64, 3, seed=2)
    s = oracle.schedule(0.5, 0.01, 3.0, 0.5)
    Wa, _ = oracle.train(W0, 5, 5, X, order, s)
    for seed in (0, 1, 99):
        Wb, flips = oracle.train_near_tie(W0, 5, 5, X, order, s, 0.0, seed)
        assert flips == 0 and np.array_equal(Wa, Wb)


def test_near_tie_training_flips_exact_ties_by_the_published_generator():
    """Two identical prototypes tie exactly at every step.  With sigma = 0
    and lr = 1 the chosen unit becomes the sample; the plain rule always
    takes unit 0, the coin rule takes unit 1 exactly at the steps whose
    SplitMix64 output (checked against its published values elsewhere) has
    its top bit set."""
    X = np.array([[1.0, 2.0], [3.0, -1.0], [0.5, 0.25]], dtype=np.float32)
    W0 = np.zeros((2, 2))
    s = sched(1.0, 0.0)
    seed = 12345
    bits = oracle.splitmix64(seed, 64) >> np.uint64(63)
    for t in range(40):
        order = np.array([t % 3], dtype=np.int32)
        W, flips = oracle.train_near_tie(W0, 1, 2, X, order, s, 0.0, seed, step0=t,
                                         total_steps=64)
        moved = 1 if bits[t] else 0
        assert flips == moved
        assert np.array_equal(W[moved], X[t % 3].astype(np.float64))
        assert np.array_equal(W[1 - moved], W0[1 - moved])
        Wp, _ = oracle.train(W0, 1, 2, X, order, s, step0=t, total_steps=64)
        assert np.array_equal(Wp[0], X[t % 3].astype(np.float64))


def test_near_tie_threshold_is_relative_to_the_smaller_distance():
    """A 1 x 2 map whose units sit at squared distances 1 and 1 + 1e-7 from
    the sample: a near tie for tie_rel >= 1e-7, not for 1e-8."""
    X = np.zeros((1, 1), dtype=np.float32)
    W0 = np.array([[1.0], [-math.sqrt(1.0 + 1e-7)]])
    D = oracle.distances(W0, X[0])
    rel = (D[1] - D[0]) / D[0]
    assert 0.99e-7 < rel < 1.01e-7
    s = sched(1.0, 0.0)
    bits = oracle.splitmix64(7, 32) >> np.uint64(63)
    order = np.zeros(32, dtype=np.int32)
    # lr = 1, sigma = 0 would move the chosen unit onto the sample and end
    # the tie, so every step is taken from the same state
    for t in range(32):
        _, f_wide = oracle.train_near_tie(W0, 1, 2, X, order[t:t + 1], s, 2e-7, 7, step0=t,
                                          total_steps=32)
        _, f_narrow = oracle.train_near_tie(W0, 1, 2, X, order[t:t + 1], s, 1e-8, 7,
                                            step0=t, total_steps=32)
        assert f_wide == int(bits[t]) and f_narrow == 0


def test_argument_errors():
    X = np.zeros((2, 3), dtype=np.float32)
    W = np.zeros((4, 3))
    with pytest.raises(ValueError):
        oracle.train(W, 2, 2, X, np.array([5]), sched(0.1, 1.0))
    with pytest.raises(ValueError):
        oracle.train_near_tie(W, 2, 2, X, np.array([0]), sched(0.1, 1.0), -1.0, 0)
    with pytest.raises(ValueError):
        oracle.train_near_tie(W, 2, 2, X, np.array([0]), sched(0.1, 1.0), float("nan"), 0)


# ------------------------------------------------------------ linear init (Sec. 6D, Fig. 2)
def _planar_data():
    """Rows mu + 3 s_i e1 + t_i e4 with s, t two orthogonal +-1 patterns of
    mean zero (Walsh rows of length 64): exactly representable, with
    covariance 9 e1 e1^T + e4 e4^T."""
    i = np.arange(64)
    s = np.where((i & 1) == 0, 1.0, -1.0)
    t = np.where((i & 2) == 0, 1.0, -1.0)
    assert s.sum() == 0 and t.sum() == 0 and (s * t).sum() == 0
    mu = np.array([1.0, 2.0, -3.0, 4.0, 0.5, 6.0])
    X = mu + 3.0 * np.outer(s, np.eye(6)[1]) + np.outer(t, np.eye(6)[4])
    return X.astype(np.float32), mu


def test_pca_of_planar_data_recovers_its_axes():
    X, mu = _planar_data()
    lam, V, m = oracle.pca_top2(X)
    assert np.allclose(lam, [9.0, 1.0], rtol=0, atol=1e-12)
    assert np.allclose(V[:, 0], np.eye(6)[1], atol=1e-12)
    assert np.allclose(V[:, 1], np.eye(6)[4], atol=1e-12)
    assert np.array_equal(m, mu)


def test_pca_sign_convention_and_definition():
    rng = np.random.default_rng(3)
    X = (rng.standard_normal((300, 12)) @ rng.standard_normal((12, 12))).astype(np.float32)
    lam, V, mu = oracle.pca_top2(X)
    Xc = X.astype(np.float64) - mu
    Cov = Xc.T @ Xc / X.shape[0]
    for a in range(2):
        v = V[:, a]
        assert abs(np.linalg.norm(v) - 1.0) < 1e-12
        assert np.linalg.norm(Cov @ v - lam[a] * v) <= 1e-9 * lam[0]
        k = int(np.argmax(np.abs(v)))
        assert v[k] > 0
    assert lam[0] >= lam[1] >= 0 and abs(V[:, 0] @ V[:, 1]) < 1e-12
    # no direction has more variance than the first component
    for u in rng.standard_normal((20, 12)):
        u /= np.linalg.norm(u)
        assert u @ Cov @ u <= lam[0] * (1 + 1e-12)


def test_map_size_heuristic_by_hand():
    # m = 100: munits = ceil(5 * 10) = 50.  lambda = (4, 1): 1 * 50 >= 4, so
    # r = 2; sqrt(50 / (2 * 0.8660)) = 5.37 -> 5; ceil(50 / 5) = 10;
    # iterations ceil(50 * 50 / 100) * 100 * 4 = 25 * 400.
    assert oracle.suggest_size(100, 4.0, 1.0) == (5, 10, 10000)
    # lambda1 > lambda2 * munits (and lambda1 = 0): r = 1;
    # sqrt(50 / 0.8660) = 7.60 -> 8; ceil(50 / 8) = 7; ceil(50 * 56 / 100) = 28.
    assert oracle.suggest_size(100, 1000.0, 1.0) == (7, 8, 11200)
    assert oracle.suggest_size(100, 0.0, 0.0) == (7, 8, 11200)
    # m = 2000: munits = ceil(223.6) = 224; r = sqrt(2);
    # sqrt(224 / (1.4142 * 0.8660)) = 13.52 -> 14; ceil(224 / 14) = 16;
    # ceil(50 * 224 / 2000) = ceil(5.6) = 6 -> 6 * 2000 * 4.
    assert oracle.suggest_size(2000, 2.0, 1.0) == (14, 16, 48000)
    # equal variances: r = 1 as in the second case
    assert oracle.suggest_size(100, 1.0, 1.0) == (7, 8, 11200)


def test_linear_init_spans_one_standard_deviation_per_component():
    X, mu = _planar_data()
    lam, V, m = oracle.pca_top2(X)
    W = oracle.linear_init(m, lam, V, 3, 4)
    e1, e4 = np.eye(6)[1], np.eye(6)[4]
    assert np.allclose(W[0], mu - 3.0 * e1 - e4, atol=1e-12)
    assert np.allclose(W[11], mu + 3.0 * e1 + e4, atol=1e-12)
    for c, a in enumerate((-1.0, -1.0 / 3.0, 1.0 / 3.0, 1.0)):
        assert np.allclose(W[4 + c], mu + 3.0 * a * e1, atol=1e-12)   # middle row
    W1 = oracle.linear_init(m, lam, V, 1, 3)
    assert np.allclose(W1[1], mu, atol=1e-12)                          # single row, centre
    assert np.allclose(W1[0], mu - 3.0 * e1, atol=1e-12)


# ------------------------------------------------------------------ batch map
def test_batch_radius_zero_is_a_k_means_step():
    # sigma = 0: each prototype becomes the mean of the samples whose BMU it
    # is; a unit without samples keeps its prototype (worked by hand)
    X = np.array([[0, 0], [0, 1], [4, 4], [5, 5], [10, 0]], np.float32)
    W = np.array([[0, 0.2], [4.5, 4.4], [9, 1], [20, 20]], np.float64)
    W1, b = oracle.train_batch(W, 2, 2, X, 1, 0.0, 0.0, trace=True)
    assert list(b[0]) == [0, 0, 1, 1, 2]
    assert np.array_equal(W1, [[0, 0.5], [4.5, 4.5], [10, 0], [20, 20]])


def test_batch_infinite_radius_gives_every_unit_the_global_mean():
    X = gaussian_mixture(40, 6, 3, 0.3, seed=8)
    W = oracle.init_uniform(2, 12, 6)
    W1, _ = oracle.train_batch(W, 3, 4, X, 1, math.inf, math.inf)
    mean = X.astype(np.float64).mean(0)
    assert np.allclose(W1, np.broadcast_to(mean, W1.shape), rtol=0, atol=1e-12)


def test_batch_two_unit_map_by_hand():
    # samples a (3 copies) and b (2 copies) on a 1 x 2 map, a -> unit 0 and
    # b -> unit 1; with h = exp(-1 / (2 sigma^2)) for the lattice neighbour,
    # w0 = (3a + 2hb) / (3 + 2h) and w1 = (3ha + 2b) / (3h + 2)
    a, b = np.array([1.0, 2.0]), np.array([5.0, -1.0])
    X = np.array([a, a, a, b, b], np.float32)
    W = np.array([[1.5, 2.0], [4.0, -1.0]])
    sigma = 0.8
    h = math.exp(-1.0 / (2 * sigma * sigma))
    W1, _ = oracle.train_batch(W, 1, 2, X, 1, sigma, sigma)
    assert np.allclose(W1[0], (3 * a + 2 * h * b) / (3 + 2 * h), rtol=1e-14)
    assert np.allclose(W1[1], (3 * h * a + 2 * b) / (3 * h + 2), rtol=1e-14)


def test_batch_radius_schedule_hits_its_endpoints():
    assert oracle.batch_sigma(0, 5, 4.0, 0.5) == 4.0
    assert oracle.batch_sigma(4, 5, 4.0, 0.5) == 0.5
    assert oracle.batch_sigma(0, 1, 4.0, 0.5) == 4.0
    mid = oracle.batch_sigma(2, 5, 4.0, 0.5, oracle.EXPONENTIAL)
    assert mid == pytest.approx(math.sqrt(4.0 * 0.5), rel=1e-15)
    assert oracle.batch_sigma(2, 5, 4.0, 0.5, oracle.LINEAR) == pytest.approx(2.25, rel=1e-15)
