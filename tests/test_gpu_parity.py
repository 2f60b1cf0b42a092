"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Criteria (per the workload contract):
  (1) BMU indices bit-exact on every sample whose oracle top-two relative
      gap (D2 - D1) / D1 exceeds 1e-4;
  (2) one training step from identical state: weights within 1e-5 max-abs;
  (3) after full training, QE and TE within 1 % relative of the oracle's.
"""
import math

import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import config, dev, golden, oracle_schedule, rel_gap, say, torch_cuda

pytestmark = pytest.mark.gpu

GAP = 1e-4
STEP_ATOL = 1e-5


def make_map(rows, cols, d, seed=0, topology=som.RECT, W=None):
    m = som.Map(rows, cols, d, seed=seed, topology=topology)
    if W is not None:
        m.weights = dev(np.asarray(W, dtype=np.float32))
    return m


# ------------------------------------------------------------ initialisation
@pytest.mark.parametrize("rows,cols,d,seed", [(10, 10, 500, 0), (3, 7, 37, 5),
                                              (1, 1, 1, 9), (20, 20, 2000, 0)])
def test_init_matches_oracle_bit_exact(rows, cols, d, seed):
    say("init", rows, cols, d, seed)
    m = make_map(rows, cols, d, seed)
    got = m.weights.cpu().numpy()
    want = oracle.init_uniform(seed, rows * cols, d).astype(np.float32)
    assert np.array_equal(got, want)
    m.close()


# ------------------------------------------------------------ batched BMU
def _bmu_case(rows, cols, d, n, seed, kind="tfidf"):
    if kind == "tfidf":
        X = workloads.small_tfidf(n, d, seed)
        W = workloads.random_weights(rows * cols, d, seed + 1, 0.0, 0.05)
        # put a few prototypes next to samples so the winners are not all ties
        k = min(rows * cols, n) // 2
        W[:k] = 0.7 * X[:k] + 0.3 * W[:k]
    else:
        X = workloads.gaussian_mixture(n, d, 8, 0.2, seed)
        W = workloads.random_weights(rows * cols, d, seed + 1, -1.0, 1.0)
    return X, W


@pytest.mark.parametrize("rows,cols,d,n,kind", [
    (10, 10, 500, 200, "tfidf"),        # tiny workload's shape
    (20, 20, 2000, 700, "tfidf"),       # several unit tiles, ragged sample tile
    (7, 9, 37, 130, "mixture"),         # d not a multiple of 4 or of the k slice
    (1, 1, 16, 5, "mixture"),           # one-unit map: no second BMU
    (1, 3, 8, 3, "mixture"),            # fewer units than candidates
    (30, 30, 5000, 300, "tfidf"),
    (100, 100, 2048, 256, "mixture"),   # stress workload's map and d
])
def test_batched_bmu_matches_oracle(rows, cols, d, n, kind):
    say("bmu", rows, cols, d, n, kind)
    torch = torch_cuda()
    X, W = _bmu_case(rows, cols, d, n, seed=rows * 31 + d)
    m = make_map(rows, cols, d, W=W)
    idx, idx2, d1 = m.bmu(dev(X), second=True)
    idx = idx.cpu().numpy()
    idx2 = idx2.cpu().numpy()
    d1 = d1.cpu().numpy()
    ev = oracle.evaluate(W.astype(np.float64), rows, cols, X)
    g1 = rel_gap(ev["d1"], ev["d2"])
    sure = g1 > GAP
    assert sure.mean() > 0.5
    assert np.array_equal(idx[sure], ev["c1"][sure])
    # everywhere: the chosen unit is within the gap of the true minimum
    assert np.all(np.abs(d1 - ev["d1"]) <= 1e-5 * np.maximum(ev["d1"], 1e-3) + 1e-6)
    if rows * cols == 1:
        assert np.all(idx2 == -1)
    else:
        # second BMU: exact where both of its gaps are clear
        D = np.stack([oracle.distances(W.astype(np.float64), X[i]) for i in range(n)])
        Ds = np.sort(D, axis=1)
        g2 = (Ds[:, 2] - Ds[:, 1]) / np.maximum(Ds[:, 1], 1e-300) if D.shape[1] > 2 \
            else np.full(n, np.inf)
        sure2 = sure & (g2 > GAP)
        assert np.array_equal(idx2[sure2], ev["c2"][sure2])
    # som_bmu alone gives the same indices
    only = m.bmu(dev(X)).cpu().numpy()
    assert np.array_equal(only, idx)
    torch.cuda.synchronize()
    m.close()


def test_exact_ties_resolve_to_lowest_index_on_gpu():
    W = np.array([[0.5, 0.5, 0, 0], [1, 0, 0, 0], [0.5, 0.5, 0, 0], [1, 0, 0, 0]],
                 dtype=np.float32)
    X = np.array([[0.5, 0.5, 0, 0], [1, 0, 0, 0], [0.75, 0.25, 0, 0]], dtype=np.float32)
    m = make_map(2, 2, 4, W=W)
    idx, idx2, _ = m.bmu(dev(X), second=True)
    assert idx.cpu().tolist() == [0, 1, 0]
    assert idx2.cpu().tolist() == [2, 3, 1]
    m.close()


# ------------------------------------------------------------ one step
@pytest.mark.parametrize("topology", [som.RECT, som.HEX])
@pytest.mark.parametrize("ci", [0, 1, 2, 3, 4])
def test_single_step_update_matches_oracle(ci, topology):
    """Criterion (2): one step from identical state, mid-schedule."""
    cfg = config(ci)
    say("single-step", cfg.name, "hex" if topology else "rect")
    X = workloads.make_data(cfg)
    rng = np.random.default_rng(ci)
    N = cfg.units
    # identical starting state: a partly trained-looking map
    W = oracle.init_uniform(cfg.init_seed, N, cfg.d).astype(np.float32)
    pick = rng.integers(0, cfg.n, size=N)
    W = (0.5 * W * 0.05 + 0.5 * X[pick]).astype(np.float32)
    i = int(rng.integers(0, cfg.n))
    T = cfg.steps
    for t in (0, T // 3, T - 1):
        m = make_map(cfg.rows, cfg.cols, cfg.d, W=W, topology=topology)
        # a one-step call of a T-step schedule: epochs * n must be 1 -> n = 1
        x1 = X[i:i + 1]
        trace = dev(np.full(1, -7, dtype=np.int32))
        m.train(dev(x1), 1, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                order=dev(np.zeros(1, dtype=np.int32)), step0=t, total_steps=T,
                bmu_trace=trace)
        got = m.weights.cpu().numpy()
        c_gpu = int(trace.cpu().numpy()[0])
        Wo, tr = oracle.train(W.astype(np.float64), cfg.rows, cfg.cols, x1,
                              np.zeros(1, dtype=np.int32), oracle_schedule(cfg),
                              step0=t, total_steps=T, topology=topology, trace=True)
        ev = oracle.evaluate(W.astype(np.float64), cfg.rows, cfg.cols, x1, topology=topology)
        if rel_gap(ev["d1"], ev["d2"])[0] > GAP:
            assert c_gpu == tr[0]
        if c_gpu == tr[0]:
            err = np.abs(got.astype(np.float64) - Wo).max()
            say(f"  t={t} bmu={c_gpu} max|dW|={err:.2e}")
            assert err <= STEP_ATOL
        m.close()


def test_radius_zero_unit_rate_copies_sample_exactly():
    X = workloads.gaussian_mixture(6, 37, 2, 0.3, seed=2)
    W = workloads.random_weights(12, 37, 3)
    m = make_map(3, 4, 37, W=W)
    trace = dev(np.full(1, -1, dtype=np.int32))
    m.train(dev(X[4:5]), 1, 1.0, 1.0, 0.0, 0.0, order=dev(np.zeros(1, np.int32)),
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
    m = make_map(3, 4, 8, W=W)
    trace = dev(np.full(1, -1, dtype=np.int32))
    m.train(dev(X), 1, 0.25, 0.25, 0.0, 0.0, order=dev(np.zeros(1, np.int32)),
            bmu_trace=trace)
    got = m.weights.cpu().numpy()
    c = int(trace.cpu().numpy()[0])
    want = W.copy()
    want[c] = W[c] + 0.25 * (X[0] - W[c])   # exact: dyadic values
    assert np.array_equal(got, want)
    m.close()


def test_infinite_radius_moves_every_unit_alike():
    W = workloads.random_weights(6, 10, 9)
    X = workloads.random_weights(1, 10, 10)
    m = make_map(2, 3, 10, W=W)
    m.train(dev(X), 1, 0.375, 0.375, math.inf, math.inf, order=dev(np.zeros(1, np.int32)))
    got = m.weights.cpu().numpy().astype(np.float64)
    want = W + 0.375 * (X[0] - W)
    assert np.abs(got - want).max() <= 1e-6
    m.close()


def test_near_duplicate_samples_in_one_block_keep_their_bmu():
    # With sigma = 0 and lr = 1 each step copies its sample into the BMU; the
    # next sample differs from it by ~1e-4 per element, so that unit is
    # closer than any other by orders of magnitude even though, in Gram
    # form, its fp32 distance is rounding noise around zero (possibly
    # negative).  Both samples of a pair fall in one block of steps.
    rng = np.random.default_rng(21)
    base = rng.random((8, 64)).astype(np.float32)
    X = np.empty((16, 64), np.float32)
    X[0::2] = base
    X[1::2] = base + (1e-4 * rng.standard_normal((8, 64))).astype(np.float32)
    W = workloads.random_weights(16, 64, 22)
    order = np.arange(16, dtype=np.int32)
    m = make_map(4, 4, 64, W=W)
    trace = dev(np.full(16, -1, dtype=np.int32))
    m.train(dev(X), 1, 1.0, 1.0, 0.0, 0.0, order=dev(order), bmu_trace=trace)
    got = trace.cpu().numpy()
    s = oracle.schedule(1.0, 1.0, 0.0, 0.0, oracle.LINEAR, oracle.LINEAR)
    Wo, tr = oracle.train(W, 4, 4, X, order, s, trace=True)
    assert np.array_equal(got, tr)
    assert np.array_equal(tr[1::2], tr[0::2])
    assert np.abs(m.weights.cpu().numpy() - Wo).max() == 0.0
    m.close()


# ------------------------------------------------------------ trajectories
def _trajectory_vs_oracle(ci, steps, topology):
    cfg = config(ci)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)[:steps]
    T = cfg.steps
    W0 = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed, topology=topology)
    trace = dev(np.full(steps, -1, dtype=np.int32))
    # som_train runs epochs * n steps: present the prefix as `steps` rows
    Xp = dev(X[order])
    m.train(Xp, 1, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
            order=dev(np.arange(steps, dtype=np.int32)), total_steps=T, bmu_trace=trace)
    got = trace.cpu().numpy()
    Wo, tr = oracle.train(W0, cfg.rows, cfg.cols, X, order, oracle_schedule(cfg),
                          total_steps=T, topology=topology, trace=True)
    first_diff = int(np.argmax(got != tr)) if np.any(got != tr) else steps
    say(f"  identical BMUs for {first_diff}/{steps} steps")
    if first_diff < steps:
        # a divergence is only allowed at a near tie of the oracle
        Wk, _ = oracle.train(W0, cfg.rows, cfg.cols, X, order[:first_diff],
                             oracle_schedule(cfg), total_steps=T, topology=topology)
        D = oracle.distances(Wk, X[order[first_diff]])
        Ds = np.sort(D)
        assert (Ds[1] - Ds[0]) / Ds[0] <= GAP, "divergence without a near tie"
    else:
        err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
        say(f"  final max|dW| = {err:.2e}")
        assert err <= 1e-4
    m.close()


@pytest.mark.parametrize("ci,steps,topology", [(0, 2000, som.RECT), (1, 600, som.RECT),
                                               (0, 400, som.HEX)])
def test_bmu_trajectory_matches_oracle_until_first_near_tie(ci, steps, topology):
    say("trajectory", config(ci).name, steps, "hex" if topology else "rect")
    _trajectory_vs_oracle(ci, steps, topology)


@pytest.mark.parametrize("ci,variant", [(0, "3"), (0, "4"), (1, "3"), (1, "4")])
def test_pipelined_variants_follow_the_oracle(ci, variant, monkeypatch):
    # variant 3 / 4: the kernel that overlaps the pass over the prototypes
    # with the grid exchanges (prototypes in LDS / streamed)
    monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    cfg = config(ci)
    m = som.Map(cfg.rows, cfg.cols, cfg.d)
    plan = m.plan()
    m.close()
    say("pipelined", cfg.name, plan)
    assert plan["variant"] == (3 if variant == "3" else 2)
    _trajectory_vs_oracle(ci, 600, som.RECT)


def test_resume_and_determinism_are_bitwise():
    cfg = config(0)
    X = dev(workloads.make_data(cfg))
    order = workloads.epoch_orders(cfg.n, 5, 0)
    o = dev(order)
    kw = dict(lr0=0.5, lr1=0.01, sigma0=5.0, sigma1=1.0)
    a = som.Map(10, 10, cfg.d, seed=0)
    a.train(X, 5, order=o, **kw)
    b = som.Map(10, 10, cfg.d, seed=0)
    b.train(X, 5, order=o, **kw)
    c = som.Map(10, 10, cfg.d, seed=0)
    T = 5 * cfg.n
    c.train(X, 2, order=dev(order[:2 * cfg.n]), total_steps=T, **kw)
    c.train(X, 3, order=dev(order[2 * cfg.n:]), step0=2 * cfg.n, total_steps=T, **kw)
    wa, wb, wc = a.weights.cpu().numpy(), b.weights.cpu().numpy(), c.weights.cpu().numpy()
    assert np.array_equal(wa, wb)
    assert np.array_equal(wa, wc)
    for m in (a, b, c):
        m.close()


def test_library_shuffle_equals_explicit_order():
    cfg = config(0)
    X = dev(workloads.make_data(cfg))
    kw = dict(lr0=0.5, lr1=0.01, sigma0=5.0, sigma1=1.0)
    order = np.concatenate([oracle.shuffle(11, e, cfg.n) for e in range(3)])
    a = som.Map(10, 10, cfg.d, seed=1)
    a.train(X, 3, shuffle_seed=11, **kw)
    b = som.Map(10, 10, cfg.d, seed=1)
    b.train(X, 3, order=dev(order), **kw)
    assert np.array_equal(a.weights.cpu().numpy(), b.weights.cpu().numpy())
    a.close()
    b.close()


# ------------------------------------------------------------ QE / TE
@pytest.mark.parametrize("rows,cols,d,n,topology", [(10, 10, 500, 200, som.RECT),
                                                    (8, 9, 37, 300, som.HEX),
                                                    (1, 1, 12, 20, som.RECT)])
def test_qe_te_of_given_weights_match_oracle(rows, cols, d, n, topology):
    X, W = _bmu_case(rows, cols, d, n, seed=d, kind="mixture")
    m = make_map(rows, cols, d, topology=topology, W=W)
    qe = m.qe(dev(X))
    te = m.te(dev(X))
    ev = oracle.evaluate(W.astype(np.float64), rows, cols, X, topology=topology)
    assert qe == pytest.approx(ev["qe"], rel=1e-5)
    assert abs(te - ev["te"]) <= 1.0 / n + 1e-12
    if rows * cols == 1:
        assert te == 0.0
    m.close()


# ------------------------------------------------------------ errors
def test_argument_and_order_errors():
    torch = torch_cuda()
    m = som.Map(4, 4, 8)
    X = dev(np.zeros((10, 8), np.float32))
    with pytest.raises(ValueError):
        m.train(torch.zeros((10, 7), device="cuda"), 1, 0.1, 0.1, 1.0, 1.0)
    with pytest.raises(som.SomError) as e:
        # no device allocation covers 2^28 rows of 8 floats (8 GiB)
        som.som_train(m.handle, X, 1 << 28, 1, som.make_schedule(0.1, 0.1, 1.0, 1.0))
    assert e.value.name == "SOM_E_ARG"
    with pytest.raises(som.SomError) as e:
        m.train(X, 1, -0.1, 0.1, 1.0, 1.0)
    assert e.value.name == "SOM_E_ARG"
    with pytest.raises(som.SomError) as e:
        m.train(X, 1, 0.1, 0.1, 0.0, 1.0, sigma_decay=som.EXPONENTIAL)
    assert e.value.name == "SOM_E_ARG"
    host = np.zeros((10, 8), np.float32)
    with pytest.raises(som.SomError) as e:
        som.som_train(m.handle, host.ctypes.data, 10, 1, som.make_schedule(0.1, 0.1, 1, 1))
    assert e.value.name == "SOM_E_ARG"          # host pointer refused
    before = m.weights.cpu().numpy()
    bad = dev(np.array([0, 1, 2, 3, 4, 5, 6, 7, 8, 10], np.int32))
    m.train(X, 1, 0.5, 0.5, 1.0, 1.0, order=bad)
    with pytest.raises(som.SomError) as e:
        m.synchronize()
    assert e.value.name == "SOM_E_BAD_ORDER"
    assert np.array_equal(m.weights.cpu().numpy(), before)   # nothing was updated
    m.synchronize()                                           # error was reported once
    m.close()


def test_tiny_and_ragged_maps_train_like_the_oracle():
    """Fewer units than workgroups, one-unit map, d not a multiple of 4."""
    for rows, cols, d, n in ((1, 1, 5, 9), (2, 3, 37, 40), (1, 300, 3, 50)):
        say("ragged", rows, cols, d, n)
        X = workloads.gaussian_mixture(n, d, 3, 0.1, seed=d)
        order = workloads.epoch_orders(n, 2, 1)
        W0 = oracle.init_uniform(2, rows * cols, d)
        m = som.Map(rows, cols, d, seed=2)
        trace = dev(np.full(2 * n, -1, np.int32))
        m.train(dev(X), 2, 0.5, 0.05, 2.0, 0.5, order=dev(order), bmu_trace=trace)
        Wo, tr = oracle.train(W0, rows, cols, X, order, oracle.schedule(0.5, 0.05, 2.0, 0.5),
                              trace=True)
        got = trace.cpu().numpy()
        if np.array_equal(got, tr):
            assert np.abs(m.weights.cpu().numpy() - Wo).max() <= 1e-4
        else:
            k = int(np.argmax(got != tr))
            Wk, _ = oracle.train(W0, rows, cols, X, order[:k],
                                 oracle.schedule(0.5, 0.05, 2.0, 0.5), total_steps=2 * n)
            Ds = np.sort(oracle.distances(Wk, X[order[k]]))
            assert (Ds[1] - Ds[0]) / Ds[0] <= GAP
        m.close()


def _train_vs_oracle(rows, cols, d, n, epochs, topology=som.RECT, seed=3):
    X = workloads.gaussian_mixture(n, d, 4, 0.15, seed=seed)
    order = workloads.epoch_orders(n, epochs, seed)
    s = oracle.schedule(0.4, 0.02, max(rows, cols) / 2.0, 0.5)
    W0 = oracle.init_uniform(seed, rows * cols, d)
    m = som.Map(rows, cols, d, seed=seed, topology=topology)
    plan = m.plan()
    trace = dev(np.full(epochs * n, -1, np.int32))
    m.train(dev(X), epochs, 0.4, 0.02, max(rows, cols) / 2.0, 0.5, order=dev(order),
            bmu_trace=trace)
    got = trace.cpu().numpy()
    Wo, tr = oracle.train(W0, rows, cols, X, order, s, topology=topology, trace=True)
    if np.array_equal(got, tr):
        err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
        say(f"  plan {plan}: identical BMUs for {len(tr)} steps, max|dW| = {err:.2e}")
        assert err <= 1e-4
    else:
        k = int(np.argmax(got != tr))
        say(f"  plan {plan}: identical BMUs for {k}/{len(tr)} steps")
        Wk, _ = oracle.train(W0, rows, cols, X, order[:k], s, total_steps=epochs * n,
                             topology=topology)
        Ds = np.sort(oracle.distances(Wk, X[order[k]]))
        assert (Ds[1] - Ds[0]) / Ds[0] <= GAP, "divergence without a near tie"
    m.close()
    return plan


# Shapes chosen to reach the kernels' edges: one float4 slice per row (two
# sweepers idle), ragged last slices, a partial last block of steps, 64 units
# per workgroup, and rows too long for the pipelined kernel's registers.
@pytest.mark.parametrize("rows,cols,d,n,epochs", [
    (7, 9, 64, 101, 2),       # one slice, M = 8, 202 steps (partial last block)
    (12, 12, 777, 83, 2),     # 4 slices (2 / 1 / 1 per sweeper), ragged last float4
    (20, 13, 1500, 61, 2),    # 6 - 8 slices
    (9, 50, 2048, 40, 1),     # 8 slices, 2 units per workgroup
    (128, 128, 16, 20, 1),    # 64 units per workgroup
    (6, 5, 3000, 30, 2),      # rows too long for the pipelined kernel
])
@pytest.mark.parametrize("variant", ["0", "3", "4", "5"])
def test_training_shapes_follow_the_oracle(rows, cols, d, n, epochs, variant, monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    say("shape", rows, cols, d, n, epochs, "variant", variant)
    try:
        plan = _train_vs_oracle(rows, cols, d, n, epochs)
    except som.SomError as e:
        if variant in ("3", "4") and e.name == "SOM_E_UNSUPPORTED":
            pytest.skip("shape outside the pipelined kernel's limits")
        raise
    if variant in ("3", "4"):
        assert plan["variant"] == (3 if variant == "3" else 2)
    if variant == "5":
        assert plan["variant"] in (0, 1)


# Every block length the pipelined kernel is built with, forced through
# SOM_TRAIN_BLOCK_M on a row length of its float4-slice count KS (row pitch
# 256 / 512, 1024, 2048, 3072 and 5120 floats: d up to 512, 1024, 2048,
# 3072 and 5120).  The LDS-resident variant runs every one of them.
@pytest.mark.parametrize("rows,cols,d,n,epochs,block_m", [
    (7, 9, 64, 101, 2, 8), (7, 9, 64, 101, 2, 4),            # KS = 1
    (12, 12, 777, 83, 2, 8), (12, 12, 777, 83, 2, 4),        # KS = 2
    (20, 13, 1500, 61, 2, 6), (9, 50, 2048, 40, 1, 6),       # KS = 3
    (20, 13, 1500, 61, 2, 4), (20, 13, 1500, 61, 2, 2),
    (6, 5, 3000, 30, 2, 4), (6, 5, 3000, 30, 2, 2),          # KS = 4
    (5, 4, 5000, 30, 1, 2),                                  # KS = 7
])
def test_pipelined_block_lengths_follow_the_oracle(rows, cols, d, n, epochs, block_m,
                                                   monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "3")
    monkeypatch.setenv("SOM_TRAIN_BLOCK_M", str(block_m))
    say("pipelined block length", block_m, "shape", rows, cols, d, n, epochs)
    plan = _train_vs_oracle(rows, cols, d, n, epochs)
    assert plan["variant"] == 3 and plan["block_steps"] == block_m


@pytest.mark.parametrize("lds_rows", ["0", "1", "7", "64"])
@pytest.mark.parametrize("rows,cols,d,n,epochs", [(20, 13, 1500, 61, 2), (11, 12, 2048, 40, 1)])
def test_streamed_variant_with_leading_rows_in_lds(rows, cols, d, n, epochs, lds_rows,
                                                   monkeypatch):
    # the streamed pipelined kernel keeps its first rows in LDS and streams
    # the rest; 8 workgroups give 33 (16) rows each, so 0, 1 and 7 split the
    # rows and 64 keeps as many as fit
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "4")
    monkeypatch.setenv("SOM_TRAIN_GRID", "8")
    monkeypatch.setenv("SOM_TRAIN_LDS_ROWS", lds_rows)
    say("streamed + LDS rows", rows, cols, d, n, epochs, "lds_rows", lds_rows)
    plan = _train_vs_oracle(rows, cols, d, n, epochs)
    assert plan["variant"] == 2 and plan["grid"] == 8


# The paper's own data shape (Table 1: several hundred short complaint
# documents over about 4.5k terms, Sec. 6B) on a small map of both
# lattices: TF-IDF rows of 637 x 4545 (23 terms each), 11 x 11 units.
@pytest.mark.parametrize("topology", [som.RECT, som.HEX])
def test_paper_shaped_tfidf_map_follows_the_oracle(topology):
    rows = cols = 11
    n, d, epochs = 637, 4545, 2
    X = workloads.tfidf_like(n, d, 0.005, 8, seed=5)
    order = workloads.epoch_orders(n, epochs, 5)
    s = oracle.schedule(0.5, 0.01, 5.5, 1.0, oracle.LINEAR, oracle.EXPONENTIAL)
    W0 = oracle.init_uniform(5, rows * cols, d)
    say("paper-shaped map, topology", topology, "n", n, "d", d, "epochs", epochs)
    m = som.Map(rows, cols, d, seed=5, topology=topology)
    trace = dev(np.full(epochs * n, -1, np.int32))
    m.train(dev(X), epochs, 0.5, 0.01, 5.5, 1.0, order=dev(order), bmu_trace=trace,
            sigma_decay=som.EXPONENTIAL)
    got = trace.cpu().numpy()
    Wo, tr = oracle.train(W0, rows, cols, X, order, s, topology=topology, trace=True)
    k = len(tr) if np.array_equal(got, tr) else int(np.argmax(got != tr))
    say(f"  plan {m.plan()}: identical BMUs for {k}/{len(tr)} steps")
    if k < len(tr):
        Wk, _ = oracle.train(W0, rows, cols, X, order[:k], s, total_steps=epochs * n,
                             topology=topology)
        Ds = np.sort(oracle.distances(Wk, X[order[k]]))
        assert (Ds[1] - Ds[0]) / Ds[0] <= GAP, "divergence without a near tie"
    else:
        err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
        say(f"  max|dW| = {err:.2e}")
        assert err <= 1e-4
    ev = oracle.evaluate(Wo, rows, cols, X, topology=topology)
    qe = m.qe(dev(X))
    assert abs(qe - ev["qe"]) <= 0.01 * ev["qe"]
    m.close()


# The blocked kernel's instances for rows too long for the pipelined one:
# each row length's longest block and the shorter one kept for maps whose
# workgroups own many rows.  Step counts leave a partial last block.
@pytest.mark.parametrize("rows,cols,d,n,epochs,block_m", [
    (5, 4, 6000, 31, 2, 4), (5, 4, 6000, 31, 2, 2),
    (4, 5, 8000, 31, 1, 4), (4, 5, 8000, 31, 1, 2),
    (4, 4, 9500, 31, 2, 3), (4, 4, 9500, 31, 2, 2),
    (3, 5, 12000, 25, 1, 2), (3, 5, 12000, 25, 1, 1),
    (3, 3, 16000, 17, 2, 2), (3, 3, 16000, 17, 2, 1),
])
@pytest.mark.parametrize("variant", ["1", "2"])
def test_blocked_block_lengths_follow_the_oracle(rows, cols, d, n, epochs, block_m, variant,
                                                 monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    monkeypatch.setenv("SOM_TRAIN_BLOCK_M", str(block_m))
    say("blocked block length", block_m, "variant", variant, "shape", rows, cols, d, n, epochs)
    plan = _train_vs_oracle(rows, cols, d, n, epochs)
    # SOM_TRAIN_VARIANT 1 asks for the LDS-resident rows (plan variant 1),
    # 2 for the streamed ones (plan variant 0)
    assert plan["variant"] == {"1": 1, "2": 0}[variant] and plan["block_steps"] == block_m


@pytest.mark.parametrize("lds_rows", ["0", "1", "2", "64"])
@pytest.mark.parametrize("rows,cols,d,n,epochs", [(6, 5, 3000, 30, 2), (5, 4, 9000, 20, 1)])
def test_blocked_streamed_variant_with_leading_rows_in_lds(rows, cols, d, n, epochs, lds_rows,
                                                           monkeypatch):
    # the streamed blocked kernel (rows too long for the pipelined one) keeps
    # its first rows in LDS and streams the rest; 4 workgroups give 8 and 5
    # rows each
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "2")
    monkeypatch.setenv("SOM_TRAIN_GRID", "4")
    monkeypatch.setenv("SOM_TRAIN_LDS_ROWS", lds_rows)
    say("blocked streamed + LDS rows", rows, cols, d, n, epochs, "lds_rows", lds_rows)
    plan = _train_vs_oracle(rows, cols, d, n, epochs)
    assert plan["variant"] == 0 and plan["grid"] == 4


def test_misaligned_samples_train_like_aligned_ones():
    # X starting one float into an allocation (d % 4 == 0 but rows not
    # 16-byte aligned) goes through the padded copy; results are bitwise
    # those of the aligned matrix.
    torch = torch_cuda()
    n, d = 90, 256
    X = workloads.gaussian_mixture(n, d, 3, 0.2, seed=11)
    order = dev(workloads.epoch_orders(n, 2, 5))
    flat = torch.zeros(n * d + 1, dtype=torch.float32, device="cuda")
    flat[1:] = torch.from_numpy(X.reshape(-1)).cuda()
    Xm = flat[1:].view(n, d)
    assert Xm.data_ptr() % 16 != 0
    out = []
    for Xd in (dev(X), Xm):
        m = som.Map(6, 7, d, seed=4)
        trace = dev(np.full(2 * n, -1, np.int32))
        m.train(Xd, 2, 0.5, 0.05, 3.0, 0.5, order=order, bmu_trace=trace)
        out.append((m.weights.cpu().numpy(), trace.cpu().numpy()))
        m.close()
    assert np.array_equal(out[0][1], out[1][1])
    assert np.array_equal(out[0][0], out[1][0])


@pytest.mark.parametrize("variant", ["0", "5"])
def test_hexagonal_lattice_shapes_follow_the_oracle(variant, monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    for rows, cols, d, n in ((9, 11, 300, 70), (16, 16, 1024, 40)):
        say("hex shape", rows, cols, d, n, "variant", variant)
        _train_vs_oracle(rows, cols, d, n, 2, topology=som.HEX)


@pytest.mark.parametrize("side", [128, 512])
def test_large_maps_at_small_d_follow_the_oracle(side):
    # Maps of the d = 64 size sweep: 16384 units (64 per workgroup) and
    # 262144 units (1024 per workgroup, the blocked kernel's LDS loop path).
    say("large map", side, side)
    _train_vs_oracle(side, side, 64, 150, 1)


# The streamed pipelined kernel on four sweeper waves (plan block 320,
# blocks of five steps): rows of 512 float4, two slices per sweeper (one for
# the last sweeper when d leaves seven), ragged row counts, 0 to all rows in
# LDS; and the same shapes forced onto three sweepers.
@pytest.mark.parametrize("rows,cols,d,n,epochs,grid", [
    (9, 50, 2048, 40, 1, 0),     # the planner's grid: 64 (four sweepers) or 128 workgroups
    (11, 12, 2048, 41, 2, 8),    # 16-17 rows per workgroup, partial last block
    (20, 13, 1500, 61, 2, 8),    # 375 float4 of 512: the last slices partly zero
    (20, 20, 1100, 17, 1, 8),    # 50 rows per workgroup, d = 1100 (row pitch 2048)
])
@pytest.mark.parametrize("lds_rows", ["0", "3", "64"])
@pytest.mark.parametrize("sweepers", ["4", "3"])
def test_streamed_pipelined_sweeper_counts_follow_the_oracle(rows, cols, d, n, epochs, grid,
                                                             lds_rows, sweepers, monkeypatch):
    if grid and rows * cols / grid > 64:
        pytest.skip("more than 64 units per workgroup")   # (the planner's grid never has)
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "4")
    monkeypatch.setenv("SOM_TRAIN_SWEEPERS", sweepers)
    monkeypatch.setenv("SOM_TRAIN_LDS_ROWS", lds_rows)
    if grid:
        monkeypatch.setenv("SOM_TRAIN_GRID", str(grid))
    say("streamed sweepers", sweepers, rows, cols, d, n, epochs, "grid", grid, "lds_rows", lds_rows)
    plan = _train_vs_oracle(rows, cols, d, n, epochs)
    assert plan["variant"] == 2 and plan["block"] == 64 * (int(sweepers) + 1)
    if sweepers == "4":
        assert plan["block_steps"] == 5


# Rows too long for the pipelined kernel's sample registers, on its
# column-walk sweep (plan variant 4): ragged row counts per workgroup, slices
# reaching past d (zeros there), sweepers with different slice counts, a
# partial last block, and 0 to 4 rows kept in LDS.
@pytest.mark.parametrize("rows,cols,d,n,epochs,grid", [
    (5, 4, 6000, 31, 2, 3),      # 6-7 rows per workgroup, 24 slices (8 each)
    (4, 4, 9500, 31, 2, 2),      # 8 rows, 40 slices (14 / 13 / 13), ragged tail slice
    (3, 5, 12000, 25, 1, 2),     # 7-8 rows, 48 slices
    (3, 3, 16000, 17, 2, 1),     # 9 rows on one workgroup, 64 slices
    (4, 3, 7001, 20, 1, 2),      # d not a multiple of 4: padded sample copy
    (10, 10, 6000, 23, 1, 10),   # 10 rows per workgroup, the kernel's bound
])
@pytest.mark.parametrize("lds_rows", ["0", "1", "4"])
def test_long_rows_pipelined_follow_the_oracle(rows, cols, d, n, epochs, grid, lds_rows,
                                               monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "4")
    monkeypatch.setenv("SOM_TRAIN_GRID", str(grid))
    monkeypatch.setenv("SOM_TRAIN_LDS_ROWS", lds_rows)
    say("long rows", rows, cols, d, n, epochs, "grid", grid, "lds_rows", lds_rows)
    plan = _train_vs_oracle(rows, cols, d, n, epochs)
    assert plan["variant"] == 4 and plan["grid"] == grid


# Runs shorter than one block, one block exactly, and one block plus one
# step, on the two kernels with the longest blocks: the four-sweeper
# streamed kernel (5 steps a block) and the column walk (8).  The sample
# products' prepass, the controller's exchanges and the sweepers' last
# update must all stop at the last real step.
@pytest.mark.parametrize("steps", [1, 2, 4, 5, 6, 7, 8, 9])
@pytest.mark.parametrize("rows,cols,d,grid,sweepers,block_steps", [
    (11, 12, 2048, 8, "4", 5),   # four sweepers, streamed rows
    (5, 4, 6000, 3, "", 8),      # column walk (two windows of rows)
])
def test_runs_shorter_than_a_block_follow_the_oracle(rows, cols, d, grid, sweepers, block_steps,
                                                     steps, monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "4")
    monkeypatch.setenv("SOM_TRAIN_GRID", str(grid))
    if sweepers:
        monkeypatch.setenv("SOM_TRAIN_SWEEPERS", sweepers)
    say("short run", rows, cols, d, "steps", steps, "grid", grid)
    plan = _train_vs_oracle(rows, cols, d, steps, 1)
    assert plan["block_steps"] == block_steps and plan["grid"] == grid


def test_long_rows_pipelined_hexagonal_and_schedule_edges(monkeypatch):
    # the column-walk sweep on a hexagonal lattice, then a unit rate with a
    # zero radius, which must copy each sample exactly into its BMU
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "4")
    say("long rows hex")
    plan = _train_vs_oracle(4, 5, 8000, 27, 2, topology=som.HEX)
    assert plan["variant"] == 4
    X = workloads.gaussian_mixture(9, 9000, 3, 0.2, seed=5)
    W = workloads.random_weights(12, 9000, 6)
    m = make_map(3, 4, 9000, W=W)
    order = np.arange(9, dtype=np.int32)
    trace = dev(np.full(9, -1, dtype=np.int32))
    m.train(dev(X), 1, 1.0, 1.0, 0.0, 0.0, order=dev(order), bmu_trace=trace)
    assert m.plan()["variant"] == 4
    s = oracle.schedule(1.0, 1.0, 0.0, 0.0, oracle.LINEAR, oracle.LINEAR)
    Wo, tr = oracle.train(W, 3, 4, X, order, s, trace=True)
    assert np.array_equal(trace.cpu().numpy(), tr)
    assert np.array_equal(m.weights.cpu().numpy().astype(np.float64), Wo)
    m.close()
