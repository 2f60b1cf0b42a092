"""Error paths of the training and evaluation calls on the GPU, each forced
from the host so that every kernel still ends normally:

  * SOM_E_NONFINITE: a NaN or an infinity in the training data stops the
    training kernel before any update (the call's scan of the samples);
  * SOM_E_OOM: SOM_MAX_BYTES below what a call needs; the map stays usable;
  * SOM_E_LAUNCH: a requested grid that cannot be co-resident is refused by
    the planner, before anything is launched;
  * SOM_E_TIMEOUT: one workgroup fewer launched than the exchanges wait for
    (SOM_DEBUG_ABSENT_WORKGROUP), with a short bound on each exchange wait
    (SOM_DEBUG_EXCHANGE_TIMEOUT_US).  Every wait of the other workgroups is
    bounded by that time, a workgroup whose exchange is given up leaves its
    block loop at the next in-workgroup barrier, and the workgroups still
    waiting see the raised status within 16 (multi-poll) or 64 (one-poll)
    polls, so the grid drains in about the bound.
"""
import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import dev, rel_gap, say, torch_cuda

pytestmark = pytest.mark.gpu

SCHED = (0.5, 0.05, 3.0, 0.5)


def _map(rows, cols, d, W):
    m = som.Map(rows, cols, d, seed=1)
    m.weights = dev(W)
    return m


def _fresh_training(rows, cols, d, W, X, order):
    """Weights after training a new map from W on X (no forcing)."""
    m = _map(rows, cols, d, W)
    m.train(dev(X), 1, *SCHED, order=dev(order))
    m.synchronize()
    out = m.weights.cpu().numpy()
    m.close()
    return out


# ------------------------------------------------------------ non-finite data
@pytest.mark.parametrize("value", [np.nan, np.inf, -np.inf])
@pytest.mark.parametrize("rows,cols,d,variant,where", [
    (7, 9, 64, "", "first"),          # planner's choice
    (7, 9, 64, "5", "last"),          # blocked kernel
    (11, 12, 2048, "4", "middle"),    # pipelined, streamed rows
    (4, 3, 7001, "4", "last"),        # long rows, padded sample copy (d % 4 != 0)
    (3, 4, 37, "", "middle"),         # padded sample copy of short rows
])
def test_nonfinite_samples_stop_training_before_any_update(rows, cols, d, variant, where,
                                                           value, monkeypatch):
    if variant:
        monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    n = 23
    X = workloads.gaussian_mixture(n, d, 3, 0.2, seed=d)
    W = workloads.random_weights(rows * cols, d, 4)
    order = workloads.epoch_orders(n, 1, 2)
    i = {"first": 0, "middle": n * d // 2 + 1, "last": n * d - 1}[where]
    bad = X.copy()
    bad.reshape(-1)[i] = value
    say("nonfinite", rows, cols, d, variant, where, value)
    m = _map(rows, cols, d, W)
    m.train(dev(bad), 1, *SCHED, order=dev(order))
    with pytest.raises(som.SomError) as e:
        m.synchronize()
    assert e.value.name == "SOM_E_NONFINITE"
    assert np.array_equal(m.weights.cpu().numpy(), W)   # nothing was updated
    m.synchronize()                                      # reported once
    # the same map then trains on clean data exactly like a new one
    m.train(dev(X), 1, *SCHED, order=dev(order))
    m.synchronize()
    assert np.array_equal(m.weights.cpu().numpy(), _fresh_training(rows, cols, d, W, X, order))
    m.close()


def test_largest_finite_values_are_not_flagged():
    X = np.zeros((8, 16), np.float32)
    X[3, 5] = np.finfo(np.float32).max
    X[6, 0] = -np.finfo(np.float32).max
    X[7, 1] = np.finfo(np.float32).tiny / 4       # a denormal
    m = som.Map(2, 2, 16, seed=0)
    m.train(dev(X), 1, 0.1, 0.1, 1.0, 1.0)
    m.synchronize()                                # no error raised
    m.close()


def test_bad_order_is_reported_before_nonfinite_data():
    # both errors in one call: the order check runs first and wins
    X = workloads.gaussian_mixture(10, 8, 2, 0.1, seed=1)
    X[4, 2] = np.nan
    m = som.Map(3, 3, 8, seed=0)
    order = dev(np.array([0, 1, 2, 3, 4, 5, 6, 7, 8, 10], np.int32))
    m.train(dev(X), 1, *SCHED, order=order)
    with pytest.raises(som.SomError) as e:
        m.synchronize()
    assert e.value.name == "SOM_E_BAD_ORDER"
    m.synchronize()
    m.close()


def test_nonfinite_sparse_values_stop_training():
    torch = torch_cuda()
    n, d = 30, 400
    X = workloads.small_tfidf(n, d, 3)
    indptr = np.zeros(n + 1, np.int64)
    cols, vals = [], []
    for i in range(n):
        nz = np.nonzero(X[i])[0]
        cols.append(nz.astype(np.int32))
        vals.append(X[i, nz])
        indptr[i + 1] = indptr[i] + len(nz)
    cols = np.concatenate(cols)
    vals = np.concatenate(vals).astype(np.float32)
    assert len(vals) > 10
    vals[len(vals) // 2] = np.inf
    W = workloads.random_weights(25, d, 5, 0.0, 0.05)
    m = _map(5, 5, d, W)
    m.train_csr(dev(indptr), dev(cols), dev(vals), 1, *SCHED)
    with pytest.raises(som.SomError) as e:
        m.synchronize()
    assert e.value.name == "SOM_E_NONFINITE"
    assert np.array_equal(m.weights.cpu().numpy(), W)
    m.synchronize()
    m.close()
    del torch


# ------------------------------------------------------------ memory cap
def _assert_bmus(got, W, rows, cols, X):
    """BMUs equal to the oracle's wherever its best two are 1e-4 apart."""
    o = oracle.evaluate(W, rows, cols, X)
    clear = rel_gap(o["d1"], o["d2"]) > 1e-4
    assert clear.mean() > 0.9
    assert np.array_equal(got[clear], o["c1"][clear])


def test_memory_cap_refuses_evaluation_scratch_and_keeps_the_map_usable(monkeypatch):
    rows, cols, d = 10, 10, 64
    W = workloads.random_weights(rows * cols, d, 2)
    X = workloads.gaussian_mixture(1000, d, 4, 0.2, seed=3)
    m = _map(rows, cols, d, W)
    small = dev(X[:10])
    want_small = m.bmu(small).cpu().numpy()
    _assert_bmus(want_small, W, rows, cols, X[:10])
    # 4096 bytes: 10 samples' scratch fits, 1000 samples' (12 bytes each) does not
    monkeypatch.setenv("SOM_MAX_BYTES", "4096")
    with pytest.raises(som.SomError) as e:
        m.bmu(dev(X))
    assert e.value.name == "SOM_E_OOM"
    with pytest.raises(som.SomError) as e:
        m.evaluate(dev(X))
    assert e.value.name == "SOM_E_OOM"
    assert np.array_equal(m.bmu(small).cpu().numpy(), want_small)
    with pytest.raises(som.SomError) as e:
        m.train_batch(dev(X), 1, 1.0, 1.0)
    assert e.value.name == "SOM_E_OOM"
    with pytest.raises(som.SomError) as e:
        som.Map(rows, cols, d, seed=0)               # the prototypes alone exceed it
    assert e.value.name == "SOM_E_OOM"
    monkeypatch.delenv("SOM_MAX_BYTES")
    # without the cap the scratch grows and the large call matches the oracle
    _assert_bmus(m.bmu(dev(X)).cpu().numpy(), W, rows, cols, X)
    m.synchronize()
    m.close()


# ------------------------------------------------------------ co-residency
def test_grid_beyond_co_residency_is_refused_before_launch(monkeypatch):
    # the blocked kernel holds one workgroup per compute unit: 1024 cannot be
    # co-resident on 256 compute units
    monkeypatch.setenv("SOM_TRAIN_VARIANT", "5")
    monkeypatch.setenv("SOM_TRAIN_GRID", "1024")
    m = som.Map(40, 40, 64, seed=0)
    before = m.weights.cpu().numpy()
    with pytest.raises(som.SomError) as e:
        m.plan()
    assert e.value.name == "SOM_E_LAUNCH"
    X = dev(workloads.gaussian_mixture(20, 64, 2, 0.1, seed=0))
    with pytest.raises(som.SomError) as e:
        m.train(X, 1, *SCHED)
    assert e.value.name == "SOM_E_LAUNCH"
    m.synchronize()
    assert np.array_equal(m.weights.cpu().numpy(), before)
    m.close()


# ------------------------------------------------------------ exchange timeout
# Kernel variants and exchange shapes: blocked LDS / streamed (one-wave
# rows <= 64 and the > 64 rows path), pipelined LDS (multi-poll, <= 16, <= 64
# and <= 256 workgroups), pipelined streamed (one poll; three and four
# sweepers) and the long-row column walk.
@pytest.mark.parametrize("rows,cols,d,variant,grid,sweepers,plan_variant", [
    (7, 9, 64, "1", 4, "", 1),
    (7, 9, 64, "2", 4, "", 0),
    (20, 20, 64, "1", 4, "", 1),
    (10, 10, 500, "3", 8, "", 3),
    (20, 20, 2000, "3", 64, "", 3),
    (30, 30, 5000, "3", 256, "", 3),
    (11, 12, 2048, "4", 8, "3", 2),
    (11, 12, 2048, "4", 8, "4", 2),
    (5, 4, 6000, "4", 3, "", 4),
])
def test_exchange_timeout_ends_the_grid_and_is_reported(rows, cols, d, variant, grid, sweepers,
                                                        plan_variant, monkeypatch):
    monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    monkeypatch.setenv("SOM_TRAIN_GRID", str(grid))
    if sweepers:
        monkeypatch.setenv("SOM_TRAIN_SWEEPERS", sweepers)
    n = 19
    X = workloads.gaussian_mixture(n, d, 3, 0.2, seed=7)
    W = workloads.random_weights(rows * cols, d, 8)
    order = workloads.epoch_orders(n, 1, 9)
    m = _map(rows, cols, d, W)
    plan = m.plan()
    say("timeout", rows, cols, d, "variant", variant, "plan", plan)
    assert plan["variant"] == plan_variant and plan["grid"] == grid
    monkeypatch.setenv("SOM_DEBUG_EXCHANGE_TIMEOUT_US", "5000")
    monkeypatch.setenv("SOM_DEBUG_ABSENT_WORKGROUP", "1")
    m.train(dev(X), 1, *SCHED, order=dev(order))
    with pytest.raises(som.SomError) as e:
        m.synchronize()
    assert e.value.name == "SOM_E_TIMEOUT"
    m.synchronize()                                   # reported once
    monkeypatch.delenv("SOM_DEBUG_ABSENT_WORKGROUP")
    monkeypatch.delenv("SOM_DEBUG_EXCHANGE_TIMEOUT_US")
    # the map trains normally afterwards, like a new one
    m.weights = dev(W)
    m.train(dev(X), 1, *SCHED, order=dev(order))
    m.synchronize()
    assert np.array_equal(m.weights.cpu().numpy(), _fresh_training(rows, cols, d, W, X, order))
    m.close()
