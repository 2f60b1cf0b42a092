"""Batch-map training (som_train_batch) against the fp64 oracle.

One epoch = BMUs of all samples, then every prototype set to the
neighbourhood-weighted mean of the samples (oracle.train_batch, on the
explicit N x N neighbourhood matrix; the GPU factors the lattice Gaussian
into a column and a row blur).  Each epoch starts from the GPU's state:
the GPU's BMUs may differ from the oracle's only at an oracle near tie
(relative top-two gap 1e-4), and the oracle's update applied to the GPU's
BMUs (oracle.batch_update) must give the GPU's prototypes within 1e-5.
"""
import math

import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import config, dev, rel_gap, say

pytestmark = pytest.mark.gpu

ATOL = 1e-5


def _mixture(n, d, k, sd, seed):
    return workloads.gaussian_mixture(n, d, k, sd, seed=seed)


def _check_epochs(rows, cols, d, n, epochs, s0, s1, topology=som.RECT, decay=oracle.EXPONENTIAL,
                  seed=3):
    """Every epoch from the GPU's state: the GPU's BMUs (the same search the
    batch call runs) equal the oracle's except at oracle near ties, where
    the GPU's unit is within the gap of the best; the oracle's update
    applied to the GPU's BMUs then gives the GPU's prototypes within ATOL,
    and with no near tie in the epoch so does the oracle's own epoch."""
    X = _mixture(n, d, 5, 0.2, seed)
    m = som.Map(rows, cols, d, seed=seed, topology=topology)
    Xd = dev(X)
    for e in range(epochs):
        sigma = oracle.batch_sigma(e, epochs, s0, s1, decay)
        Wg_prev = m.weights.cpu().numpy().astype(np.float64)
        c_gpu = m.bmu(Xd).cpu().numpy().astype(np.int64)
        m.train_batch(Xd, 1, sigma, sigma, decay)
        Wg = m.weights.cpu().numpy().astype(np.float64)
        ev = oracle.evaluate(Wg_prev, rows, cols, X, topology=topology)
        gap = rel_gap(ev["d1"], ev["d2"])
        diff = np.nonzero(c_gpu != ev["c1"])[0]
        for i in diff:
            D = oracle.distances(Wg_prev, X[i])
            assert gap[i] <= 1e-4 and D[c_gpu[i]] - ev["d1"][i] <= 1e-4 * ev["d1"][i], i
        err = np.abs(Wg - oracle.batch_update(Wg_prev, rows, cols, X, c_gpu, sigma,
                                              topology)).max()
        say(f"  epoch {e} sigma {sigma:.3g}: {diff.size} near-tie BMUs, "
            f"max|dW| {err:.2e} under the GPU's BMUs, min gap {gap.min():.2e}")
        assert err <= ATOL
        if gap.min() > 1e-4:
            Wo, _ = oracle.train_batch(Wg_prev, rows, cols, X, 1, sigma, sigma, decay,
                                       topology=topology)
            assert np.abs(Wg - Wo).max() <= ATOL
    m.close()


@pytest.mark.parametrize("rows,cols,d,n,topology", [
    (10, 10, 64, 500, som.RECT),
    (7, 9, 37, 300, som.RECT),      # ragged units and columns
    (13, 70, 300, 400, som.RECT),   # more than 64 lattice columns
    (70, 3, 20, 200, som.RECT),     # more than 64 lattice rows
    (9, 8, 50, 300, som.HEX),
    (66, 65, 12, 600, som.HEX),
    (1, 1, 5, 40, som.RECT),
])
def test_batch_epochs_match_oracle(rows, cols, d, n, topology):
    say("batch", rows, cols, d, n, "hex" if topology else "rect")
    _check_epochs(rows, cols, d, n, 3, max(rows, cols) / 2.0, 0.7, topology)


def _random_batch_cases(seed, count):
    """Random (rows, cols, d, n, topology): lattices up to 48 x 48 and rows
    of up to 1500 floats, with N^2 d bounded for the oracle's explicit
    neighbourhood matrix."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        rows, cols = int(rng.integers(1, 49)), int(rng.integers(1, 49))
        d = int(rng.integers(1, 1501))
        while d > 1 and (rows * cols) ** 2 * d > 2e9:
            d //= 2
        out.append((rows, cols, d, int(rng.integers(1, 801)),
                    som.HEX if rng.random() < 0.4 else som.RECT))
    return out


@pytest.mark.parametrize("case", _random_batch_cases(41, 12),
                         ids=[f"batch-{i}" for i in range(12)])
def test_random_batch_shapes_match_oracle(case):
    rows, cols, d, n, topology = case
    say("random batch", rows, cols, d, n, "hex" if topology else "rect")
    _check_epochs(rows, cols, d, n, 2, max(rows, cols) / 2.0, 0.7, topology,
                  seed=rows * 7919 + cols * 104729 + d)


def test_radius_zero_is_k_means_and_infinite_radius_the_mean():
    X = _mixture(300, 16, 4, 0.3, 5)
    m = som.Map(4, 5, 16, seed=2)
    W0 = m.weights.cpu().numpy().astype(np.float64)
    m.train_batch(dev(X), 1, 0.0, 0.0)
    Wo, _ = oracle.train_batch(W0, 4, 5, X, 1, 0.0, 0.0)
    assert np.abs(m.weights.cpu().numpy() - Wo).max() <= ATOL
    m.train_batch(dev(X), 1, math.inf, math.inf)
    mean = X.astype(np.float64).mean(0)
    assert np.abs(m.weights.cpu().numpy() - mean[None, :]).max() <= ATOL
    m.close()


def test_linear_decay_and_errors():
    X = dev(_mixture(100, 8, 2, 0.3, 6))
    m = som.Map(3, 3, 8)
    m.train_batch(X, 4, 2.0, 0.5, som.LINEAR)
    for bad in [(-1.0, 1.0, som.EXPONENTIAL), (2.0, 0.0, som.EXPONENTIAL), (2.0, 1.0, 7),
                (math.nan, 1.0, som.LINEAR)]:
        with pytest.raises(som.SomError) as e:
            m.train_batch(X, 1, *bad)
        assert e.value.name == "SOM_E_ARG"
    with pytest.raises(som.SomError):
        som.som_train_batch(m.handle, X, 100, 0, 1.0, 1.0)
    m.close()


def test_workload_sized_epoch_on_sampled_units():
    # 100,000 x 2048 mixture on the 100 x 100 map: one epoch on the GPU,
    # then the oracle's rule for 24 sampled units from the GPU's own BMUs
    # (the BMUs are checked by the batched-BMU tests): w_u = sum_i h(u,
    # c_i) x_i / sum_i h(u, c_i)
    cfg = config(4)
    say("batch epoch at", cfg.name)
    X = workloads.make_data(cfg)
    Xd = dev(X)
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed)
    c = m.bmu(Xd).cpu().numpy()
    sigma = 12.0
    m.train_batch(Xd, 1, sigma, sigma)
    Wg = m.weights.cpu().numpy()
    rng = np.random.default_rng(0)
    units = rng.choice(cfg.units, 24, replace=False)
    Xd64 = X.astype(np.float64)
    for u in units:
        # h(u, c_i) for every sample (the Gaussian is symmetric in u and c)
        hu = oracle.neighbourhood(cfg.rows, cfg.cols, oracle.RECT, int(u), 1.0, sigma)[c]
        want = (hu[:, None] * Xd64).sum(0) / hu.sum()
        err = np.abs(Wg[u] - want).max()
        assert err <= ATOL, (u, err)
    say(f"  24 sampled units within {ATOL}")
    m.close()
