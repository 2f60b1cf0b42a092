"""Batch-map training (som_train_batch) against the fp64 oracle.

One epoch = BMUs of all samples, then every prototype set to the
neighbourhood-weighted mean of the samples (oracle.train_batch, on the
explicit N x N neighbourhood matrix; the GPU factors the lattice Gaussian
into a column and a row blur).  With identical BMUs the prototypes must
agree within 1e-5; BMUs may differ only where the oracle's top-two gap is
a near tie (relative 1e-4).
"""
import math

import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import config, dev, say

pytestmark = pytest.mark.gpu

ATOL = 1e-5


def _mixture(n, d, k, sd, seed):
    return workloads.gaussian_mixture(n, d, k, sd, seed=seed)


def _check_epochs(rows, cols, d, n, epochs, s0, s1, topology=som.RECT, decay=oracle.EXPONENTIAL,
                  seed=3):
    X = _mixture(n, d, 5, 0.2, seed)
    m = som.Map(rows, cols, d, seed=seed, topology=topology)
    Xd = dev(X)
    for e in range(epochs):
        # one epoch at a time, each against the oracle from the GPU's state,
        # so a near-tie BMU in one epoch cannot mask the next
        sigma = oracle.batch_sigma(e, epochs, s0, s1, decay)
        Wg_prev = m.weights.cpu().numpy().astype(np.float64)
        m.train_batch(Xd, 1, sigma, sigma, decay)
        Wg = m.weights.cpu().numpy().astype(np.float64)
        Wo, b = oracle.train_batch(Wg_prev, rows, cols, X, 1, sigma, sigma, decay,
                                   topology=topology, trace=True)
        ev = oracle.evaluate(Wg_prev, rows, cols, X, topology=topology)
        gap = (ev["d2"] - ev["d1"]) / np.maximum(ev["d1"], 1e-300)
        err = np.abs(Wg - Wo).max()
        say(f"  epoch {e} sigma {sigma:.3g}: max|dW| {err:.2e}, min gap {gap.min():.2e}")
        if gap.min() > 1e-4:
            assert err <= ATOL
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
