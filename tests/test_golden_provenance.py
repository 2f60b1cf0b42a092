"""The stored end-to-end values are the oracle's.

tests/golden/make_golden.py writes the expected QE / TE of each workload
from the fp64 oracle alone.  Re-running its steps for the smallest workload
(both lattices, a fraction of a second) must give the stored numbers, and the
inputs must hash as recorded, so the GPU end-to-end tests compare against the
oracle and not against an earlier GPU run.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("topology,suffix", [(oracle.RECT, ""), (oracle.HEX, "_hex")])
def test_smallest_workload_golden_regenerates_from_the_oracle(topology, suffix):
    cfg = workloads.WORKLOADS[0]
    with open(os.path.join(GOLD, f"e2e_{cfg.name}{suffix}.json")) as f:
        g = json.load(f)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    W = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    assert workloads.sha256_of(X) == g["sha256_X"]
    assert workloads.sha256_of(order) == g["sha256_order"]
    assert workloads.sha256_of(W.astype(np.float32)) == g["sha256_W0_f32"]
    s = oracle.schedule(cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                        oracle.LINEAR, oracle.EXPONENTIAL)
    W, _ = oracle.train(W, cfg.rows, cfg.cols, X, order, s, total_steps=cfg.steps,
                        topology=topology)
    ev = oracle.evaluate(W, cfg.rows, cfg.cols, X, topology=topology)
    # the writer trains epoch by epoch; the oracle's steps do not depend on
    # how a run is split, so the numbers agree to the last bits
    assert ev["qe"] == pytest.approx(g["qe"], rel=1e-12)
    assert ev["te"] == pytest.approx(g["te"], abs=1e-15)
