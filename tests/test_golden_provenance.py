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


def test_te_spread_records_are_the_oracles():
    """Every stored ensemble of equally valid trainings refers to the same
    inputs as its workload's golden run, and its first training of the
    2000 x 2000 workload (a few seconds) regenerates from the oracle."""
    import glob
    import sys

    sys.path.insert(0, GOLD)
    import make_te_spread as mts

    found = sorted(glob.glob(os.path.join(GOLD, "te_spread_*.json")))
    assert found, "no stored oracle ensembles"
    for path in found:
        with open(path) as f:
            sp = json.load(f)
        suffix = "_hex" if sp["topology"] == "hex" else ""
        with open(os.path.join(GOLD, f"e2e_{sp['config']}{suffix}.json")) as f:
            g = json.load(f)
        assert sp["sha256_X"] == g["sha256_X"] and sp["sha256_order"] == g["sha256_order"]
        assert sp["written_by"].startswith("tests/golden/make_te_spread.py")
        assert len({r["k"] for r in sp["runs"]}) == len(sp["runs"])
    cfg = workloads.WORKLOADS[1]
    with open(os.path.join(GOLD, f"te_spread_{cfg.name}.json")) as f:
        sp = json.load(f)
    rec = next(r for r in sp["runs"] if r["k"] == 1)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    W = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    s = oracle.schedule(cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                        oracle.LINEAR, oracle.EXPONENTIAL)
    flips = 0
    for e in range(cfg.epochs):
        sl = order[e * cfg.n:(e + 1) * cfg.n]
        W, f = oracle.train_near_tie(W, cfg.rows, cfg.cols, X, sl, s, mts.TIE_REL, 1001,
                                     step0=e * cfg.n, total_steps=cfg.steps,
                                     nthreads=min(4, oracle.default_threads()))
        flips += f
    ev = oracle.evaluate(W, cfg.rows, cfg.cols, X)
    assert flips == rec["near_ties_flipped"]
    assert ev["qe"] == pytest.approx(rec["qe"], rel=1e-12)
    assert round(ev["te"] * cfg.n) == rec["te_count"]
