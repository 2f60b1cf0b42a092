"""End-to-end parity (criterion 3): train each workload over its full
schedule on the GPU from the seeded initial map and compare the final QE and
TE with the fp64 oracle's, written by tests/golden/make_golden.py."""
import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import config, dev, golden, say

pytestmark = pytest.mark.gpu

REL = 0.01


@pytest.mark.parametrize("ci", [0, 1, 2, 3, 4])
def test_full_training_matches_oracle_quality(ci):
    cfg = config(ci)
    g = golden(cfg)
    if g is None:
        pytest.skip(f"no oracle golden values for {cfg.name} yet")
    say("e2e", cfg.name)
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    assert workloads.sha256_of(X) == g["sha256_X"], "input data differs from the golden run"
    assert workloads.sha256_of(order) == g["sha256_order"]
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed)
    assert workloads.sha256_of(m.weights.cpu().numpy()) == g["sha256_W0_f32"]
    Xd = dev(X)
    m.train(Xd, cfg.epochs, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1, order=dev(order))
    m.synchronize()
    qe, te = m.qe(Xd), m.te(Xd)
    say(f"  gpu qe={qe:.6f} te={te:.6f} | oracle qe={g['qe']:.6f} te={g['te']:.6f}")
    # cross-evaluation: the oracle's evaluator on the GPU's trained map
    W = m.weights.cpu().numpy().astype(np.float64)
    sub = slice(0, min(cfg.n, 4000))
    ev = oracle.evaluate(W, cfg.rows, cfg.cols, X[sub])
    idx = m.bmu(dev(X[sub])).cpu().numpy()
    agree = float(np.mean(idx == ev["c1"]))
    say(f"  cross-eval on {X[sub].shape[0]} samples: BMU agreement {agree:.5f}")
    assert agree >= 0.999
    if sub.stop >= cfg.n:
        assert qe == pytest.approx(ev["qe"], rel=1e-5)
    assert qe == pytest.approx(g["qe"], rel=REL)
    if g["te"] == 0.0:
        assert te == 0.0
    else:
        assert te == pytest.approx(g["te"], rel=REL)
    m.close()
