"""Helpers shared by the GPU tests (no test functions here)."""
import json
import os

import numpy as np

import oracle
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    return torch


def dev(a, dtype=None):
    torch = torch_cuda()
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def rel_gap(d1, d2):
    """(D2 - D1) / D1 of the oracle's best two squared distances."""
    d1 = np.asarray(d1, dtype=np.float64)
    d2 = np.asarray(d2, dtype=np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        g = np.where(d1 > 0, (d2 - d1) / d1, np.where(d2 > d1, np.inf, 0.0))
    return g


def oracle_schedule(cfg):
    return oracle.schedule(cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                           oracle.LINEAR, oracle.EXPONENTIAL)


def golden(cfg, hex_lattice=False):
    p = os.path.join(GOLD, f"e2e_{cfg.name}{'_hex' if hex_lattice else ''}.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        return json.load(f)


def te_spread(cfg, hex_lattice=False):
    """The oracle's own ensemble of equally valid trainings of a workload
    (tests/golden/make_te_spread.py), or None."""
    p = os.path.join(GOLD, f"te_spread_{cfg.name}{'_hex' if hex_lattice else ''}.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        return json.load(f)


# Tolerance of the end-of-training TE (criterion 3): 1 % of the oracle's
# count, widened where the oracle itself spreads further.
TE_REL = 0.01
TE_MIN_ENSEMBLE = 3


def te_band(cfg, g, hex_lattice=False):
    """(centre, half-width, basis) of the accepted TE count of a full
    training.  The oracle's own trainings that decide near ties by a coin
    (make_te_spread.py) are as valid as the stored one; with the stored run
    they form an ensemble of m counts.  One more equally valid training --
    the GPU's -- lies in the ensemble's 99 % prediction interval
    mean +- t(0.995, m - 1) sd sqrt(1 + 1/m).  The band is that interval,
    and never narrower than 1 % of the stored count around it; with fewer
    than TE_MIN_ENSEMBLE counts it is the stored count +- 1 %."""
    from scipy.stats import t as student_t

    sp = te_spread(cfg, hex_lattice)
    counts = [int(g["te_count"])]
    if sp is not None:
        assert sp["sha256_X"] == g["sha256_X"] and sp["sha256_order"] == g["sha256_order"]
        counts += [int(r["te_count"]) for r in sp["runs"]]
    m = len(counts)
    floor = TE_REL * counts[0]
    if m < TE_MIN_ENSEMBLE:
        return float(counts[0]), floor, f"1 % of the stored count ({m} oracle training(s))"
    mean = float(np.mean(counts))
    sd = float(np.std(counts, ddof=1))
    half = float(student_t.ppf(0.995, m - 1)) * sd * np.sqrt(1.0 + 1.0 / m)
    return mean, max(floor, half), (f"99 % prediction interval of {m} oracle trainings "
                                    f"(counts {min(counts)}..{max(counts)}, sd {sd:.1f})")


def say(*a):
    print("[gpu-test]", *a, flush=True)


def config(i):
    return workloads.WORKLOADS[i]
