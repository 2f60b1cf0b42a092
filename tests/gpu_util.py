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


def say(*a):
    print("[gpu-test]", *a, flush=True)


def config(i):
    return workloads.WORKLOADS[i]
