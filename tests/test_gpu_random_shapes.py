"""Seeded random shapes against the oracle: map sizes, row lengths (edge
values of the float4 slicing and random ones), run lengths, topologies and
forced kernel plans (variant, grid, sweeper count, rows kept in LDS), in
three families:

  * any: everything the planner accepts (a forced plan it refuses raises
    before any launch and is skipped);
  * wide: the four-sweeper streamed kernel (rows of 385-512 float4, few
    workgroups, 5-step blocks);
  * cols: the column walk (rows of 3073-16384 floats, at most 10 per
    workgroup, 8-step blocks, two windows of rows).

Each case trains on the GPU and must follow the oracle's BMU sequence until
an oracle near tie (relative top-two gap <= 1e-4), with weights within
1e-4 where the whole sequence agrees.  A fourth family draws evaluation
shapes (up to 80 x 80 units, 3000 samples) for the batched BMU, QE and TE."""
import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import dev, rel_gap, say

pytestmark = pytest.mark.gpu

GAP = 1e-4
ENV = ("SOM_TRAIN_VARIANT", "SOM_TRAIN_GRID", "SOM_TRAIN_SWEEPERS", "SOM_TRAIN_LDS_ROWS")
D_EDGE = [1, 3, 4, 5, 63, 64, 65, 127, 128, 255, 256, 257, 511, 512, 513, 1023, 1024, 1025,
          1535, 1536, 1537, 2047, 2048, 2049, 3071, 3072, 3073, 5119, 5120, 5121, 12288, 16384]


def _cases(family, seed, count):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        env = {}
        if family == "wide":
            g = int(rng.choice([1, 2, 3, 4, 8, 16]))
            rows, cols = int(rng.integers(2, 17)), int(rng.integers(2, 17))
            while rows * cols > 64 * g:
                cols = max(1, cols // 2)
            d = int(rng.integers(1537, 2049))
            env = {"SOM_TRAIN_VARIANT": "4", "SOM_TRAIN_SWEEPERS": "4", "SOM_TRAIN_GRID": str(g)}
        elif family == "cols":
            g = int(rng.choice([1, 2, 3, 4, 8, 16, 32]))
            rows, cols = int(rng.integers(1, 11)), int(rng.integers(1, 11))
            while rows * cols > 10 * g:
                cols = max(1, cols // 2)
                rows = max(1, rows - 1)
            d = int(rng.integers(3073, 16385))
            env = {"SOM_TRAIN_VARIANT": "4", "SOM_TRAIN_GRID": str(g)}
        else:
            rows, cols = int(rng.integers(1, 33)), int(rng.integers(1, 33))
            d = int(rng.choice(D_EDGE)) if rng.random() < 0.7 else int(rng.integers(1, 16385))
            v = str(rng.choice(["", "1", "2", "3", "4", "5"]))
            if v:
                env["SOM_TRAIN_VARIANT"] = v
            if rng.random() < 0.4:
                env["SOM_TRAIN_GRID"] = str(int(rng.choice([1, 2, 3, 8, 16, 64, 256])))
            if rng.random() < 0.3:
                env["SOM_TRAIN_SWEEPERS"] = str(int(rng.choice([3, 4])))
        if family != "any" or rng.random() < 0.3:
            if rng.random() < 0.6:
                env["SOM_TRAIN_LDS_ROWS"] = str(int(rng.choice([0, 1, 2, 3, 64])))
        n = int(rng.integers(1, 30))
        epochs = int(rng.integers(1, 3))
        topology = som.HEX if rng.random() < 0.3 else som.RECT
        out.append((rows, cols, d, n, epochs, topology, tuple(sorted(env.items()))))
    return out


CASES = ([("any", 11, c) for c in _cases("any", 11, 16)] +
         [("wide", 12, c) for c in _cases("wide", 12, 10)] +
         [("cols", 13, c) for c in _cases("cols", 13, 10)])


@pytest.mark.parametrize("family,seed,case", CASES,
                         ids=[f"{f}-{i}" for i, (f, _, _) in enumerate(CASES)])
def test_random_shape_follows_the_oracle(family, seed, case, monkeypatch):
    rows, cols, d, n, epochs, topology, env = case
    for k in ENV:
        monkeypatch.delenv(k, raising=False)
    for k, v in env:
        monkeypatch.setenv(k, v)
    say("random", family, rows, cols, d, n, epochs, topology, dict(env))
    k0 = rows * 7919 + cols * 104729 + d  # per-case data seed
    X = workloads.gaussian_mixture(n, d, 3, 0.2, seed=k0 % 100003)
    order = workloads.epoch_orders(n, epochs, k0 % 997)
    sig0 = max(rows, cols) / 2.0
    s = oracle.schedule(0.4, 0.02, sig0, 0.5)
    W0 = oracle.init_uniform(k0 % 65521, rows * cols, d)
    m = som.Map(rows, cols, d, seed=k0 % 65521, topology=topology)
    try:
        plan = m.plan()
    except som.SomError as e:
        m.close()
        assert family == "any", (family, e.name)
        pytest.skip(f"plan refused before launch: {e.name}")
    if family == "wide":
        assert (plan["variant"], plan["block"], plan["block_steps"]) == (2, 320, 5)
    if family == "cols":
        assert (plan["variant"], plan["block_steps"]) == (4, 8)
    trace = dev(np.full(epochs * n, -1, np.int32))
    m.train(dev(X), epochs, 0.4, 0.02, sig0, 0.5, order=dev(order), bmu_trace=trace)
    got = trace.cpu().numpy()
    Wo, tr = oracle.train(W0, rows, cols, X, order, s, topology=topology, trace=True)
    if np.array_equal(got, tr):
        err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
        say(f"  plan {plan}: identical BMUs for {len(tr)} steps, max|dW| = {err:.2e}")
        assert err <= 1e-4
    else:
        k = int(np.argmax(got != tr))
        Wk, _ = oracle.train(W0, rows, cols, X, order[:k], s, total_steps=epochs * n,
                             topology=topology)
        Ds = np.sort(oracle.distances(Wk, X[order[k]]))
        say(f"  plan {plan}: identical BMUs for {k}/{len(tr)} steps")
        assert len(Ds) > 1 and (Ds[1] - Ds[0]) / Ds[0] <= GAP, "divergence without a near tie"
    m.close()


# ---------------------------------------------------------------- batched BMU
def _bmu_cases(seed, count):
    """Random (rows, cols, d, n, topology): up to 80 x 80 units, d at the
    slicing edges or random, n up to 3000, with n N d kept within what the
    oracle evaluates in about a second."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        rows, cols = int(rng.integers(1, 81)), int(rng.integers(1, 81))
        d = int(rng.choice(D_EDGE)) if rng.random() < 0.5 else int(rng.integers(1, 12001))
        n = int(rng.integers(1, 3001))
        while n > 1 and n * rows * cols * d > 1.5e9:
            n //= 2
        out.append((rows, cols, d, n, som.HEX if rng.random() < 0.3 else som.RECT))
    return out


@pytest.mark.parametrize("case", _bmu_cases(21, 24), ids=[f"bmu-{i}" for i in range(24)])
def test_random_shape_batched_bmu_and_quality_follow_the_oracle(case):
    """BMUs and second BMUs where the oracle's gaps are clear, the BMU
    distance everywhere, QE to 1e-5 and the TE count up to the samples whose
    BMU or second BMU is an oracle near tie, through som_bmu2 and
    som_evaluate (the fused or split candidate search the planner picks)."""
    rows, cols, d, n, topology = case
    say("random bmu", rows, cols, d, n, topology)
    k0 = rows * 7919 + cols * 104729 + d + n
    X = workloads.gaussian_mixture(n, d, 8, 0.2, seed=k0 % 100003)
    W = workloads.random_weights(rows * cols, d, k0 % 65521, -1.0, 1.0)
    m = som.Map(rows, cols, d, seed=0, topology=topology)
    m.weights = dev(W)
    Xd = dev(X)
    idx, idx2, d1 = (t.cpu().numpy() for t in m.bmu(Xd, second=True))
    _, qe, te = m.evaluate(Xd, with_bmu=False)
    m.close()
    W64 = W.astype(np.float64)
    ev = oracle.evaluate(W64, rows, cols, X, topology=topology)
    D = np.stack([oracle.distances(W64, X[i]) for i in range(n)])
    Ds = np.sort(D, axis=1)
    g1 = rel_gap(Ds[:, 0], Ds[:, 1]) if D.shape[1] > 1 else np.full(n, np.inf)
    g2 = rel_gap(Ds[:, 1], Ds[:, 2]) if D.shape[1] > 2 else np.full(n, np.inf)
    sure = g1 > GAP
    assert np.array_equal(idx[sure], ev["c1"][sure])
    assert np.all(np.abs(d1 - ev["d1"]) <= 1e-5 * np.maximum(ev["d1"], 1e-3) + 1e-6)
    if rows * cols == 1:
        assert np.all(idx2 == -1)
    else:
        sure2 = sure & (g2 > GAP)
        assert np.array_equal(idx2[sure2], ev["c2"][sure2])
    assert qe == pytest.approx(ev["qe"], rel=1e-5)
    unsure = int(np.sum(~(sure & (g2 > GAP))))
    assert abs(round(te * n) - round(ev["te"] * n)) <= unsure
