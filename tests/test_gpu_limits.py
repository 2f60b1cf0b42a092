"""Edge sizes of the path on the GPU: empty inputs, the longest rows the
training kernels take (d = 16384) against the oracle, rows one float
longer (evaluated, not trained), and more units than the training kernels'
per-unit state holds."""
import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import dev, rel_gap, say, torch_cuda

pytestmark = pytest.mark.gpu

GAP = 1e-4


def test_empty_inputs_are_argument_errors():
    torch = torch_cuda()
    m = som.Map(3, 4, 8, seed=0)
    before = m.weights.cpu().numpy()
    X0 = torch.zeros((0, 8), dtype=torch.float32, device="cuda")
    calls = [
        lambda: m.train(X0, 1, 0.5, 0.1, 2.0, 1.0),
        lambda: m.train_batch(X0, 1, 2.0, 1.0),
        lambda: m.bmu(X0),
        lambda: m.bmu(X0, second=True),
        lambda: m.qe(X0),
        lambda: m.te(X0),
        lambda: m.evaluate(X0),
        # n = 0 rows of CSR, through the ABI (the binding refuses such an
        # indptr itself)
        lambda: som.som_train_csr(m.handle, torch.zeros(1, dtype=torch.int64, device="cuda"),
                                  None, None, 0, 1, som.make_schedule(0.5, 0.1, 2.0, 1.0)),
    ]
    for i, call in enumerate(calls):
        with pytest.raises(som.SomError) as e:
            call()
        assert e.value.name == "SOM_E_ARG", i
    m.synchronize()
    assert np.array_equal(m.weights.cpu().numpy(), before)
    m.close()


@pytest.mark.parametrize("variant", ["", "5"])   # planner's choice (column walk), blocked
@pytest.mark.parametrize("rows,cols,n,epochs", [(2, 3, 7, 2), (3, 4, 13, 1)])
def test_longest_trainable_rows_follow_the_oracle(rows, cols, n, epochs, variant, monkeypatch):
    if variant:
        monkeypatch.setenv("SOM_TRAIN_VARIANT", variant)
    d = 16384  # 4 * 256 lanes * 16 float4: the longest row a training kernel holds
    X = workloads.gaussian_mixture(n, d, 3, 0.2, seed=9)
    order = workloads.epoch_orders(n, epochs, 4)
    s = oracle.schedule(0.5, 0.05, 2.0, 0.5)
    W0 = oracle.init_uniform(5, rows * cols, d)
    m = som.Map(rows, cols, d, seed=5)
    trace = dev(np.full(epochs * n, -1, np.int32))
    m.train(dev(X), epochs, 0.5, 0.05, 2.0, 0.5, order=dev(order), bmu_trace=trace)
    say("d = 16384", rows, cols, "plan", m.plan())
    got = trace.cpu().numpy()
    Wo, tr = oracle.train(W0, rows, cols, X, order, s, trace=True)
    if np.array_equal(got, tr):
        err = np.abs(m.weights.cpu().numpy().astype(np.float64) - Wo).max()
        say(f"  identical BMUs for {len(tr)} steps, max|dW| = {err:.2e}")
        assert err <= 1e-4
    else:
        k = int(np.argmax(got != tr))
        Wk, _ = oracle.train(W0, rows, cols, X, order[:k], s, total_steps=epochs * n)
        Ds = np.sort(oracle.distances(Wk, X[order[k]]))
        assert (Ds[1] - Ds[0]) / Ds[0] <= GAP, "divergence without a near tie"
    m.close()


def test_rows_beyond_the_training_kernels_are_evaluated_not_trained():
    rows, cols, d, n = 3, 3, 16385, 40
    X = workloads.gaussian_mixture(n, d, 3, 0.2, seed=2)
    W = workloads.random_weights(rows * cols, d, 3, -1.0, 1.0)
    m = som.Map(rows, cols, d, seed=0)
    m.weights = dev(W)
    with pytest.raises(som.SomError) as e:
        m.plan()
    assert e.value.name == "SOM_E_UNSUPPORTED"
    with pytest.raises(som.SomError) as e:
        m.train(dev(X), 1, 0.5, 0.1, 2.0, 1.0)
    assert e.value.name == "SOM_E_UNSUPPORTED"
    m.synchronize()
    assert np.array_equal(m.weights.cpu().numpy(), W)   # nothing was launched
    # the batched BMU takes any row length
    got = m.bmu(dev(X)).cpu().numpy()
    o = oracle.evaluate(W, rows, cols, X)
    clear = rel_gap(o["d1"], o["d2"]) > GAP
    assert clear.mean() > 0.9
    assert np.array_equal(got[clear], o["c1"][clear])
    m.close()


def test_more_units_than_the_training_state_holds_is_unsupported():
    # 1,049,600 units at d = 4: above the 4096 units per workgroup (on 256
    # workgroups) that the blocked kernel's per-unit LDS state holds
    m = som.Map(1025, 1024, 4, seed=0)
    with pytest.raises(som.SomError) as e:
        m.plan()
    assert e.value.name == "SOM_E_UNSUPPORTED"
    X = dev(workloads.gaussian_mixture(16, 4, 2, 0.1, seed=0))
    with pytest.raises(som.SomError) as e:
        m.train(X, 1, 0.5, 0.1, 2.0, 1.0)
    assert e.value.name == "SOM_E_UNSUPPORTED"
    # evaluation still runs on a map that size
    idx = m.bmu(X).cpu().numpy()
    assert idx.min() >= 0 and idx.max() < 1025 * 1024
    m.close()
