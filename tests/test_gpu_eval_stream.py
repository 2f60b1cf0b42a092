"""som_evaluate (the BMU, QE and TE of every sample from one BMU search)
against the separate calls and the oracle, and the in-place stream that
serves as the training kernels' memory reference."""
import ctypes as C

import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som
import workloads
from gpu_util import dev, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows,cols,d,n,topology", [(7, 9, 37, 301, som.RECT),
                                                    (12, 10, 256, 1000, som.HEX),
                                                    (1, 1, 8, 5, som.RECT)])
def test_evaluate_equals_separate_calls_and_oracle(rows, cols, d, n, topology):
    say("evaluate", rows, cols, d, n, topology)
    W = workloads.random_weights(rows * cols, d, seed=3)
    X = workloads.random_weights(n, d, seed=4)
    m = som.Map(rows, cols, d, seed=0, topology=topology)
    m.weights = W
    Xd = dev(X)
    idx, qe, te = m.evaluate(Xd)
    assert np.array_equal(idx.cpu().numpy(), m.bmu(Xd).cpu().numpy())
    assert qe == m.qe(Xd)
    assert te == m.te(Xd)
    _, qe2, te2 = m.evaluate(Xd, with_bmu=False)
    assert (qe2, te2) == (qe, te)
    ev = oracle.evaluate(W.astype(np.float64), rows, cols, X, topology=topology)
    assert qe == pytest.approx(ev["qe"], rel=1e-5)
    # every sample here has a clear top-two gap, so TE is exact
    assert te == ev["te"]
    assert np.array_equal(idx.cpu().numpy(), ev["c1"])
    m.close()


def test_evaluate_argument_errors():
    torch = torch_cuda()
    m = som.Map(3, 3, 16, seed=0)
    X = torch.zeros((10, 16), dtype=torch.float32, device="cuda")
    L = som.lib()
    q = C.c_double()
    assert L.som_evaluate(m.handle, X.data_ptr(), 10, None, None, None) == 1
    assert L.som_evaluate(m.handle, X.data_ptr(), 0, None, C.byref(q), None) == 1
    assert L.som_evaluate(m.handle, None, 10, None, C.byref(q), None) == 1
    host = np.zeros((10, 16), np.float32)
    assert L.som_evaluate(m.handle, host.ctypes.data, 10, None, C.byref(q), None) == 1
    with pytest.raises(ValueError):
        m.evaluate(torch.zeros((10, 15), dtype=torch.float32, device="cuda"))
    m.close()


@pytest.mark.parametrize("nbytes,grid,passes", [(16, 1, 1), (4096 * 16 + 48, 7, 3),
                                                (1 << 20, 256, 2), (123456 * 16, 1024, 1)])
def test_stream_inplace_leaves_the_buffer_unchanged(nbytes, grid, passes):
    torch = torch_cuda()
    say("stream", nbytes, grid, passes)
    rng = np.random.default_rng(nbytes)
    host = rng.standard_normal(nbytes // 4 + 8).astype(np.float32)
    buf = dev(host)
    som.som_stream_inplace(buf, nbytes, passes, grid, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert np.array_equal(buf.cpu().numpy(), host)


def test_stream_inplace_argument_errors():
    torch = torch_cuda()
    buf = torch.zeros(1024, dtype=torch.float32, device="cuda")
    L = som.lib()
    p = buf.data_ptr()
    assert L.som_stream_inplace(None, 4096, 1, 1, None) == 1
    assert L.som_stream_inplace(p, 4095, 1, 1, None) == 1
    assert L.som_stream_inplace(p, 0, 1, 1, None) == 1
    assert L.som_stream_inplace(p, 4096, 0, 1, None) == 1
    assert L.som_stream_inplace(p, 4096, 1, 0, None) == 1
    assert L.som_stream_inplace(p, 4096, 1, 1025, None) == 1
    assert L.som_stream_inplace(p + 4, 4096, 1, 1, None) == 1
    host = np.zeros(1024, np.float32)
    assert L.som_stream_inplace(host.ctypes.data, 4096, 1, 1, None) == 1
    torch.cuda.synchronize()
