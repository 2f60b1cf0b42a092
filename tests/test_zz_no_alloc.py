"""som_bmu2_noalloc (the evaluation entry point that allocates nothing)
against som_bmu2 through the C ABI: identical BMUs, second BMUs and BMU
distances on two calls in a row, the second with fewer samples, and the
size limit of its fixed scratch."""
import ctypes as C

import numpy as np
import pytest

import paper_1905_09598_amd as som
import workloads
from gpu_util import dev, say, torch_cuda

pytestmark = pytest.mark.gpu


def _outputs(torch, n):
    return (torch.full((n,), -7, dtype=torch.int32, device="cuda"),
            torch.full((n,), -7, dtype=torch.int32, device="cuda"),
            torch.full((n,), -1.0, dtype=torch.float32, device="cuda"))


def _call(fn, m, X, n, outs, idx=True):
    L = som.lib()
    i1, i2, d1 = outs
    rc = getattr(L, fn)(m.handle, X.data_ptr(), n, i1.data_ptr() if idx else None,
                        i2.data_ptr(), d1.data_ptr())
    assert rc == 0, (fn, som.som_status_string(rc))


@pytest.mark.parametrize("rows,cols,d,n1,n2,topology",
                         [(20, 20, 2000, 2000, 333, som.RECT),
                          (7, 9, 37, 1000, 65, som.HEX),
                          (100, 100, 2048, 40000, 5000, som.RECT)])
def test_noalloc_equals_bmu2_on_two_calls(rows, cols, d, n1, n2, topology):
    torch = torch_cuda()
    say("noalloc", rows, cols, d, n1, n2, topology)
    m = som.Map(rows, cols, d, seed=1, topology=topology)
    X = dev(workloads.random_weights(n1, d, seed=11))
    for n in (n1, n2):
        Xn = X[:n].contiguous()
        ref = _outputs(torch, n)
        got = _outputs(torch, n)
        m._bind_stream()
        _call("som_bmu2", m, Xn, n, ref)
        _call("som_bmu2_noalloc", m, Xn, n, got)
        torch.cuda.synchronize()
        for a, b in zip(ref, got):
            assert torch.equal(a, b)
        assert int(ref[0].min()) >= 0
        # with out_idx NULL the BMUs go to the scratch; the other outputs stay
        got2 = _outputs(torch, n)
        _call("som_bmu2_noalloc", m, Xn, n, got2, idx=False)
        torch.cuda.synchronize()
        assert torch.equal(got2[1], ref[1]) and torch.equal(got2[2], ref[2])
        assert int(got2[0].min()) == -7 and int(got2[0].max()) == -7
    m.close()


def test_noalloc_rejects_inputs_beyond_its_scratch():
    torch = torch_cuda()
    L = som.lib()
    m = som.Map(16, 16, 64, seed=0)
    # 16 x 256 units, n = 600,000 > 8 MiB of candidate lists (32 bytes a sample)
    n = 600000
    X = torch.zeros((n, 64), dtype=torch.float32, device="cuda")
    i1 = torch.empty(n, dtype=torch.int32, device="cuda")
    m._bind_stream()
    rc = L.som_bmu2_noalloc(m.handle, X.data_ptr(), n, i1.data_ptr(), None, None)
    assert som.STATUS[rc] == "SOM_E_UNSUPPORTED"
    assert L.som_bmu2_noalloc(m.handle, None, n, i1.data_ptr(), None, None) == 1
    assert L.som_bmu2_noalloc(None, X.data_ptr(), n, i1.data_ptr(), None, None) == 1
    # a smaller call still works after the refusal
    rc = L.som_bmu2_noalloc(m.handle, X.data_ptr(), 1000, i1.data_ptr(), None, None)
    assert rc == 0
    torch.cuda.synchronize()
    assert int(i1[:1000].min()) >= 0
    m.close()
