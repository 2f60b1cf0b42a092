"""The C ABI library loads, exports every symbol som.h declares and rejects
bad arguments on the host before any device work (no GPU needed)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle
import paper_1905_09598_amd as som

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "som.h")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|som_status)\s*(som_\w+)\s*\(",
                                 text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    L = som.lib()
    names = declared_symbols()
    assert len(names) >= 14
    assert set(names) == set(som.EXPORTED)
    for name in names:
        assert hasattr(L, name), name


def header_status_codes():
    body = re.search(r"typedef enum som_status \{(.*?)\} som_status;", open(HEADER).read(),
                     flags=re.S).group(1)
    return {int(v): k for k, v in re.findall(r"(SOM_\w+)\s*=\s*(\d+)", body)}


def test_status_strings():
    codes = header_status_codes()
    assert codes == som.STATUS                     # the binding's names are the header's
    assert codes[8] == "SOM_E_NONFINITE" and codes[5] == "SOM_E_TIMEOUT"
    assert som.som_status_string(0) == "ok"
    texts = {som.som_status_string(code) for code in codes if code}
    assert len(texts) == len(codes) - 1 and "unknown status" not in texts
    assert som.som_status_string(99) == "unknown status"


def test_memory_cap_refuses_a_map_before_device_work(monkeypatch):
    # a 10 x 10 map of d = 64 needs 100 rows of at least 64 floats
    monkeypatch.setenv("SOM_MAX_BYTES", str(100 * 64 * 4 - 1))
    with pytest.raises(som.SomError) as e:
        som.som_create(10, 10, 64, 0)
    assert e.value.name == "SOM_E_OOM"
    monkeypatch.setenv("SOM_MAX_BYTES", "1")
    with pytest.raises(som.SomError) as e:
        som.som_create(1, 1, 1, 0)
    assert e.value.name == "SOM_E_OOM"


@pytest.mark.parametrize("rows,cols,d", [(0, 3, 4), (3, 0, 4), (3, 3, 0), (-1, 2, 2),
                                         (4097, 4096, 1)])
def test_create_rejects_bad_shapes_before_device_work(rows, cols, d):
    with pytest.raises(som.SomError) as e:
        som.som_create(rows, cols, d, 0)
    assert e.value.name == "SOM_E_ARG"


def test_create_rejects_null_out_pointer():
    assert som.lib().som_create(2, 2, 4, C.c_uint64(0), None) == 1


def test_calls_on_null_map_are_argument_errors():
    L = som.lib()
    s = som.make_schedule(0.5, 0.01, 3.0, 1.0)
    assert L.som_train(None, None, 10, 1, C.byref(s)) == 1
    assert L.som_train_csr(None, None, None, None, 10, 1, C.byref(s)) == 1
    assert L.som_train_batch(None, None, 10, 1, 2.0, 1.0, 1) == 1
    assert L.som_bmu(None, None, 10, None) == 1
    assert L.som_bmu2(None, None, 10, None, None, None) == 1
    assert L.som_synchronize(None) == 1
    assert L.som_set_topology(None, 0) == 1
    assert L.som_get_weights(None, None) == 1
    assert L.som_set_weights(None, None) == 1
    v = C.c_double()
    assert L.som_quantization_error(None, None, 5, C.byref(v)) == 1
    assert L.som_topographic_error(None, None, 5, C.byref(v)) == 1
    assert L.som_destroy(None) == 0
    assert L.som_get_shape(None, None, None, None, None) == 1
    assert L.som_train_plan(None, None, None, None, None) == 1
    assert L.som_evaluate(None, None, 5, None, C.byref(v), None) == 1
    assert L.som_stream_inplace(None, 16, 1, 1, None) == 1
    assert L.som_stream_inplace(None, 15, 1, 1, None) == 1


def test_shuffle_argument_errors():
    with pytest.raises(som.SomError):
        som.som_shuffle(0, 0, 0)
    with pytest.raises(som.SomError):
        som.som_shuffle(0, -1, 5)


@pytest.mark.parametrize("seed,epoch,n", [(0, 0, 1), (0, 0, 2), (7, 3, 100), (123, 9, 5000)])
def test_library_shuffle_matches_independent_oracle_shuffle(seed, epoch, n):
    lib_perm = som.som_shuffle(seed, epoch, n)
    assert np.array_equal(lib_perm, oracle.shuffle(seed, epoch, n))
    assert sorted(lib_perm.tolist()) == list(range(n))


def test_library_size_heuristic_equals_independent_oracle():
    rng = np.random.default_rng(5)
    cases = [(100, 4.0, 1.0), (100, 1000.0, 1.0), (100, 0.0, 0.0), (2000, 2.0, 1.0),
             (1, 1.0, 1.0), (637, 3.7, 1.2)]
    for _ in range(200):
        m = int(rng.integers(1, 200000))
        l1 = float(rng.uniform(0.0, 10.0))
        cases.append((m, l1, float(rng.uniform(0.0, l1))))
    for m, l1, l2 in cases:
        assert som.som_suggest_size(m, l1, l2) == oracle.suggest_size(m, l1, l2), (m, l1, l2)


def test_pca_and_linear_init_argument_errors():
    L = som.lib()
    lam = (C.c_double * 2)()
    assert L.som_pca2(None, 10, 4, None, lam, None, None, None) == 1
    assert L.som_pca2(1, 0, 4, None, lam, None, None, None) == 1
    assert L.som_pca2(1, 10, 0, None, lam, None, None, None) == 1
    assert L.som_pca2(1, 10, 4, None, None, None, None, None) == 1
    assert L.som_init_linear(None, 1, 10) == 1
    r = C.c_int32()
    assert L.som_suggest_size(0, 1.0, 1.0, C.byref(r), None, None) == 1
    assert L.som_suggest_size(10, 1.0, 2.0, C.byref(r), None, None) == 1
    assert L.som_suggest_size(10, -1.0, -2.0, C.byref(r), None, None) == 1
    assert L.som_suggest_size(10, float("nan"), 0.0, C.byref(r), None, None) == 1
