"""The synthetic inputs have the shapes and statistics the workloads call for."""
import numpy as np
import pytest

import workloads as w


def test_workload_table():
    assert len(w.WORKLOADS) == 5
    c = w.WORKLOADS
    assert (c[0].n, c[0].d, c[0].units, c[0].steps) == (200, 500, 100, 2000)
    assert (c[1].n, c[1].d, c[1].units, c[1].steps) == (2000, 2000, 400, 40000)
    assert (c[2].n, c[2].d, c[2].units, c[2].steps) == (5000, 5000, 900, 250000)
    assert (c[3].n, c[3].d, c[3].units, c[3].steps) == (20000, 10000, 2500, 400000)
    assert (c[4].n, c[4].d, c[4].units, c[4].steps) == (100000, 2048, 10000, 500000)
    assert [x.nnz_per_row for x in c[:4]] == [10, 20, 25, 30]


@pytest.mark.parametrize("i", [0, 1])
def test_tfidf_rows_are_sparse_unit_norm_and_deterministic(i):
    cfg = w.WORKLOADS[i]
    X = w.make_data(cfg)
    assert X.shape == (cfg.n, cfg.d) and X.dtype == np.float32
    nnz = (X != 0).sum(axis=1)
    assert np.all(nnz <= cfg.nnz_per_row)
    assert nnz.mean() >= 0.9 * cfg.nnz_per_row        # idf = 0 terms are rare
    norms = np.sqrt((X.astype(np.float64) ** 2).sum(axis=1))
    assert np.all(np.abs(norms[norms > 0] - 1.0) < 1e-6)
    assert np.all(X >= 0)
    assert np.array_equal(X, w.make_data(cfg))


def test_tfidf_topics_use_different_vocabularies():
    X, topic = w.tfidf_like(400, 300, 0.05, 4, seed=9, return_topics=True)
    support = [(X[topic == k] != 0).sum(axis=0) for k in range(4)]
    heads = [set(np.argsort(-s)[:10].tolist()) for s in support]
    for a in range(4):
        for b in range(a + 1, 4):
            assert len(heads[a] & heads[b]) <= 4


def test_tfidf_term_frequencies_follow_zipf_head():
    X = w.tfidf_like(2000, 1000, 0.02, 1, seed=4)
    df = (X != 0).sum(axis=0)
    top = np.sort(df)[::-1]
    # rank-1 term appears in far more documents than a mid-rank term
    assert top[0] > 5 * top[100]


def test_gaussian_mixture_statistics():
    X, lab = w.gaussian_mixture(4000, 64, 4, 0.2, seed=1, return_labels=True)
    assert X.dtype == np.float32 and X.shape == (4000, 64)
    for k in range(4):
        Xk = X[lab == k].astype(np.float64)
        assert abs(Xk.std(axis=0).mean() - 0.2) < 0.01
        mu = Xk.mean(axis=0)
        assert np.all(np.abs(mu) < 1.05)
    # chunked generation gives the same stream as one block
    Xa = w.gaussian_mixture(100, 8, 3, 0.2, seed=5, chunk=7)
    Xb = w.gaussian_mixture(100, 8, 3, 0.2, seed=5, chunk=1000)
    assert np.array_equal(Xa, Xb)


def test_epoch_orders_are_fresh_permutations():
    o = w.epoch_orders(50, 4, seed=3)
    assert o.dtype == np.int32 and o.shape == (200,)
    for e in range(4):
        assert sorted(o[e * 50:(e + 1) * 50].tolist()) == list(range(50))
    assert not np.array_equal(o[:50], o[50:100])
    assert np.array_equal(w.epoch_orders(50, 2, seed=3, first_epoch=2), o[100:])
