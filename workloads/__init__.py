"""Seeded synthetic inputs for the online-SOM hot path.

This module only draws inputs.  It holds none of the method's arithmetic: no
distances, no best-matching unit, no neighbourhood, no update.  Both the HIP
library's tests and the fp64 oracle's tests consume the arrays it returns, so
the two sides see bit-identical inputs.

Stand-ins for the paper's data.  The paper trains on TF and TF-IDF
document-term matrices of bank complaints, L2-normalised before training
(Sec. 6B, Eq. 2 and Sec. 6D; Table 1 gives 440-676 documents by 3917-4545
terms).  Those corpora are not available, so every workload here is synthetic:

* ``tfidf_like``: documents drawn from latent topics.  Each topic has its own
  random permutation of the vocabulary.  Each document draws a fixed number of
  distinct term ranks from a Zipf(s) law truncated to [1, d], maps them through
  its topic's permutation, and draws term frequencies from Poisson(2)
  conditioned on being at least 1.  The inverse document frequency follows
  Eq. 2 with the natural log, idf_t = ln(n / df_t).  Rows are x = tf * idf,
  L2-normalised (a zero row stays zero, Sec. 6D), and stored dense fp32.
* ``gaussian_mixture``: K cluster means drawn U[-1, 1]^d, each sample is its
  cluster's mean plus N(0, sd^2 I) noise, not normalised.

Every array is produced in float64 by numpy's PCG64 generator and rounded
once to float32, so the bits do not depend on the host's SIMD width.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional

import numpy as np

__all__ = [
    "SomConfig", "WORKLOADS", "tfidf_like", "gaussian_mixture", "make_data",
    "epoch_orders", "sha256_of",
]


@dataclasses.dataclass(frozen=True)
class SomConfig:
    """One training workload: data shape, map shape and decay schedule.

    ``lr`` decays linearly from ``lr0`` to ``lr1`` and the neighbourhood
    radius ``sigma`` exponentially from ``sigma0`` to ``sigma1`` over the
    ``epochs * n`` per-sample steps.
    """

    name: str
    n: int
    d: int
    rows: int
    cols: int
    epochs: int
    lr0: float
    lr1: float
    sigma0: float
    sigma1: float
    kind: str                      # "tfidf" or "mixture"
    density: float = 0.0           # fraction of nonzero terms per document
    topics: int = 1
    zipf_s: float = 1.1
    clusters: int = 0
    cluster_sd: float = 0.0
    data_seed: int = 0
    init_seed: int = 0
    shuffle_seed: int = 0

    @property
    def units(self) -> int:
        return self.rows * self.cols

    @property
    def steps(self) -> int:
        return self.epochs * self.n

    @property
    def nnz_per_row(self) -> int:
        return int(round(self.density * self.d))


# Five workloads: a tiny one the oracle finishes in well under a second, three
# TF-IDF-shaped ones of growing size and a dense Gaussian-mixture stress case.
WORKLOADS = (
    SomConfig("tfidf_n200_d500_map10x10", n=200, d=500, rows=10, cols=10,
              epochs=10, lr0=0.5, lr1=0.01, sigma0=5.0, sigma1=1.0,
              kind="tfidf", density=0.02, topics=1, data_seed=0),
    SomConfig("tfidf_n2000_d2000_map20x20", n=2000, d=2000, rows=20, cols=20,
              epochs=20, lr0=0.5, lr1=0.01, sigma0=10.0, sigma1=1.0,
              kind="tfidf", density=0.01, topics=8, data_seed=1),
    SomConfig("tfidf_n5000_d5000_map30x30", n=5000, d=5000, rows=30, cols=30,
              epochs=50, lr0=0.3, lr1=0.005, sigma0=15.0, sigma1=1.0,
              kind="tfidf", density=0.005, topics=16, data_seed=2),
    SomConfig("tfidf_n20000_d10000_map50x50", n=20000, d=10000, rows=50,
              cols=50, epochs=20, lr0=0.3, lr1=0.005, sigma0=25.0,
              sigma1=1.0, kind="tfidf", density=0.003, topics=32,
              data_seed=3),
    SomConfig("mixture_n100000_d2048_map100x100", n=100000, d=2048,
              rows=100, cols=100, epochs=5, lr0=0.5, lr1=0.01, sigma0=50.0,
              sigma1=1.0, kind="mixture", clusters=16, cluster_sd=0.2,
              data_seed=4),
)


def _truncated_zipf_cdf(d: int, s: float) -> np.ndarray:
    ranks = np.arange(1, d + 1, dtype=np.float64)
    p = ranks ** (-s)
    cdf = np.cumsum(p)
    return cdf / cdf[-1]


def _distinct_ranks(rng: np.random.Generator, cdf: np.ndarray, k: int) -> np.ndarray:
    """k distinct 0-based ranks from the truncated Zipf law, duplicates rejected.

    Draws are taken in order and a rank already drawn is skipped, so the
    result is a sample without replacement in draw order.
    """
    d = cdf.shape[0]
    if k > d:
        raise ValueError("more distinct terms than vocabulary")
    got: list[int] = []
    seen: set[int] = set()
    while len(got) < k:
        u = rng.random(2 * (k - len(got)) + 4)
        idx = np.minimum(np.searchsorted(cdf, u, side="right"), d - 1)
        for r in idx.tolist():
            if r not in seen:
                seen.add(r)
                got.append(r)
                if len(got) == k:
                    break
    return np.asarray(got, dtype=np.int64)


def _poisson_at_least_one(rng: np.random.Generator, lam: float, k: int) -> np.ndarray:
    tf = rng.poisson(lam, size=k)
    while True:
        zero = tf == 0
        nz = int(zero.sum())
        if nz == 0:
            return tf.astype(np.float64)
        tf[zero] = rng.poisson(lam, size=nz)


def tfidf_like(n: int, d: int, density: float, topics: int, seed: int,
               zipf_s: float = 1.1, return_topics: bool = False):
    """TF-IDF-shaped document vectors, L2-normalised, dense fp32 (n, d)."""
    if n <= 0 or d <= 0:
        raise ValueError("n and d must be positive")
    k = max(1, int(round(density * d)))
    rng = np.random.Generator(np.random.PCG64(seed))
    perms = np.stack([rng.permutation(d) for _ in range(topics)])
    topic = rng.integers(0, topics, size=n)
    cdf = _truncated_zipf_cdf(d, zipf_s)
    cols = np.empty((n, k), dtype=np.int64)
    tf = np.empty((n, k), dtype=np.float64)
    for i in range(n):
        ranks = _distinct_ranks(rng, cdf, k)
        cols[i] = perms[topic[i]][ranks]
        tf[i] = _poisson_at_least_one(rng, 2.0, k)
    df = np.bincount(cols.ravel(), minlength=d).astype(np.float64)
    idf = np.zeros(d, dtype=np.float64)
    present = df > 0
    idf[present] = np.log(n / df[present])
    val = tf * idf[cols]
    norm = np.sqrt(np.sum(val * val, axis=1))
    scale = np.where(norm > 0.0, 1.0 / np.where(norm > 0.0, norm, 1.0), 0.0)
    val = val * scale[:, None]
    X = np.zeros((n, d), dtype=np.float32)
    rows = np.repeat(np.arange(n), k)
    X[rows, cols.ravel()] = val.ravel().astype(np.float32)
    if return_topics:
        return X, topic.astype(np.int32)
    return X


def gaussian_mixture(n: int, d: int, clusters: int, sd: float, seed: int,
                     return_labels: bool = False, chunk: int = 8192):
    """Samples mu_k + sd * N(0, I), k uniform over ``clusters`` means U[-1,1]^d."""
    rng = np.random.Generator(np.random.PCG64(seed))
    means = rng.uniform(-1.0, 1.0, size=(clusters, d))
    label = rng.integers(0, clusters, size=n)
    X = np.empty((n, d), dtype=np.float32)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        z = rng.standard_normal((e - s, d))
        X[s:e] = (means[label[s:e]] + sd * z).astype(np.float32)
    if return_labels:
        return X, label.astype(np.int32)
    return X


def make_data(cfg: SomConfig) -> np.ndarray:
    """The (n, d) fp32 data matrix of a workload."""
    if cfg.kind == "tfidf":
        return tfidf_like(cfg.n, cfg.d, cfg.density, cfg.topics,
                          cfg.data_seed, cfg.zipf_s)
    if cfg.kind == "mixture":
        return gaussian_mixture(cfg.n, cfg.d, cfg.clusters, cfg.cluster_sd,
                                cfg.data_seed)
    raise ValueError(f"unknown workload kind {cfg.kind!r}")


def epoch_orders(n: int, epochs: int, seed: int = 0,
                 first_epoch: int = 0) -> np.ndarray:
    """Sample order for ``epochs`` epochs: one fresh permutation per epoch.

    Epoch e uses the PCG64 stream seeded with (seed, e), so any range of
    epochs can be produced on its own.  Returns int32 of length epochs * n.
    """
    out = np.empty(epochs * n, dtype=np.int32)
    for e in range(epochs):
        rng = np.random.Generator(np.random.PCG64([seed, first_epoch + e]))
        out[e * n:(e + 1) * n] = rng.permutation(n).astype(np.int32)
    return out


def sha256_of(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def small_tfidf(n: int, d: int, seed: int, density: float = 0.02,
                topics: int = 2) -> np.ndarray:
    """A small TF-IDF-shaped matrix for unit tests (at least one term per row)."""
    return tfidf_like(n, d, max(density, 1.0 / d), topics, seed)


def random_weights(N: int, d: int, seed: int, low: float = 0.0,
                   high: float = 1.0) -> np.ndarray:
    """Arbitrary fp32 prototype matrices for single-step tests."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.uniform(low, high, size=(N, d)).astype(np.float32)
