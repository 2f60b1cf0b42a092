"""ctypes wrapper of the fp64 CPU oracle (``som_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg are the only callers.  The HIP library never
imports this module, and this module never imports the HIP library.

All functions take and return numpy arrays.  Weights are float64 (N, d);
data is float32 (n, d) and widened exactly inside the C code.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "som_oracle.c")
# SOM_ORACLE_SANITIZE=1 selects an AddressSanitizer + UndefinedBehaviorSanitizer
# build in a file of its own (the process must have libasan preloaded; see
# run_sanitized.py beside this file).
SANITIZE = os.environ.get("SOM_ORACLE_SANITIZE", "") == "1"
_LIB = os.path.join(_HERE, "libsom_oracle_san.so" if SANITIZE else "libsom_oracle.so")
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer",
                  "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]

RECT, HEX = 0, 1
LINEAR, EXPONENTIAL = 0, 1


class Schedule(C.Structure):
    _fields_ = [("lr0", C.c_double), ("lr1", C.c_double),
                ("lr_decay", C.c_int32),
                ("sigma0", C.c_double), ("sigma1", C.c_double),
                ("sigma_decay", C.c_int32)]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, no FMA contraction;
    with SOM_ORACLE_SANITIZE=1, -O1 under ASan and UBSan instead)."""
    if force or not os.path.exists(_LIB):
        opt = SANITIZE_FLAGS if SANITIZE else ["-O2"]
        cmd = ["gcc", *opt, "-std=gnu11", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-shared", "-fPIC", "-Wall", "-Wextra",
               "-o", _LIB + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = C.CDLL(_LIB)
        dp = C.POINTER(C.c_double)
        fp = C.POINTER(C.c_float)
        ip = C.POINTER(C.c_int32)
        up = C.POINTER(C.c_uint64)
        L.som_oracle_splitmix64.argtypes = [C.c_uint64, C.c_int64, up]
        L.som_oracle_init_uniform.argtypes = [C.c_uint64, C.c_int64, dp]
        L.som_oracle_shuffle.argtypes = [C.c_uint64, C.c_int64, C.c_int64, ip]
        L.som_oracle_schedule_at.argtypes = [C.c_int64, C.c_int64,
                                             C.POINTER(Schedule), dp, dp]
        L.som_oracle_position.argtypes = [C.c_int32, C.c_int32, C.c_int64, dp, dp]
        L.som_oracle_neighbourhood.argtypes = [C.c_int32, C.c_int32, C.c_int32,
                                               C.c_int64, C.c_double, C.c_double, dp]
        L.som_oracle_distances.argtypes = [dp, C.c_int64, C.c_int64, fp, dp]
        L.som_oracle_train.argtypes = [dp, C.c_int32, C.c_int32, C.c_int32,
                                       C.c_int64, fp, C.c_int64, ip, C.c_int64,
                                       C.c_int64, C.c_int64, C.POINTER(Schedule),
                                       ip, C.c_int]
        L.som_oracle_train.restype = C.c_int
        L.som_oracle_train_near_tie.argtypes = [
            dp, C.c_int32, C.c_int32, C.c_int32, C.c_int64, fp, C.c_int64, ip,
            C.c_int64, C.c_int64, C.c_int64, C.POINTER(Schedule), C.c_double,
            C.c_uint64, C.POINTER(C.c_int64), C.c_int]
        L.som_oracle_train_near_tie.restype = C.c_int
        L.som_oracle_evaluate.argtypes = [dp, C.c_int32, C.c_int32, C.c_int32,
                                          C.c_int64, fp, C.c_int64, ip, ip, dp,
                                          dp, dp, dp, C.c_int]
        L.som_oracle_evaluate.restype = C.c_int
        _lib = L
    return _lib


def _p(a, ct):
    return a.ctypes.data_as(C.POINTER(ct))


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def schedule(lr0, lr1, sigma0, sigma1, lr_decay=LINEAR,
             sigma_decay=EXPONENTIAL) -> Schedule:
    return Schedule(float(lr0), float(lr1), int(lr_decay), float(sigma0),
                    float(sigma1), int(sigma_decay))


def splitmix64(seed: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.uint64)
    lib().som_oracle_splitmix64(C.c_uint64(seed), count, _p(out, C.c_uint64))
    return out


def init_uniform(seed: int, N: int, d: int) -> np.ndarray:
    """Initial prototypes U[0,1) on the 2^-24 grid, (N, d) float64."""
    out = np.empty((N, d), dtype=np.float64)
    lib().som_oracle_init_uniform(C.c_uint64(seed), N * d, _p(out, C.c_double))
    return out


def shuffle(seed: int, epoch: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    lib().som_oracle_shuffle(C.c_uint64(seed), epoch, n, _p(out, C.c_int32))
    return out


def schedule_at(t: int, T: int, s: Schedule):
    lr = C.c_double()
    sg = C.c_double()
    lib().som_oracle_schedule_at(t, T, C.byref(s), C.byref(lr), C.byref(sg))
    return lr.value, sg.value


def position(topology: int, cols: int, u: int):
    y = C.c_double()
    x = C.c_double()
    lib().som_oracle_position(topology, cols, u, C.byref(y), C.byref(x))
    return y.value, x.value


def neighbourhood(rows, cols, topology, c, lr, sigma) -> np.ndarray:
    h = np.empty(rows * cols, dtype=np.float64)
    lib().som_oracle_neighbourhood(rows, cols, topology, c, float(lr),
                                   float(sigma), _p(h, C.c_double))
    return h


def distances(W: np.ndarray, x: np.ndarray) -> np.ndarray:
    W = np.ascontiguousarray(W, dtype=np.float64)
    x = np.ascontiguousarray(x, dtype=np.float32)
    N, d = W.shape
    D = np.empty(N, dtype=np.float64)
    lib().som_oracle_distances(_p(W, C.c_double), N, d, _p(x, C.c_float),
                               _p(D, C.c_double))
    return D


def train(W: np.ndarray, rows: int, cols: int, X: np.ndarray,
          order: np.ndarray, s: Schedule, step0: int = 0,
          total_steps: Optional[int] = None, topology: int = RECT,
          nthreads: Optional[int] = None, trace: bool = False):
    """Run len(order) online steps on a float64 copy of W; returns (W, trace)."""
    W = np.array(W, dtype=np.float64, order="C", copy=True)
    X = np.ascontiguousarray(X, dtype=np.float32)
    order = np.ascontiguousarray(order, dtype=np.int32)
    n, d = X.shape
    assert W.shape == (rows * cols, d)
    nsteps = order.shape[0]
    T = step0 + nsteps if total_steps is None else int(total_steps)
    tr = np.full(nsteps, -1, dtype=np.int32) if trace else None
    rc = lib().som_oracle_train(
        _p(W, C.c_double), rows, cols, topology, d, _p(X, C.c_float), n,
        _p(order, C.c_int32), nsteps, step0, T, C.byref(s),
        _p(tr, C.c_int32) if trace else None,
        default_threads() if nthreads is None else nthreads)
    if rc != 0:
        raise ValueError(f"som_oracle_train: bad arguments (rc={rc})")
    return W, tr


def train_near_tie(W: np.ndarray, rows: int, cols: int, X: np.ndarray,
                   order: np.ndarray, s: Schedule, tie_rel: float, seed: int,
                   step0: int = 0, total_steps: Optional[int] = None,
                   topology: int = RECT, nthreads: Optional[int] = None):
    """train() with every near tie (D2 - D1 <= tie_rel * D1) decided by a
    seeded coin; returns (W, number of steps that took the second unit)."""
    W = np.array(W, dtype=np.float64, order="C", copy=True)
    X = np.ascontiguousarray(X, dtype=np.float32)
    order = np.ascontiguousarray(order, dtype=np.int32)
    n, d = X.shape
    assert W.shape == (rows * cols, d)
    nsteps = order.shape[0]
    T = step0 + nsteps if total_steps is None else int(total_steps)
    flips = C.c_int64()
    rc = lib().som_oracle_train_near_tie(
        _p(W, C.c_double), rows, cols, topology, d, _p(X, C.c_float), n,
        _p(order, C.c_int32), nsteps, step0, T, C.byref(s), float(tie_rel),
        C.c_uint64(seed), C.byref(flips),
        default_threads() if nthreads is None else nthreads)
    if rc != 0:
        raise ValueError(f"som_oracle_train_near_tie: bad arguments (rc={rc})")
    return W, flips.value


def evaluate(W: np.ndarray, rows: int, cols: int, X: np.ndarray,
             topology: int = RECT, nthreads: Optional[int] = None) -> dict:
    """First/second BMU, squared distances, QE and TE of every sample."""
    W = np.ascontiguousarray(W, dtype=np.float64)
    X = np.ascontiguousarray(X, dtype=np.float32)
    n, d = X.shape
    c1 = np.empty(n, dtype=np.int32)
    c2 = np.empty(n, dtype=np.int32)
    d1 = np.empty(n, dtype=np.float64)
    d2 = np.empty(n, dtype=np.float64)
    qe = C.c_double()
    te = C.c_double()
    rc = lib().som_oracle_evaluate(
        _p(W, C.c_double), rows, cols, topology, d, _p(X, C.c_float), n,
        _p(c1, C.c_int32), _p(c2, C.c_int32), _p(d1, C.c_double),
        _p(d2, C.c_double), C.byref(qe), C.byref(te),
        default_threads() if nthreads is None else nthreads)
    if rc != 0:
        raise ValueError(f"som_oracle_evaluate: bad arguments (rc={rc})")
    return {"c1": c1, "c2": c2, "d1": d1, "d2": d2, "qe": qe.value,
            "te": te.value}


# ------------------------------------------------------------------ linear init
# Sec. 6D: the prototypes start as a regular two-dimensional grid in the
# hyperplane spanned by the two largest principal components of the data;
# Fig. 2 derives the map size and the iteration count from the data size and
# those components.  Plain numpy in fp64; the eigen-decomposition is numpy's.

def pca_top2(X: np.ndarray):
    """Fig. 2 steps 3-4: the two largest eigenvalues lambda1 >= lambda2 of the
    covariance (1/m) sum_i (x_i - mu)(x_i - mu)^T of the m rows of X, their
    unit eigenvectors (columns of V; sign fixed so that the component of
    largest magnitude, lowest index on ties, is positive) and the mean mu."""
    X64 = np.asarray(X, dtype=np.float64)
    m = X64.shape[0]
    mu = X64.mean(axis=0)
    Xc = X64 - mu
    Cov = Xc.T @ Xc / m
    w, V = np.linalg.eigh(Cov)  # ascending
    lam = w[::-1][:2].copy()
    V = V[:, ::-1][:, :2].copy()
    for a in range(V.shape[1]):
        k = int(np.argmax(np.abs(V[:, a])))
        if V[k, a] < 0:
            V[:, a] = -V[:, a]
    return lam, V, mu


def suggest_size(m: int, lambda1: float, lambda2: float):
    """Fig. 2 steps 2 and 5-15: (rows, cols, iterations) for m samples whose
    two largest principal-component variances are lambda1 >= lambda2.
    munits = ceil(5 sqrt(m)); r = sqrt(lambda1 / lambda2), or 1 when
    lambda1 = 0 or lambda2 * munits < lambda1; size1 = the nearest integer to
    sqrt(munits / (r sqrt(3/4))), within [1, munits]; size2 =
    ceil(munits / size1); rows = min, cols = max; iterations =
    ceil(50 rows cols / m) * m * 4."""
    munits = int(np.ceil(5.0 * np.sqrt(m)))
    if lambda1 == 0.0 or lambda2 * munits < lambda1:
        r = 1.0
    else:
        r = float(np.sqrt(lambda1 / lambda2))
    size1 = int(np.floor(np.sqrt(munits / (r * np.sqrt(0.75))) + 0.5))
    size1 = max(1, min(munits, size1))
    size2 = -(-munits // size1)
    rows, cols = min(size1, size2), max(size1, size2)
    iters = int(np.ceil(50.0 * rows * cols / m)) * m * 4
    return rows, cols, iters


def linear_init(mu: np.ndarray, lam, V: np.ndarray, rows: int, cols: int) -> np.ndarray:
    """Sec. 6D: unit (r, c) starts at mu + a_c sqrt(lambda1) v1 +
    b_r sqrt(lambda2) v2 with a_c = 2c/(cols-1) - 1 and b_r = 2r/(rows-1) - 1
    (0 for a single column or row): the longer side of the map spans the
    first component, the grid covering one standard deviation either side."""
    W = np.empty((rows * cols, mu.size), dtype=np.float64)
    s1, s2 = np.sqrt(max(lam[0], 0.0)), np.sqrt(max(lam[1], 0.0))
    for r in range(rows):
        b = 2.0 * r / (rows - 1) - 1.0 if rows > 1 else 0.0
        for c in range(cols):
            a = 2.0 * c / (cols - 1) - 1.0 if cols > 1 else 0.0
            W[r * cols + c] = mu + a * s1 * V[:, 0] + b * s2 * V[:, 1]
    return W


# ------------------------------------------------------------------ batch map
# Sec. 4 names the batch form of the SOM as the variant most GPU SOMs
# implement ([25], [26]); the paper itself trains online (Eq. (1)).  The
# batch rule here is Kohonen's: every epoch assigns all samples to their
# BMUs under the current prototypes, then sets each prototype to the
# neighbourhood-weighted mean of the samples,
#     w_u = sum_i h(u, c_i) x_i / sum_i h(u, c_i),
# with h the Gaussian of Eq. (1) without the learning rate (a delta at the
# BMU for sigma = 0, 1 everywhere for sigma = inf); a unit whose weights all
# vanish keeps its prototype.  sigma decays over the epochs by the same law
# as the online schedule, at p = e / (E - 1).  Plain numpy in fp64 on the
# explicit N x N neighbourhood matrix.

def batch_sigma(e: int, epochs: int, sigma0: float, sigma1: float,
                sigma_decay: int = EXPONENTIAL) -> float:
    """The radius of epoch e of a batch run of `epochs` epochs."""
    s = schedule(1.0, 1.0, sigma0, sigma1, LINEAR, sigma_decay)
    return schedule_at(e, epochs, s)[1]


def batch_update(W: np.ndarray, rows: int, cols: int, X: np.ndarray, c: np.ndarray,
                 sigma: float, topology: int = RECT) -> np.ndarray:
    """One batch-map update given every sample's BMU c (a float64 copy of W
    is returned): unit u becomes sum_k h(u, k) S_k / sum_k h(u, k) n_k, with
    S_k and n_k the sum and count of the samples whose BMU is k; a unit whose
    denominator is 0 keeps its prototype."""
    W = np.array(W, dtype=np.float64, order="C", copy=True)
    X = np.ascontiguousarray(X, dtype=np.float32)
    c = np.asarray(c, dtype=np.int64)
    N = rows * cols
    H = np.stack([neighbourhood(rows, cols, topology, k, 1.0, sigma)
                  for k in range(N)], axis=1)          # H[u, k] = h(u, k)
    S = np.zeros((N, X.shape[1]), dtype=np.float64)
    np.add.at(S, c, X.astype(np.float64))
    cnt = np.bincount(c, minlength=N).astype(np.float64)
    num = H @ S
    den = H @ cnt
    keep = den > 0
    W[keep] = num[keep] / den[keep, None]
    return W


def train_batch(W: np.ndarray, rows: int, cols: int, X: np.ndarray, epochs: int,
                sigma0: float, sigma1: float, sigma_decay: int = EXPONENTIAL,
                topology: int = RECT, nthreads: Optional[int] = None, trace: bool = False):
    """`epochs` batch epochs from W (float64 copy); returns (W, BMUs per epoch)."""
    W = np.array(W, dtype=np.float64, order="C", copy=True)
    X = np.ascontiguousarray(X, dtype=np.float32)
    bmus = []
    for e in range(epochs):
        sigma = batch_sigma(e, epochs, sigma0, sigma1, sigma_decay)
        c = evaluate(W, rows, cols, X, topology=topology, nthreads=nthreads)["c1"]
        if trace:
            bmus.append(c)
        W = batch_update(W, rows, cols, X, c, sigma, topology)
    return W, bmus
