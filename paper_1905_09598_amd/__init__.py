"""MI355X-native online self-organizing map (SOM) training.

Thin ctypes binding of ``libsom.so`` (C ABI in ``include/som.h``).  Every
step of training and evaluation runs in the library's HIP kernels; this
module only marshals arguments.  PyTorch supplies device memory and the
stream: tensors passed in must be contiguous CUDA (HIP) tensors of the
stated dtype, and calls are ordered on torch's current stream.

The library is loaded on first use.  If it has not been built
(``python -m paper_1905_09598_amd.build``) every call raises
``LibraryMissing``: there is no CPU fallback.

Functions carry the C names (``som_create``, ``som_train``, ``som_bmu``,
``som_bmu2``, ``som_quantization_error``, ``som_topographic_error``,
``som_get_weights``, ``som_set_weights``, ...); ``Map`` wraps them.
"""
from __future__ import annotations

import ctypes as C
import math
import os
from typing import Optional

__all__ = [
    "SomError", "LibraryMissing", "Schedule", "Map", "lib", "library_path",
    "som_create", "som_destroy", "som_set_topology", "som_set_stream",
    "som_train", "som_train_csr", "som_train_batch", "som_bmu", "som_bmu2",
    "som_quantization_error", "som_topographic_error", "som_get_weights", "som_set_weights",
    "som_synchronize", "som_get_shape", "som_shuffle", "som_train_plan",
    "som_pca2", "som_suggest_size", "som_init_linear", "som_evaluate", "som_stream_inplace",
    "som_bmu2_noalloc", "som_status_string", "RECT", "HEX", "LINEAR", "EXPONENTIAL", "EXPORTED",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsom.so")

RECT, HEX = 0, 1
LINEAR, EXPONENTIAL = 0, 1

STATUS = {0: "SOM_OK", 1: "SOM_E_ARG", 2: "SOM_E_OOM", 3: "SOM_E_DEVICE",
          4: "SOM_E_LAUNCH", 5: "SOM_E_TIMEOUT", 6: "SOM_E_UNSUPPORTED",
          7: "SOM_E_BAD_ORDER", 8: "SOM_E_NONFINITE"}

# Every symbol include/som.h declares.
EXPORTED = (
    "som_create", "som_destroy", "som_set_topology", "som_set_stream",
    "som_train", "som_train_csr", "som_train_batch", "som_bmu", "som_bmu2", "som_quantization_error",
    "som_topographic_error", "som_get_weights", "som_set_weights",
    "som_synchronize", "som_get_shape", "som_shuffle", "som_train_plan",
    "som_pca2", "som_suggest_size", "som_init_linear", "som_evaluate", "som_stream_inplace",
    "som_bmu2_noalloc", "som_status_string",
)


class LibraryMissing(RuntimeError):
    pass


class SomError(RuntimeError):
    def __init__(self, code: int, call: str):
        self.code = code
        self.name = STATUS.get(code, f"status {code}")
        super().__init__(f"{call}: {self.name} ({_status_text(code)})")


class Schedule(C.Structure):
    """``som_schedule`` of include/som.h."""

    _fields_ = [("lr0", C.c_double), ("lr1", C.c_double), ("lr_decay", C.c_int32),
                ("sigma0", C.c_double), ("sigma1", C.c_double),
                ("sigma_decay", C.c_int32), ("shuffle_seed", C.c_uint64),
                ("order", C.c_void_p), ("step0", C.c_int64),
                ("total_steps", C.c_int64), ("bmu_trace", C.c_void_p)]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def lib():
    """The loaded libsom (raises LibraryMissing if it was never built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise LibraryMissing(
            f"{_LIB_PATH} is missing: build it with `python -m paper_1905_09598_amd.build`")
    L = C.CDLL(_LIB_PATH)
    vp, i32, i64, u64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64
    pp = C.POINTER(C.c_void_p)
    sig = {
        "som_create": [i32, i32, i32, u64, pp],
        "som_destroy": [vp],
        "som_set_topology": [vp, i32],
        "som_set_stream": [vp, vp],
        "som_train": [vp, vp, i64, i32, C.POINTER(Schedule)],
        "som_train_csr": [vp, vp, vp, vp, i64, i32, C.POINTER(Schedule)],
        "som_train_batch": [vp, vp, i64, i32, C.c_double, C.c_double, i32],
        "som_bmu": [vp, vp, i64, vp],
        "som_bmu2": [vp, vp, i64, vp, vp, vp],
        "som_bmu2_noalloc": [vp, vp, i64, vp, vp, vp],
        "som_quantization_error": [vp, vp, i64, C.POINTER(C.c_double)],
        "som_topographic_error": [vp, vp, i64, C.POINTER(C.c_double)],
        "som_get_weights": [vp, vp],
        "som_set_weights": [vp, vp],
        "som_synchronize": [vp],
        "som_get_shape": [vp, C.POINTER(i32), C.POINTER(i32), C.POINTER(i32),
                          C.POINTER(i32)],
        "som_shuffle": [u64, i64, i64, vp],
        "som_train_plan": [vp, C.POINTER(i32), C.POINTER(i32), C.POINTER(i32), C.POINTER(i32)],
        "som_pca2": [vp, i64, i32, vp, C.POINTER(C.c_double), vp, vp, vp],
        "som_suggest_size": [i64, C.c_double, C.c_double, C.POINTER(i32), C.POINTER(i32),
                             C.POINTER(i64)],
        "som_init_linear": [vp, vp, i64],
        "som_evaluate": [vp, vp, i64, vp, C.POINTER(C.c_double), C.POINTER(C.c_double)],
        "som_stream_inplace": [vp, i64, i32, i32, vp],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = C.c_int
    L.som_status_string.argtypes = [C.c_int]
    L.som_status_string.restype = C.c_char_p
    _lib = L
    return L


def _status_text(code: int) -> str:
    try:
        return lib().som_status_string(code).decode()
    except LibraryMissing:
        return STATUS.get(code, "?")


def _check(code: int, call: str) -> None:
    if code != 0:
        raise SomError(code, call)


def _ptr(t) -> Optional[int]:
    """Device address of a torch tensor (None passes NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _require(t, dtype_name: str, what: str):
    import torch
    want = getattr(torch, dtype_name)
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch tensor")
    if t.dtype != want:
        raise TypeError(f"{what} must be {dtype_name}, got {t.dtype}")
    if not t.is_cuda:
        raise TypeError(f"{what} must live on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")


def _current_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


# ---------------------------------------------------------------- C names
def som_create(rows: int, cols: int, d: int, seed: int = 0) -> int:
    h = C.c_void_p()
    _check(lib().som_create(rows, cols, d, C.c_uint64(seed), C.byref(h)), "som_create")
    return h.value


def som_destroy(handle: int) -> None:
    _check(lib().som_destroy(handle), "som_destroy")


def som_set_topology(handle: int, topology: int) -> None:
    _check(lib().som_set_topology(handle, topology), "som_set_topology")


def som_set_stream(handle: int, stream: Optional[int]) -> None:
    _check(lib().som_set_stream(handle, stream), "som_set_stream")


def som_train(handle: int, X, n: int, epochs: int, sched: Schedule) -> None:
    _check(lib().som_train(handle, _ptr(X), n, epochs, C.byref(sched)), "som_train")


def som_train_csr(handle: int, indptr, indices, values, n: int, epochs: int,
                  sched: Schedule) -> None:
    _check(lib().som_train_csr(handle, _ptr(indptr), _ptr(indices), _ptr(values), n, epochs,
                               C.byref(sched)), "som_train_csr")


def som_train_batch(handle: int, X, n: int, epochs: int, sigma0: float, sigma1: float,
                    sigma_decay: int = EXPONENTIAL) -> None:
    _check(lib().som_train_batch(handle, _ptr(X), n, epochs, float(sigma0), float(sigma1),
                                 int(sigma_decay)), "som_train_batch")


def som_bmu(handle: int, X, n: int, out_idx) -> None:
    _check(lib().som_bmu(handle, _ptr(X), n, _ptr(out_idx)), "som_bmu")


def som_bmu2(handle: int, X, n: int, out_idx, out_idx2=None, out_d1=None) -> None:
    _check(lib().som_bmu2(handle, _ptr(X), n, _ptr(out_idx), _ptr(out_idx2),
                          _ptr(out_d1)), "som_bmu2")


def som_bmu2_noalloc(handle: int, X, n: int, out_idx, out_idx2=None, out_d1=None) -> None:
    _check(lib().som_bmu2_noalloc(handle, _ptr(X), n, _ptr(out_idx), _ptr(out_idx2),
                                  _ptr(out_d1)), "som_bmu2_noalloc")


def som_quantization_error(handle: int, X, n: int) -> float:
    v = C.c_double()
    _check(lib().som_quantization_error(handle, _ptr(X), n, C.byref(v)),
           "som_quantization_error")
    return v.value


def som_topographic_error(handle: int, X, n: int) -> float:
    v = C.c_double()
    _check(lib().som_topographic_error(handle, _ptr(X), n, C.byref(v)),
           "som_topographic_error")
    return v.value


def som_get_weights(handle: int, dst) -> None:
    _check(lib().som_get_weights(handle, _ptr(dst)), "som_get_weights")


def som_set_weights(handle: int, src) -> None:
    _check(lib().som_set_weights(handle, _ptr(src)), "som_set_weights")


def som_synchronize(handle: int) -> None:
    _check(lib().som_synchronize(handle), "som_synchronize")


def som_get_shape(handle: int):
    r, c, d, t = C.c_int32(), C.c_int32(), C.c_int32(), C.c_int32()
    _check(lib().som_get_shape(handle, C.byref(r), C.byref(c), C.byref(d), C.byref(t)),
           "som_get_shape")
    return r.value, c.value, d.value, t.value


def som_shuffle(seed: int, epoch: int, n: int):
    import numpy as np
    out = np.empty(n, dtype=np.int32)
    _check(lib().som_shuffle(C.c_uint64(seed), epoch, n, out.ctypes.data), "som_shuffle")
    return out


def som_train_plan(handle: int):
    g, b, v, m = C.c_int32(), C.c_int32(), C.c_int32(), C.c_int32()
    _check(lib().som_train_plan(handle, C.byref(g), C.byref(b), C.byref(v), C.byref(m)),
           "som_train_plan")
    return {"grid": g.value, "block": b.value, "variant": v.value, "block_steps": m.value}


def som_pca2(X, n: int, d: int, stream=None, mean=None, v1=None, v2=None):
    """Two largest covariance eigenvalues of X (host floats); the means and
    unit eigenvectors go to the optional device arrays."""
    lam = (C.c_double * 2)()
    _check(lib().som_pca2(_ptr(X), n, d, stream, lam, _ptr(mean), _ptr(v1), _ptr(v2)),
           "som_pca2")
    return lam[0], lam[1]


def som_suggest_size(m: int, lambda1: float, lambda2: float):
    r, c, t = C.c_int32(), C.c_int32(), C.c_int64()
    _check(lib().som_suggest_size(m, lambda1, lambda2, C.byref(r), C.byref(c), C.byref(t)),
           "som_suggest_size")
    return r.value, c.value, t.value


def som_init_linear(handle: int, X, n: int) -> None:
    _check(lib().som_init_linear(handle, _ptr(X), n), "som_init_linear")


def som_evaluate(handle: int, X, n: int, out_idx=None):
    """(QE, TE) of the n rows of X from one BMU search; the BMUs go to
    out_idx when given."""
    qe, te = C.c_double(), C.c_double()
    _check(lib().som_evaluate(handle, _ptr(X), n, _ptr(out_idx), C.byref(qe), C.byref(te)),
           "som_evaluate")
    return qe.value, te.value


def som_stream_inplace(buf, nbytes: int, passes: int, grid: int, stream=None) -> None:
    _check(lib().som_stream_inplace(_ptr(buf), int(nbytes), int(passes), int(grid), stream),
           "som_stream_inplace")


def som_status_string(code: int) -> str:
    return lib().som_status_string(code).decode()


def pca2(X):
    """(lambda1, lambda2, mean, v1, v2) of the rows of the device matrix X."""
    import torch
    _require(X, "float32", "X")
    n, d = X.shape
    mean, v1, v2 = (torch.empty(d, dtype=torch.float32, device=X.device) for _ in range(3))
    l1, l2 = som_pca2(X, n, d, _current_stream(), mean, v1, v2)
    return l1, l2, mean, v1, v2


# ---------------------------------------------------------------- wrapper
def make_schedule(lr0: float, lr1: float, sigma0: float, sigma1: float,
                  lr_decay: int = LINEAR, sigma_decay: int = EXPONENTIAL,
                  shuffle_seed: int = 0, order=None, step0: int = 0,
                  total_steps: int = 0, bmu_trace=None) -> Schedule:
    return Schedule(float(lr0), float(lr1), int(lr_decay), float(sigma0),
                    float(sigma1), int(sigma_decay), int(shuffle_seed),
                    _ptr(order), int(step0), int(total_steps), _ptr(bmu_trace))


class Map:
    """A rows x cols map of d-dimensional fp32 prototypes on the GPU."""

    def __init__(self, rows: int, cols: int, d: int, seed: int = 0,
                 topology: int = RECT):
        import torch
        self.rows, self.cols, self.d = int(rows), int(cols), int(d)
        self.handle = som_create(self.rows, self.cols, self.d, seed)
        if topology != RECT:
            som_set_topology(self.handle, topology)
        self.topology = topology
        self._torch = torch

    @property
    def units(self) -> int:
        return self.rows * self.cols

    def _bind_stream(self):
        som_set_stream(self.handle, _current_stream())

    def close(self):
        if getattr(self, "handle", None):
            som_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - best effort
        try:
            self.close()
        except Exception:
            pass

    def train(self, X, epochs: int, lr0: float, lr1: float, sigma0: float,
              sigma1: float, lr_decay: int = LINEAR,
              sigma_decay: int = EXPONENTIAL, order=None, shuffle_seed: int = 0,
              step0: int = 0, total_steps: int = 0, bmu_trace=None) -> None:
        self._check_x(X)
        if order is not None:
            _require(order, "int32", "order")
        if bmu_trace is not None:
            _require(bmu_trace, "int32", "bmu_trace")
        s = make_schedule(lr0, lr1, sigma0, sigma1, lr_decay, sigma_decay,
                          shuffle_seed, order, step0, total_steps, bmu_trace)
        self._bind_stream()
        som_train(self.handle, X, X.shape[0], int(epochs), s)

    def train_csr(self, indptr, indices, values, epochs: int, lr0: float, lr1: float,
                  sigma0: float, sigma1: float, lr_decay: int = LINEAR,
                  sigma_decay: int = EXPONENTIAL, order=None, shuffle_seed: int = 0,
                  step0: int = 0, total_steps: int = 0, bmu_trace=None) -> None:
        """Train from the n rows of a CSR matrix (int64 indptr of n + 1
        offsets, int32 column indices sorted within each row, fp32 values,
        all on the GPU)."""
        _require(indptr, "int64", "indptr")
        _require(indices, "int32", "indices")
        _require(values, "float32", "values")
        if indptr.dim() != 1 or indptr.numel() < 2:
            raise ValueError("indptr must be 1-D with n + 1 entries")
        if indices.numel() != values.numel():
            raise ValueError("indices and values must have the same length")
        if order is not None:
            _require(order, "int32", "order")
        if bmu_trace is not None:
            _require(bmu_trace, "int32", "bmu_trace")
        s = make_schedule(lr0, lr1, sigma0, sigma1, lr_decay, sigma_decay,
                          shuffle_seed, order, step0, total_steps, bmu_trace)
        self._bind_stream()
        nnz = indices.numel()
        som_train_csr(self.handle, indptr, indices if nnz else None, values if nnz else None,
                      indptr.numel() - 1, int(epochs), s)

    def train_batch(self, X, epochs: int, sigma0: float, sigma1: float,
                    sigma_decay: int = EXPONENTIAL) -> None:
        """Batch-map epochs over the rows of X (see som_train_batch)."""
        self._check_x(X)
        self._bind_stream()
        som_train_batch(self.handle, X, X.shape[0], int(epochs), sigma0, sigma1, sigma_decay)

    def bmu(self, X, second: bool = False):
        self._check_x(X)
        torch = self._torch
        n = X.shape[0]
        idx = torch.empty(n, dtype=torch.int32, device=X.device)
        self._bind_stream()
        if not second:
            som_bmu(self.handle, X, n, idx)
            return idx
        idx2 = torch.empty(n, dtype=torch.int32, device=X.device)
        d1 = torch.empty(n, dtype=torch.float32, device=X.device)
        som_bmu2(self.handle, X, n, idx, idx2, d1)
        return idx, idx2, d1

    def _check_x(self, X):
        _require(X, "float32", "X")
        if X.dim() != 2 or X.shape[1] != self.d:
            raise ValueError(f"X must be (n, {self.d})")

    def qe(self, X) -> float:
        self._check_x(X)
        self._bind_stream()
        return som_quantization_error(self.handle, X, X.shape[0])

    def te(self, X) -> float:
        self._check_x(X)
        self._bind_stream()
        return som_topographic_error(self.handle, X, X.shape[0])

    def evaluate(self, X, with_bmu: bool = True):
        """(BMUs or None, QE, TE) of the rows of X from one BMU search."""
        self._check_x(X)
        idx = None
        if with_bmu:
            idx = self._torch.empty(X.shape[0], dtype=self._torch.int32, device=X.device)
        self._bind_stream()
        qe, te = som_evaluate(self.handle, X, X.shape[0], idx)
        return idx, qe, te

    @property
    def weights(self):
        torch = self._torch
        out = torch.empty((self.units, self.d), dtype=torch.float32, device="cuda")
        self._bind_stream()
        som_get_weights(self.handle, out)
        return out

    @weights.setter
    def weights(self, W):
        torch = self._torch
        W = torch.as_tensor(W, dtype=torch.float32)
        if tuple(W.shape) != (self.units, self.d):
            raise ValueError(f"weights must be ({self.units}, {self.d})")
        W = W.contiguous()
        self._bind_stream()
        som_set_weights(self.handle, W if W.is_cuda else W.data_ptr())

    def synchronize(self):
        som_synchronize(self.handle)

    def plan(self) -> dict:
        return som_train_plan(self.handle)

    def init_linear(self, X) -> None:
        """Prototypes on the plane of X's two largest principal components."""
        self._check_x(X)
        self._bind_stream()
        som_init_linear(self.handle, X, X.shape[0])
