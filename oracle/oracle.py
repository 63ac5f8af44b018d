"""ctypes wrapper of the CPU oracle (pnn_oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, the package smoke check and the benchmark's
CPU-baseline leg may import this module; the GPU library and its Python binding never do.
The oracle is built with gcc (no fast-math, no contraction of multiply-adds) into
``oracle/_build/liboracle.so`` on first use.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pnn_oracle.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD, "liboracle.so")
_lock = threading.Lock()
_lib = None

SIGMOID, TANH, RELU, LEAKY_RELU, SOFTMAX = 0, 1, 2, 3, 4
LOSS_MSE, LOSS_XENT = 0, 1
EXACT, BF16 = 0, 1


class OrConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32),
        ("sizes", ctypes.c_int32 * 9),
        ("act", ctypes.c_int32 * 8),
        ("loss", ctypes.c_int32),
        ("precision", ctypes.c_int32),
        ("replicas", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("lr", ctypes.c_float),
    ]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc; returns the path of the shared library."""
    os.makedirs(_BUILD, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                               "-fno-fast-math", "-Wall", "-o", tmp, _SRC, "-lm", "-lpthread"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    with _lock:
        if _lib is None:
            L = ctypes.CDLL(build())
            P = ctypes.POINTER
            d, f, i32, i64 = ctypes.c_double, ctypes.c_float, ctypes.c_int32, ctypes.c_int64
            cfg = P(OrConfig)
            L.or_param_count.argtypes = [cfg]
            L.or_param_count.restype = i64
            L.or_shard.argtypes = [i64, i32, i32, P(i64), P(i64)]
            L.or_round_bf16.argtypes = [d]
            L.or_round_bf16.restype = d
            L.or_train_epoch.argtypes = [cfg, P(d), P(f), P(i32), i64, i32]
            L.or_train_replicas.argtypes = [cfg, P(d), P(i32), i32, P(f), P(i32), i64]
            L.or_merge.argtypes = [cfg, P(d), P(d)]
            L.or_merge_weighted.argtypes = [cfg, P(d), P(d), P(d)]
            L.or_forward.argtypes = [cfg, P(d), P(f), i64, P(d)]
            L.or_predict.argtypes = [cfg, P(d), P(f), i64, P(i32), P(i32)]
            L.or_predict.restype = i64
            L.or_cost.argtypes = [cfg, P(d), P(f), P(i32), i64]
            L.or_cost.restype = d
            L.or_gradient.argtypes = [cfg, P(d), P(f), P(i32), i64, P(d)]
            L.or_trace.argtypes = [cfg, P(d), P(f), i32, P(d), P(d), P(d)]
            _lib = L
        return _lib


def _ptr(a: Optional[np.ndarray], ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class Oracle:
    """Plain fp64 reference of the PNN method for one configuration."""

    def __init__(self, sizes: Sequence[int], acts: Sequence[int], loss: int, precision: int = EXACT,
                 replicas: int = 1, batch: int = 1, lr: float = 0.1):
        c = OrConfig()
        c.n_layers = len(sizes) - 1
        for i, s in enumerate(sizes):
            c.sizes[i] = int(s)
        for i, a in enumerate(acts):
            c.act[i] = int(a)
        c.loss, c.precision, c.replicas, c.batch = int(loss), int(precision), int(replicas), int(batch)
        c.lr = float(lr)
        self.c = c
        self.sizes = tuple(int(s) for s in sizes)
        self.P = int(lib().or_param_count(ctypes.byref(c)))

    @classmethod
    def from_workload(cls, w, **over):
        kw = dict(sizes=w.sizes, acts=w.acts, loss=w.loss, precision=w.precision, replicas=w.replicas,
                  batch=w.batch, lr=w.lr)
        kw.update(over)
        return cls(**kw)

    # layout helpers ------------------------------------------------------------------
    def split(self, theta: np.ndarray):
        """[(W1, b1), (W2, b2), ...] views of one flat parameter vector."""
        out, o = [], 0
        for l in range(len(self.sizes) - 1):
            n_in, n_out = self.sizes[l], self.sizes[l + 1]
            W = theta[o:o + n_out * n_in].reshape(n_out, n_in)
            o += n_out * n_in
            b = theta[o:o + n_out]
            o += n_out
            out.append((W, b))
        return out

    def shard(self, n: int, k: int):
        s, ln = ctypes.c_int64(), ctypes.c_int64()
        lib().or_shard(n, self.c.replicas, k, ctypes.byref(s), ctypes.byref(ln))
        return s.value, ln.value

    # method ---------------------------------------------------------------------------
    def replicate(self, theta0: np.ndarray) -> np.ndarray:
        """K copies of theta0 as a [K, P] float64 array."""
        return np.tile(np.asarray(theta0, dtype=np.float64)[None, :], (self.c.replicas, 1))

    def train_epoch(self, theta: np.ndarray, X: np.ndarray, y: np.ndarray, threads: int = 1) -> None:
        """One epoch of every child network on its slice, in place on theta [K, P] float64."""
        assert theta.dtype == np.float64 and theta.shape == (self.c.replicas, self.P) and theta.flags.c_contiguous
        X = np.ascontiguousarray(X, dtype=np.float32)
        y = np.ascontiguousarray(y, dtype=np.int32)
        assert X.shape == (y.shape[0], self.sizes[0])
        lib().or_train_epoch(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(X, ctypes.c_float),
                             _ptr(y, ctypes.c_int32), X.shape[0], int(threads))

    def train_replicas(self, theta_sub: np.ndarray, ids: Sequence[int], X: np.ndarray, y: np.ndarray) -> None:
        """One epoch of the listed child networks only (theta_sub [len(ids), P], in place)."""
        ids_a = np.ascontiguousarray(ids, dtype=np.int32)
        assert theta_sub.dtype == np.float64 and theta_sub.shape == (len(ids_a), self.P)
        X = np.ascontiguousarray(X, dtype=np.float32)
        y = np.ascontiguousarray(y, dtype=np.int32)
        lib().or_train_replicas(ctypes.byref(self.c), _ptr(theta_sub, ctypes.c_double),
                                _ptr(ids_a, ctypes.c_int32), len(ids_a), _ptr(X, ctypes.c_float),
                                _ptr(y, ctypes.c_int32), X.shape[0])

    def merge(self, theta: np.ndarray) -> np.ndarray:
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        assert theta.shape == (self.c.replicas, self.P)
        out = np.empty(self.P, dtype=np.float64)
        lib().or_merge(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(out, ctypes.c_double))
        return out

    def merge_weighted(self, theta: np.ndarray, w: Sequence[float]) -> np.ndarray:
        """sum_k w_k theta_k / sum_k w_k over the K CNs (weights >= 0, positive sum)."""
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        wv = np.ascontiguousarray(w, dtype=np.float64)
        assert theta.shape == (self.c.replicas, self.P) and wv.shape == (self.c.replicas,)
        assert np.all(wv >= 0) and wv.sum() > 0
        out = np.empty(self.P, dtype=np.float64)
        lib().or_merge_weighted(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(wv, ctypes.c_double),
                                _ptr(out, ctypes.c_double))
        return out

    def forward(self, theta: np.ndarray, X: np.ndarray) -> np.ndarray:
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        X = np.ascontiguousarray(X, dtype=np.float32)
        out = np.empty((X.shape[0], self.sizes[-1]), dtype=np.float64)
        lib().or_forward(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(X, ctypes.c_float),
                         X.shape[0], _ptr(out, ctypes.c_double))
        return out

    def predict(self, theta: np.ndarray, X: np.ndarray, y: Optional[np.ndarray] = None):
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        X = np.ascontiguousarray(X, dtype=np.float32)
        pred = np.empty(X.shape[0], dtype=np.int32)
        yy = None if y is None else np.ascontiguousarray(y, dtype=np.int32)
        correct = lib().or_predict(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(X, ctypes.c_float),
                                   X.shape[0], _ptr(yy, ctypes.c_int32), _ptr(pred, ctypes.c_int32))
        return pred, int(correct)

    def cost(self, theta: np.ndarray, X: np.ndarray, y: np.ndarray) -> float:
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        X = np.ascontiguousarray(X, dtype=np.float32)
        y = np.ascontiguousarray(y, dtype=np.int32)
        return float(lib().or_cost(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(X, ctypes.c_float),
                                   _ptr(y, ctypes.c_int32), X.shape[0]))

    def gradient(self, theta: np.ndarray, X: np.ndarray, y: np.ndarray) -> np.ndarray:
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        X = np.ascontiguousarray(X, dtype=np.float32)
        y = np.ascontiguousarray(y, dtype=np.int32)
        g = np.empty(self.P, dtype=np.float64)
        lib().or_gradient(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(X, ctypes.c_float),
                          _ptr(y, ctypes.c_int32), X.shape[0], _ptr(g, ctypes.c_double))
        return g

    def trace(self, theta: np.ndarray, x: np.ndarray, label: int):
        """Per-layer (z, x, delta) lists of one sample."""
        theta = np.ascontiguousarray(theta, dtype=np.float64)
        x = np.ascontiguousarray(x, dtype=np.float32)
        n = sum(self.sizes[1:])
        z, a, d = (np.empty(n, dtype=np.float64) for _ in range(3))
        lib().or_trace(ctypes.byref(self.c), _ptr(theta, ctypes.c_double), _ptr(x, ctypes.c_float), int(label),
                       _ptr(z, ctypes.c_double), _ptr(a, ctypes.c_double), _ptr(d, ctypes.c_double))
        out, o = [], 0
        for w in self.sizes[1:]:
            out.append((z[o:o + w], a[o:o + w], d[o:o + w]))
            o += w
        return out


def round_bf16(v: float) -> float:
    return float(lib().or_round_bf16(float(v)))
