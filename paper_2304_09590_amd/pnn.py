"""Python binding of libpnn.so (the C ABI declared in include/pnn.h).

Argument marshalling only: every step of training, merging and inference runs in the
library's HIP kernels.  Device tensors come from PyTorch (memory and streams only).  There
is no fallback: if the compiled library is missing, importing the binding raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpnn.so")

PNN_OK, PNN_EINVAL, PNN_ESHAPE, PNN_ENOMEM, PNN_EHIP, PNN_ESTATE = 0, -1, -2, -3, -4, -5
SIGMOID, TANH, RELU, LEAKY_RELU, SOFTMAX = 0, 1, 2, 3, 4
LOSS_MSE, LOSS_XENT = 0, 1
FP32, BF16_MIXED = 0, 1

STATUS_NAMES = {0: "PNN_OK", -1: "PNN_EINVAL", -2: "PNN_ESHAPE", -3: "PNN_ENOMEM", -4: "PNN_EHIP", -5: "PNN_ESTATE"}


class PnnConfig(ctypes.Structure):
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


class PnnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Load libpnn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2304_09590_amd/build.py "
                              "(there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        cfg = P(PnnConfig)
        L.pnn_config_check.argtypes = [cfg]
        L.pnn_config_check.restype = i32
        L.pnn_param_count.argtypes = [cfg]
        L.pnn_param_count.restype = i64
        L.pnn_shard.argtypes = [i64, i32, i32, P(i64), P(i64)]
        L.pnn_shard.restype = i32
        L.pnn_init.argtypes = [cfg, P(ctypes.c_float), vp, P(vp)]
        L.pnn_init.restype = i32
        L.pnn_train_epoch.argtypes = [vp, vp, vp, i64, vp]
        L.pnn_train_epoch.restype = i32
        L.pnn_merge.argtypes = [vp, i32, vp]
        L.pnn_merge.restype = i32
        L.pnn_infer.argtypes = [vp, i32, vp, i64, vp, vp, P(i64), vp, vp]
        L.pnn_infer.restype = i32
        L.pnn_eval.argtypes = [vp, i32, vp, vp, i64, P(i64), P(ctypes.c_double), vp]
        L.pnn_eval_noalloc.argtypes = [vp, i32, vp, vp, i64, P(i64), P(ctypes.c_double), vp]
        L.pnn_eval_noalloc.restype = i32
        L.pnn_merge_weighted.argtypes = [vp, P(ctypes.c_double), i32, vp]
        L.pnn_train_epoch_order.argtypes = [vp, vp, vp, i64, vp, vp]
        L.pnn_train_epoch_order.restype = i32
        L.pnn_merge_weighted.restype = i32
        L.pnn_eval.restype = i32
        L.pnn_get_params.argtypes = [vp, i32, P(ctypes.c_float)]
        L.pnn_get_params.restype = i32
        L.pnn_set_params.argtypes = [vp, i32, P(ctypes.c_float)]
        L.pnn_set_params.restype = i32
        L.pnn_last_error.argtypes = [vp]
        L.pnn_last_error.restype = ctypes.c_char_p
        L.pnn_plan.argtypes = [vp]
        L.pnn_plan.restype = ctypes.c_char_p
        L.pnn_profile.argtypes = [vp, i32]
        L.pnn_profile.restype = i32
        L.pnn_profile_read.argtypes = [vp, P(ctypes.c_char_p), P(ctypes.c_double), P(i64), i32]
        L.pnn_profile_read.restype = i32
        L.pnn_destroy.argtypes = [vp]
        L.pnn_destroy.restype = None
        _lib = L
    return _lib


def make_config(sizes: Sequence[int], acts: Sequence[int], loss: int, precision: int = FP32, replicas: int = 1,
                batch: int = 1, lr: float = 0.1) -> PnnConfig:
    c = PnnConfig()
    c.n_layers = len(sizes) - 1
    for i, s in enumerate(sizes):
        c.sizes[i] = int(s)
    for i, a in enumerate(acts):
        c.act[i] = int(a)
    c.loss, c.precision, c.replicas, c.batch = int(loss), int(precision), int(replicas), int(batch)
    c.lr = float(lr)
    return c


def config_from_workload(w, **over) -> PnnConfig:
    kw = dict(sizes=w.sizes, acts=w.acts, loss=w.loss, precision=w.precision, replicas=w.replicas, batch=w.batch,
              lr=w.lr)
    kw.update(over)
    return make_config(**kw)


def param_count(cfg: PnnConfig) -> int:
    return int(lib().pnn_param_count(ctypes.byref(cfg)))


def config_check(cfg: PnnConfig) -> int:
    return int(lib().pnn_config_check(ctypes.byref(cfg)))


def shard(n: int, k_total: int, k: int) -> Tuple[int, int]:
    s, ln = ctypes.c_int64(), ctypes.c_int64()
    st = lib().pnn_shard(n, k_total, k, ctypes.byref(s), ctypes.byref(ln))
    if st != PNN_OK:
        raise PnnError(st, "pnn_shard")
    return s.value, ln.value


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _dev_ptr(t, dtype_name: str):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous() or str(t.dtype) != dtype_name:
        raise ValueError(f"expected a contiguous CUDA tensor of {dtype_name}, got {t.dtype} on {t.device}")
    return t.data_ptr()


class PNN:
    """One handle of the library: K child networks plus the merged network."""

    def __init__(self, cfg: PnnConfig, theta0: np.ndarray, stream=None):
        self._lib = lib()
        self.cfg = cfg
        self.P = param_count(cfg)
        self.K = int(cfg.replicas)
        if self.P == 0:
            raise PnnError(PNN_EINVAL, "invalid configuration")
        th = np.ascontiguousarray(theta0, dtype=np.float32)
        if th.size != self.P:
            raise ValueError(f"theta0 has {th.size} values, the configuration needs {self.P}")
        h = ctypes.c_void_p()
        st = self._lib.pnn_init(ctypes.byref(cfg), th.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                _stream_handle(stream), ctypes.byref(h))
        if st != PNN_OK:
            raise PnnError(st, self._lib.pnn_last_error(None).decode())
        self.h = h

    def _check(self, st: int, what: str):
        if st != PNN_OK:
            raise PnnError(st, f"{what}: {self._lib.pnn_last_error(self.h).decode()}")

    def train_epoch(self, x, y, stream=None) -> None:
        self._check(self._lib.pnn_train_epoch(self.h, _dev_ptr(x, "torch.float32"), _dev_ptr(y, "torch.int32"),
                                              x.shape[0], _stream_handle(stream)), "pnn_train_epoch")

    def train_epoch_order(self, x, y, order, stream=None) -> None:
        """One epoch over x[order], y[order] (order: int32 device tensor of N row indices)."""
        self._check(self._lib.pnn_train_epoch_order(self.h, _dev_ptr(x, "torch.float32"), _dev_ptr(y, "torch.int32"),
                                                    x.shape[0], _dev_ptr(order, "torch.int32"),
                                                    _stream_handle(stream)), "pnn_train_epoch_order")

    def merge(self, broadcast: bool = False, stream=None) -> None:
        self._check(self._lib.pnn_merge(self.h, 1 if broadcast else 0, _stream_handle(stream)), "pnn_merge")

    def infer(self, x, pred, which: int = -1, out=None, y=None, count: bool = False, stream=None) -> Optional[int]:
        c = ctypes.c_int64(-1)
        self._check(self._lib.pnn_infer(self.h, which, _dev_ptr(x, "torch.float32"), x.shape[0],
                                        _dev_ptr(pred, "torch.int32"), _dev_ptr(out, "torch.float32"),
                                        ctypes.byref(c) if count else None, _dev_ptr(y, "torch.int32"),
                                        _stream_handle(stream)), "pnn_infer")
        return c.value if count else None

    def merge_weighted(self, weights, broadcast: bool = False, stream=None) -> None:
        w = np.ascontiguousarray(weights, dtype=np.float64)
        if w.shape != (self.K,):
            raise ValueError(f"expected {self.K} weights, got shape {w.shape}")
        self._check(self._lib.pnn_merge_weighted(self.h, w.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                                 1 if broadcast else 0, _stream_handle(stream)), "pnn_merge_weighted")

    def evaluate(self, x, y, which: int = -1, stream=None):
        """(correct count, mean cost) of one network on labelled rows (pnn_eval)."""
        c = ctypes.c_int64(-1)
        cost = ctypes.c_double(float("nan"))
        self._check(self._lib.pnn_eval(self.h, which, _dev_ptr(x, "torch.float32"), _dev_ptr(y, "torch.int32"),
                                       x.shape[0], ctypes.byref(c), ctypes.byref(cost), _stream_handle(stream)),
                    "pnn_eval")
        return c.value, cost.value

    def evaluate_noalloc(self, x, y, which: int = -1, stream=None):
        """(correct count, mean cost) as evaluate, on the library's fixed workspace
        (pnn_eval_noalloc: no device allocation)."""
        c = ctypes.c_int64(-1)
        cost = ctypes.c_double(float("nan"))
        self._check(self._lib.pnn_eval_noalloc(self.h, which, _dev_ptr(x, "torch.float32"),
                                               _dev_ptr(y, "torch.int32"), x.shape[0], ctypes.byref(c),
                                               ctypes.byref(cost), _stream_handle(stream)), "pnn_eval_noalloc")
        return c.value, cost.value

    def get_params(self, which: int = -1) -> np.ndarray:
        out = np.empty(self.P, dtype=np.float32)
        self._check(self._lib.pnn_get_params(self.h, which, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float))),
                    "pnn_get_params")
        return out

    def set_params(self, which: int, theta: np.ndarray) -> None:
        th = np.ascontiguousarray(theta, dtype=np.float32)
        assert th.size == self.P
        self._check(self._lib.pnn_set_params(self.h, which, th.ctypes.data_as(ctypes.POINTER(ctypes.c_float))),
                    "pnn_set_params")

    def profile(self, enable: bool) -> None:
        self._check(self._lib.pnn_profile(self.h, 1 if enable else 0), "pnn_profile")

    def profile_read(self) -> dict:
        cap = 64
        names = (ctypes.c_char_p * cap)()
        ms = (ctypes.c_double * cap)()
        cnt = (ctypes.c_int64 * cap)()
        n = self._lib.pnn_profile_read(self.h, names, ms, cnt, cap)
        return {names[i].decode(): (ms[i], cnt[i]) for i in range(min(n, cap))}

    @property
    def plan(self) -> str:
        """Training plan chosen at init (see pnn_plan in include/pnn.h)."""
        return self._lib.pnn_plan(self.h).decode()

    def close(self) -> None:
        if getattr(self, "h", None):
            self._lib.pnn_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
