"""Host-side checks of the C ABI that need no GPU: the library loads, exports every entry
point declared in include/pnn.h, validates configurations before touching the device, and
its host-side split and parameter counts agree with the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import pnn_inputs as I
from oracle import oracle as O
from paper_2304_09590_amd import pnn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    with open(os.path.join(ROOT, "include", "pnn.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pnn_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    syms = declared_symbols()
    assert {"pnn_init", "pnn_train_epoch", "pnn_merge", "pnn_infer"} <= set(syms)
    L = pnn.lib()
    for s in syms:
        assert hasattr(L, s), f"{s} is declared in pnn.h but not exported"


@pytest.mark.parametrize("w", I.WORKLOADS, ids=lambda w: w.name)
def test_param_count_matches_oracle(w):
    cfg = pnn.config_from_workload(w)
    assert pnn.config_check(cfg) == pnn.PNN_OK
    assert pnn.param_count(cfg) == O.Oracle.from_workload(w).P == w.param_count()


@pytest.mark.parametrize("n,k", [(2000, 1), (60000, 4), (600000, 256), (11, 3), (5, 5)])
def test_shard_matches_oracle(n, k):
    o = O.Oracle((8, 2), (O.SIGMOID,), O.LOSS_MSE, replicas=k)
    for i in range(k):
        assert pnn.shard(n, k, i) == o.shard(n, i)


BAD = [
    dict(sizes=(784, 16, 10), acts=(pnn.SOFTMAX, pnn.SIGMOID), loss=pnn.LOSS_XENT),   # softmax not on output
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, pnn.SOFTMAX), loss=pnn.LOSS_MSE),    # softmax without xent
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, pnn.TANH), loss=pnn.LOSS_XENT),      # xent on tanh output
    dict(sizes=(784, 16, 17), acts=(pnn.SIGMOID, pnn.SIGMOID), loss=pnn.LOSS_MSE),    # output too wide
    dict(sizes=(784, 15, 10), acts=(pnn.SIGMOID, pnn.SIGMOID), loss=pnn.LOSS_MSE),    # hidden not multiple of 8
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, pnn.SIGMOID), loss=pnn.LOSS_MSE, replicas=0),
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, pnn.SIGMOID), loss=pnn.LOSS_MSE, batch=0),
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, pnn.SIGMOID), loss=pnn.LOSS_MSE, lr=float("nan")),
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, pnn.SIGMOID), loss=pnn.LOSS_MSE, precision=7),
    dict(sizes=(784, 16, 10), acts=(pnn.SIGMOID, 9), loss=pnn.LOSS_MSE),
]


@pytest.mark.parametrize("kw", BAD)
def test_invalid_configs_are_rejected_before_any_device_work(kw):
    cfg = pnn.make_config(**kw)
    assert pnn.config_check(cfg) == pnn.PNN_EINVAL
    assert pnn.param_count(cfg) == 0
    h = ctypes.c_void_p(123)
    th = np.zeros(16, np.float32)
    st = pnn.lib().pnn_init(ctypes.byref(cfg), th.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), None,
                            ctypes.byref(h))
    assert st == pnn.PNN_EINVAL and h.value is None
    assert pnn.lib().pnn_last_error(None).decode().startswith("invalid config")


def test_null_arguments_are_rejected():
    L = pnn.lib()
    cfg = pnn.config_from_workload(I.WORKLOADS[0])
    assert L.pnn_init(ctypes.byref(cfg), None, None, ctypes.byref(ctypes.c_void_p())) == pnn.PNN_EINVAL
    assert L.pnn_init(ctypes.byref(cfg), None, None, None) == pnn.PNN_EINVAL
    assert L.pnn_train_epoch(None, None, None, 10, None) == pnn.PNN_EINVAL
    assert L.pnn_merge(None, 0, None) == pnn.PNN_EINVAL
    assert L.pnn_eval(None, -1, None, None, 10, None, None, None) == pnn.PNN_EINVAL
    assert L.pnn_shard(10, 0, 0, None, None) == pnn.PNN_EINVAL
    assert L.pnn_plan(None) == b""
    L.pnn_destroy(None)  # ignored
