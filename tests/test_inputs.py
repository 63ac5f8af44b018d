"""The seeded synthetic input recipe (MNIST-shaped stand-in data and Xavier initial parameters)."""
import numpy as np

import pnn_inputs as I


def test_workload_presets_have_the_stated_shapes():
    P = [w.param_count() for w in I.WORKLOADS]
    assert P == [12_730, 101_770, 203_530, 535_818, 814_090]
    assert [w.replicas for w in I.WORKLOADS] == [1, 4, 16, 64, 256]
    assert [w.batch for w in I.WORKLOADS] == [1, 1, 32, 64, 128]


def test_samples_are_seeded_bounded_and_labelled():
    w = I.WORKLOADS[2]
    x1, y1 = I.train_set(w, 500)
    x2, y2 = I.train_set(w, 500)
    assert np.array_equal(x1, x2) and np.array_equal(y1, y2)
    assert x1.dtype == np.float32 and x1.shape == (500, 784)
    assert x1.min() >= 0.0 and x1.max() <= 1.0
    assert set(np.unique(y1)) <= set(range(10)) and len(np.unique(y1)) == 10
    xt, _ = I.test_set(w, 500)
    assert not np.array_equal(xt, x1)
    # the noise around the prototype has the stated spread (before clipping)
    protos = I.prototypes(w)
    assert protos.shape == (200, 784)


def test_init_is_xavier_uniform_with_zero_bias():
    w = I.WORKLOADS[1]
    th = I.init_params(w)
    assert th.dtype == np.float32 and th.size == w.param_count()
    W1 = th[:128 * 784]
    a = np.sqrt(6 / (784 + 128))
    assert np.abs(W1).max() <= a and np.abs(W1).max() > 0.95 * a
    assert np.all(th[128 * 784:128 * 785] == 0)
    assert np.array_equal(th, I.init_params(w))
