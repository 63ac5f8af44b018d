"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Every test here runs without a GPU.  Each one is chosen so that a plausible mistake in
the oracle (a dropped term, a wrong sign or index, a transposed operand, a wrong scale,
a wrong split or merge) fails at least one of them:

* hand-derived single steps of eq. (2)-(13) (tests/golden),
* central finite differences of the cost (independent of back-propagation),
* torch.autograd in float64 (a library routine computing the same derivative),
* invariants of the method: shard partition, merge identities, mini-batch averaging,
  eta = 0, K = 1, replica independence, softmax normalisation,
* bf16 rounding against torch's float32 -> bfloat16 conversion, and a hand-derived bf16-mixed
  step in which every rounding point of the mixed-precision reading changes the result.
"""
import json
import os

import numpy as np
import pytest

import pnn_inputs as I
from oracle import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")
ACT = {"sigmoid": O.SIGMOID, "tanh": O.TANH, "relu": O.RELU, "leaky_relu": O.LEAKY_RELU, "softmax": O.SOFTMAX}


def _flat(d):
    return np.concatenate([np.ravel(d["W1"]), d["b1"], np.ravel(d["W2"]), d["b2"]]).astype(np.float64)


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ------------------------------------------------------------------------------------
# worked single steps

@pytest.mark.parametrize("loss", ["mse", "xent"])
def test_worked_2_2_1_sigmoid(loss):
    g = _load("worked_2_2_1_sigmoid.json")
    o = O.Oracle(g["sizes"], [ACT[a] for a in g["acts"]], O.LOSS_MSE if loss == "mse" else O.LOSS_XENT,
                 lr=g["lr"])
    th = _flat(g)
    x = np.array(g["x"], dtype=np.float32)
    (z1, a1, d1), (z2, a2, d2) = o.trace(th, x, g["label"])
    exp = g[loss]
    ref = g["mse"]
    np.testing.assert_allclose(z1, ref["z1"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(a1, ref["a1"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(z2, ref["z2"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(a2, ref["a2"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(d2, exp["d2"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(d1, exp["d1"], rtol=0, atol=1e-10)
    if loss == "mse":
        assert o.cost(th, x[None, :], np.array([g["label"]], np.int32)) == pytest.approx(ref["cost"], abs=1e-10)
    theta = th[None, :].copy()
    o.train_epoch(theta, x[None, :], np.array([g["label"]], np.int32))
    (W1, b1), (W2, b2) = o.split(theta[0])
    np.testing.assert_allclose(W1, exp["W1_new"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(b1, exp["b1_new"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(W2, exp["W2_new"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(b2, exp["b2_new"], rtol=0, atol=1e-10)


def test_worked_2_2_2_relu_softmax():
    g = _load("worked_2_2_2_relu_softmax.json")
    o = O.Oracle(g["sizes"], [ACT[a] for a in g["acts"]], O.LOSS_XENT, lr=g["lr"])
    th = _flat(g)
    x = np.array(g["x"], dtype=np.float32)
    (z1, a1, d1), (z2, a2, d2) = o.trace(th, x, g["label"])
    for got, key in ((z1, "z1"), (a1, "a1"), (z2, "z2"), (a2, "a2"), (d2, "d2"), (d1, "d1")):
        np.testing.assert_allclose(got, g[key], rtol=0, atol=1e-10, err_msg=key)
    assert z1[0] == 0.0  # the rectifier derivative at exactly zero is exercised
    assert o.cost(th, x[None, :], np.array([0], np.int32)) == pytest.approx(g["cost"], abs=1e-10)
    theta = th[None, :].copy()
    o.train_epoch(theta, x[None, :], np.array([0], np.int32))
    (W1, b1), (W2, b2) = o.split(theta[0])
    for got, key in ((W1, "W1_new"), (b1, "b1_new"), (W2, "W2_new"), (b2, "b2_new")):
        np.testing.assert_allclose(got, g[key], rtol=0, atol=1e-10, err_msg=key)


# ------------------------------------------------------------------------------------
# gradients: finite differences and torch.autograd

NETS = [
    # sizes, hidden activations, output activation, loss
    ((5, 4, 3), (O.SIGMOID,), O.SIGMOID, O.LOSS_MSE),
    ((5, 4, 3), (O.TANH,), O.SIGMOID, O.LOSS_MSE),
    ((5, 4, 3), (O.SIGMOID,), O.SIGMOID, O.LOSS_XENT),
    ((5, 4, 3), (O.RELU,), O.SOFTMAX, O.LOSS_XENT),
    ((5, 4, 3), (O.LEAKY_RELU,), O.TANH, O.LOSS_MSE),
    ((6, 5, 4, 3), (O.RELU, O.TANH), O.SOFTMAX, O.LOSS_XENT),
    ((7, 3, 5, 2), (O.SIGMOID, O.RELU), O.SIGMOID, O.LOSS_MSE),
]


@pytest.mark.parametrize("net", NETS, ids=lambda n: "x".join(map(str, n[0])) + f"-a{n[1]}-{n[2]}-l{n[3]}")
def test_gradient_matches_finite_differences(net):
    sizes, hid, out, loss = net
    o = O.Oracle(sizes, list(hid) + [out], loss)
    th = I.random_params(sizes, seed=11).astype(np.float64)
    x, y = I.random_batch(sizes[0], sizes[-1], 3, seed=12)
    g = o.gradient(th, x, y)
    h = 1e-6
    fd = np.empty_like(th)
    for i in range(th.size):
        tp, tm = th.copy(), th.copy()
        tp[i] += h
        tm[i] -= h
        fd[i] = (o.cost(tp, x, y) - o.cost(tm, x, y)) / (2 * h)
    scale = np.abs(fd).max()
    assert np.abs(g - fd).max() <= 1e-6 * scale


def _torch_grad(sizes, acts, loss, th, x, y):
    torch = pytest.importorskip("torch")
    t = torch.tensor(th, dtype=torch.float64, requires_grad=True)
    a = torch.tensor(x, dtype=torch.float64)
    o = 0
    L = len(sizes) - 1
    for l in range(L):
        n_in, n_out = sizes[l], sizes[l + 1]
        W = t[o:o + n_in * n_out].reshape(n_out, n_in)
        o += n_in * n_out
        b = t[o:o + n_out]
        o += n_out
        z = a @ W.T + b
        f = acts[l]
        if f == O.SIGMOID:
            a = torch.sigmoid(z)
        elif f == O.TANH:
            a = torch.tanh(z)
        elif f == O.RELU:
            a = torch.relu(z)
        elif f == O.LEAKY_RELU:
            a = torch.nn.functional.leaky_relu(z, 0.01)
        else:
            a = torch.softmax(z, dim=1)
    e = torch.nn.functional.one_hot(torch.tensor(y, dtype=torch.int64), sizes[-1]).to(torch.float64)
    if loss == O.LOSS_MSE:
        c = 0.5 * ((a - e) ** 2).sum(dim=1)
    elif acts[-1] == O.SOFTMAX:
        c = -(e * torch.log(a)).sum(dim=1)
    else:
        c = -(e * torch.log(a) + (1 - e) * torch.log(1 - a)).sum(dim=1)
    c.mean().backward()
    return t.grad.numpy()


@pytest.mark.parametrize("net", NETS, ids=lambda n: "x".join(map(str, n[0])) + f"-a{n[1]}-{n[2]}-l{n[3]}")
def test_gradient_matches_torch_autograd(net):
    sizes, hid, out, loss = net
    acts = list(hid) + [out]
    o = O.Oracle(sizes, acts, loss)
    th = I.random_params(sizes, seed=21).astype(np.float64)
    x, y = I.random_batch(sizes[0], sizes[-1], 8, seed=22)  # random inputs: no pre-activation is exactly 0
    np.testing.assert_allclose(o.gradient(th, x, y), _torch_grad(sizes, acts, loss, th, x, y), rtol=1e-10,
                               atol=1e-13)


def test_relu_derivative_at_zero_is_one():
    # a hidden unit whose pre-activation is exactly 0 passes the error back (eq. 4 branch z >= 0)
    o = O.Oracle((1, 1, 1), (O.RELU, O.SIGMOID), O.LOSS_MSE)
    th = np.array([0.0, 0.0, 2.0, 0.0])  # z1 = 0*x + 0 = 0
    (z1, a1, d1), (_, _, d2) = o.trace(th, np.array([1.0], np.float32), 0)
    assert z1[0] == 0.0 and a1[0] == 0.0
    assert d1[0] == pytest.approx(2.0 * d2[0], abs=0)


# ------------------------------------------------------------------------------------
# training schedule invariants

def test_one_batch_step_is_eta_times_mean_of_per_sample_gradients():
    sizes = (6, 5, 3)
    o = O.Oracle(sizes, (O.TANH, O.SIGMOID), O.LOSS_MSE, batch=4, lr=0.3)
    th = I.random_params(sizes, seed=31).astype(np.float64)
    x, y = I.random_batch(6, 3, 4, seed=32)
    per = np.mean([o.gradient(th, x[i:i + 1], y[i:i + 1]) for i in range(4)], axis=0)
    theta = th[None, :].copy()
    o.train_epoch(theta, x, y)
    np.testing.assert_allclose(theta[0], th - np.float32(0.3) * per, rtol=1e-12, atol=1e-15)


def test_partial_last_batch_uses_its_own_size():
    sizes = (6, 5, 3)
    lr = np.float64(np.float32(0.2))
    o = O.Oracle(sizes, (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, batch=2, lr=0.2)
    th = I.random_params(sizes, seed=41).astype(np.float64)
    x, y = I.random_batch(6, 3, 5, seed=42)  # batches of 2, 2, 1
    ref = th.copy()
    for s, e in ((0, 2), (2, 4), (4, 5)):
        ref = ref - lr * o.gradient(ref, x[s:e], y[s:e])
    theta = th[None, :].copy()
    o.train_epoch(theta, x, y)
    np.testing.assert_allclose(theta[0], ref, rtol=1e-12, atol=1e-15)


def test_batch_of_copies_equals_one_per_sample_step():
    sizes = (6, 5, 3)
    th = I.random_params(sizes, seed=51).astype(np.float64)
    x, y = I.random_batch(6, 3, 1, seed=52)
    a = O.Oracle(sizes, (O.RELU, O.SOFTMAX), O.LOSS_XENT, batch=8, lr=0.1)
    b = O.Oracle(sizes, (O.RELU, O.SOFTMAX), O.LOSS_XENT, batch=1, lr=0.1)
    ta, tb = th[None].copy(), th[None].copy()
    a.train_epoch(ta, np.repeat(x, 8, 0), np.repeat(y, 8))
    b.train_epoch(tb, x, y)
    np.testing.assert_allclose(ta, tb, rtol=1e-13, atol=1e-16)


def test_zero_learning_rate_is_a_no_op():
    sizes = (6, 5, 3)
    o = O.Oracle(sizes, (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, replicas=2, batch=3, lr=0.0)
    th = o.replicate(I.random_params(sizes, seed=61))
    before = th.copy()
    x, y = I.random_batch(6, 3, 10, seed=62)
    o.train_epoch(th, x, y)
    assert np.array_equal(th, before)


def test_sample_order_matters_for_sgd():
    # per-sample SGD visits the slice in order; a reversed slice ends elsewhere
    sizes = (6, 5, 3)
    o = O.Oracle(sizes, (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, lr=0.5)
    th = I.random_params(sizes, seed=71)
    x, y = I.random_batch(6, 3, 6, seed=72)
    a, b = o.replicate(th), o.replicate(th)
    o.train_epoch(a, x, y)
    o.train_epoch(b, x[::-1], y[::-1])
    assert not np.allclose(a, b)
    # and equals the composition of single steps in shard order
    c = o.replicate(th)
    for i in range(6):
        o.train_epoch(c, x[i:i + 1], y[i:i + 1])
    np.testing.assert_array_equal(a, c)


# ------------------------------------------------------------------------------------
# split, replicas, merge

@pytest.mark.parametrize("n,k", [(2000, 1), (60000, 4), (60000, 16), (240000, 64), (600000, 256), (10, 3), (7, 7)])
def test_shards_partition_the_data(n, k):
    o = O.Oracle((4, 2), (O.SIGMOID,), O.LOSS_MSE, replicas=k)
    spans = [o.shard(n, i) for i in range(k)]
    assert spans[0][0] == 0
    for (s0, l0), (s1, _) in zip(spans, spans[1:]):
        assert s0 + l0 == s1
    assert spans[-1][0] + spans[-1][1] == n
    lens = [l for _, l in spans]
    assert max(lens) - min(lens) <= 1 and lens == sorted(lens, reverse=True)
    if (n, k) == (600000, 256):
        assert lens[:192] == [2344] * 192 and lens[192:] == [2343] * 64


def test_each_replica_trains_only_on_its_own_slice():
    sizes = (6, 5, 3)
    K = 3
    o = O.Oracle(sizes, (O.TANH, O.SIGMOID), O.LOSS_MSE, replicas=K, batch=2, lr=0.2)
    single = O.Oracle(sizes, (O.TANH, O.SIGMOID), O.LOSS_MSE, replicas=1, batch=2, lr=0.2)
    th0 = I.random_params(sizes, seed=81)
    x, y = I.random_batch(6, 3, 11, seed=82)
    th = o.replicate(th0)
    o.train_epoch(th, x, y, threads=3)
    for k in range(K):
        s, n = o.shard(11, k)
        t = single.replicate(th0)
        single.train_epoch(t, x[s:s + n], y[s:s + n])
        np.testing.assert_array_equal(th[k], t[0])
    # threads do not change the result
    th1 = o.replicate(th0)
    o.train_epoch(th1, x, y, threads=1)
    np.testing.assert_array_equal(th, th1)
    # and the sampled-replica entry point agrees
    sub = np.tile(np.asarray(th0, np.float64), (2, 1))
    o.train_replicas(sub, [2, 0], x, y)
    np.testing.assert_array_equal(sub[0], th[2])
    np.testing.assert_array_equal(sub[1], th[0])


def test_k1_pnn_equals_snn():
    sizes = (6, 5, 3)
    o = O.Oracle(sizes, (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, replicas=1, batch=1, lr=0.3)
    th0 = I.random_params(sizes, seed=91)
    x, y = I.random_batch(6, 3, 9, seed=92)
    th = o.replicate(th0)
    o.train_epoch(th, x, y)
    merged = o.merge(th)
    np.testing.assert_array_equal(merged, th[0])
    ref = np.asarray(th0, np.float64).copy()
    for i in range(9):
        ref = ref - np.float64(np.float32(0.3)) * o.gradient(ref, x[i:i + 1], y[i:i + 1])
    np.testing.assert_allclose(merged, ref, rtol=1e-12, atol=1e-15)


def test_merge_of_identical_replicas_is_identity():
    o = O.Oracle((6, 5, 3), (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, replicas=7)
    th0 = I.random_params((6, 5, 3), seed=101)
    assert np.array_equal(o.merge(o.replicate(th0)), np.asarray(th0, np.float64))


@pytest.mark.parametrize("K", [2, 3, 64, 256])
def test_merge_of_k_is_mean_index(K):
    o = O.Oracle((3, 2), (O.SIGMOID,), O.LOSS_MSE, replicas=K)
    th = np.repeat(np.arange(K, dtype=np.float64)[:, None], o.P, axis=1)
    assert np.all(o.merge(th) == (K - 1) / 2)


@pytest.mark.parametrize("K", [2, 5, 64, 256])
def test_weighted_merge_closed_form(K):
    # theta_k = k everywhere, w_k = k + 1: sum k (k + 1) / sum (k + 1) = 2 (K - 1) / 3
    o = O.Oracle((3, 2), (O.SIGMOID,), O.LOSS_MSE, replicas=K)
    th = np.repeat(np.arange(K, dtype=np.float64)[:, None], o.P, axis=1)
    got = o.merge_weighted(th, np.arange(1, K + 1, dtype=np.float64))
    np.testing.assert_allclose(got, 2.0 * (K - 1) / 3.0, rtol=1e-15, atol=0)


def test_weighted_merge_special_cases():
    K = 6
    o = O.Oracle((6, 5, 3), (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, replicas=K)
    th = np.stack([np.asarray(I.random_params((6, 5, 3), seed=300 + k), np.float64) for k in range(K)])
    # equal weights: the plain average
    np.testing.assert_allclose(o.merge_weighted(th, [2.5] * K), o.merge(th), rtol=1e-15, atol=1e-18)
    # a one-hot weight selects that CN exactly
    for j in (0, 3):
        w = np.zeros(K)
        w[j] = 0.7
        assert np.array_equal(o.merge_weighted(th, w), th[j])
    # scaling every weight changes nothing; a weight of 2 counts a CN twice
    w = np.array([1.0, 2.0, 0.0, 3.0, 1.0, 0.5])
    np.testing.assert_allclose(o.merge_weighted(th, 4 * w), o.merge_weighted(th, w), rtol=1e-15, atol=1e-18)
    dup = np.concatenate([th, th[1:2]])
    o7 = O.Oracle((6, 5, 3), (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, replicas=K + 1)
    w7 = np.array([1.0, 1.0, 0.0, 3.0, 1.0, 0.5, 1.0])
    np.testing.assert_allclose(o.merge_weighted(th, w), o7.merge_weighted(dup, w7), rtol=1e-14, atol=1e-17)


def test_merge_is_the_mean():
    K = 5
    o = O.Oracle((6, 5, 3), (O.SIGMOID, O.SIGMOID), O.LOSS_MSE, replicas=K)
    rng = np.random.default_rng(5)
    th = rng.standard_normal((K, o.P))
    np.testing.assert_allclose(o.merge(th), th.mean(axis=0), rtol=1e-15, atol=1e-16)


# ------------------------------------------------------------------------------------
# output layer, classification

def test_softmax_outputs_sum_to_one_and_argmax_lowest_index():
    sizes = (6, 5, 4)
    o = O.Oracle(sizes, (O.RELU, O.SOFTMAX), O.LOSS_XENT)
    th = I.random_params(sizes, seed=111)
    x, y = I.random_batch(6, 4, 20, seed=112)
    out = o.forward(th, x)
    np.testing.assert_allclose(out.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    pred, correct = o.predict(th, x, y)
    assert np.array_equal(pred, out.argmax(axis=1)) and correct == int((pred == y).sum())
    # ties: all-zero weights give equal outputs, the lowest index wins
    pred0, _ = o.predict(np.zeros(o.P), x)
    assert np.all(pred0 == 0)


# ------------------------------------------------------------------------------------
# bf16 rounding points

def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    v = np.concatenate([rng.standard_normal(2000).astype(np.float32),
                        (rng.standard_normal(200) * 1e-38).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0, 3.0e38], np.float32)])
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([O.round_bf16(float(a)) for a in v])
    np.testing.assert_array_equal(got, ref)


def test_worked_2_2_2_sigmoid_softmax_bf16_step():
    """One bf16-mixed step against a hand derivation (tests/golden/derive_bf16_step.py) in which
    every rounding point of the reading changes the result: the oracle matches the derived
    intermediates and updated parameters to 1e-12, and each variant with one rounding point moved
    or dropped (x, operand weights, a1, d2, d1 unrounded; d1 rounded before the derivative
    product; the derivative taken from the unrounded a1) is at least 5e-5 away from it."""
    g = _load("worked_2_2_2_sigmoid_softmax_bf16.json")
    o = O.Oracle(g["sizes"], [ACT[a] for a in g["acts"]], O.LOSS_XENT, precision=O.BF16, lr=g["lr"])
    th = _flat(g)
    x = np.array(g["x"], dtype=np.float32)
    assert np.array_equal(x.astype(np.float64), g["x"])  # (the inputs are float32 values)
    (z1, a1, d1), (z2, a2, d2) = o.trace(th, x, g["label"])
    np.testing.assert_allclose(z1, g["z1"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(a1, g["a1b"], rtol=0, atol=0)       # hidden activation stored in bf16
    np.testing.assert_allclose(z2, g["z2"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(a2, g["a2"], rtol=0, atol=1e-12)    # softmax output not rounded
    np.testing.assert_allclose(d2, g["d2b"], rtol=0, atol=0)
    np.testing.assert_allclose(d1, g["d1b"], rtol=0, atol=0)
    theta = th[None, :].copy()
    o.train_epoch(theta, x[None, :], np.array([g["label"]], np.int32))
    got = theta[0]
    want = _flat({"W1": g["W1_new"], "b1": g["b1_new"], "W2": g["W2_new"], "b2": g["b2_new"]})
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    for name, v in g["variants"].items():
        alt = _flat({"W1": v["W1_new"], "b1": v["b1_new"], "W2": v["W2_new"], "b2": v["b2_new"]})
        assert np.max(np.abs(alt - want)) >= 5e-5, name


def test_bf16_mode_equals_exact_mode_when_nothing_needs_rounding():
    # one weight layer, bf16-representable inputs and weights, softmax output: the only
    # rounding point left is the stored output error, so the forward pass is exact and the
    # gradient is within one bf16 rounding of the exact one
    sizes = (8, 4)
    e = O.Oracle(sizes, (O.SOFTMAX,), O.LOSS_XENT)
    b = O.Oracle(sizes, (O.SOFTMAX,), O.LOSS_XENT, precision=O.BF16)
    th = np.array([O.round_bf16(v) for v in I.random_params(sizes, seed=121)])
    x, y = I.random_batch(8, 4, 1, seed=122)
    x = np.array([[O.round_bf16(v) for v in x[0]]], np.float32)
    np.testing.assert_array_equal(e.forward(th, x), b.forward(th, x))
    ge, gb = e.gradient(th, x, y), b.gradient(th, x, y)
    assert not np.array_equal(ge, gb)
    np.testing.assert_allclose(gb, ge, rtol=2 ** -8, atol=1e-12)


def test_bf16_mode_is_close_to_exact_mode():
    sizes = (20, 12, 6, 4)
    e = O.Oracle(sizes, (O.RELU, O.RELU, O.SOFTMAX), O.LOSS_XENT)
    b = O.Oracle(sizes, (O.RELU, O.RELU, O.SOFTMAX), O.LOSS_XENT, precision=O.BF16)
    th = I.random_params(sizes, seed=131)
    x, y = I.random_batch(20, 4, 16, seed=132)
    fe, fb = e.forward(th, x), b.forward(th, x)
    assert not np.array_equal(fe, fb)
    np.testing.assert_allclose(fb, fe, rtol=0, atol=3e-2)


# ------------------------------------------------------------------------------------
# the method learns (qualitative smoke signal on synthetic data)

def test_synthetic_workload_is_learned():
    w = I.WORKLOADS[0]
    o = O.Oracle.from_workload(w)
    x, y = I.train_set(w, 1000)
    xt, yt = I.test_set(w, 1000)
    th = o.replicate(I.init_params(w))
    o.train_epoch(th, x, y)
    _, correct = o.predict(o.merge(th), xt, yt)
    assert correct / 1000 > 0.5
