"""How much the oracle itself moves when its start moves by one fp32 ulp (CPU only).

The GPU parity bars compare two implementations whose arithmetic differs in the order of fp32
(or bf16) roundings.  A bar measures the implementation only where the method does not amplify
rounding differences to its own size.  For each GPU parity case this test runs the oracle from
theta0 and from theta0 with every value moved by one fp32 ulp (seeded signs), and asserts:

* fp32 epoch cases (tests/cases.py): the oracle's own divergence stays below half the 1e-3
  epoch bar;
* the sensitive fp32 cases (a tanh hidden layer under sigmoid outputs with the cross-entropy
  error): some element reaches half the bar for some seed, every layer stays below a tenth of
  it normwise (so the GPU compares those epochs normwise, and every step elementwise);
* the reduced bf16-mixed epoch case: the tensors held elementwise (tests/cases.py
  BF16_ELEMENTWISE) stay below half the 2e-2 bar for every seed; every other tensor reaches half
  the bar for some seed (so it is compared normwise only); every layer stays below a tenth of
  the bar normwise;
* the bf16-mixed workload at full size (784-512-256-10, one CN, one 3,750-row epoch): every
  weight tensor reaches half the bar elementwise, every layer stays below a fifth of it normwise.
"""
import numpy as np
import pytest

import pnn_inputs as I
from oracle import oracle as O
from tests.cases import BF16_ELEMENTWISE, CHUNKED_CASES, EPOCH_CASES, SENSITIVE_FP32_CASES, case_key
from tests.parity import BF16_TOL, EPOCH_TOL, layer_err, oracle_replicas, rel_err


def one_ulp(theta0: np.ndarray, seed: int) -> np.ndarray:
    """Every value moved to its fp32 neighbour, up or down by a seeded sign."""
    rng = np.random.default_rng(seed)
    t = theta0.astype(np.float32)
    up = rng.choice([False, True], t.shape)
    return np.where(up, np.nextafter(t, np.float32(np.inf)), np.nextafter(t, np.float32(-np.inf))).astype(np.float64)


def run(w, theta0, X, y, epochs):
    """The oracle's epochs (with the workload's merges); the CNs after each epoch."""
    o = O.Oracle.from_workload(w)
    th = np.tile(theta0, (w.replicas, 1))
    out = []
    for _ in range(epochs):
        o.train_epoch(th, X, y, threads=8)
        out.append(th.copy())
        if w.merge_every_epoch:
            th[:] = o.merge(th)[None, :]
    return out


FP32_CASES = [c for c in EPOCH_CASES if I.WORKLOADS[c[0]].scaled(**c[1]).precision == I.FP32] + \
             [(1, over, N, 1) for over, N in CHUNKED_CASES]


@pytest.mark.parametrize("idx,over,N,epochs", FP32_CASES)
def test_fp32_epoch_bar_is_above_the_oracles_own_sensitivity(idx, over, N, epochs):
    w = I.WORKLOADS[idx].scaled(**over)
    X, y = I.train_set(w, N)
    th0 = I.init_params(w).astype(np.float64)
    a = run(w, th0, X, y, epochs)
    b = run(w, one_ulp(th0, 0), X, y, epochs)
    worst = max(max(rel_err(w.sizes, b[e][k], a[e][k]).values()) for e in range(epochs) for k in range(w.replicas))
    assert worst <= EPOCH_TOL / 2, worst


@pytest.mark.parametrize("idx,over,N,epochs", SENSITIVE_FP32_CASES)
def test_sensitive_fp32_cases_are_chaotic_elementwise_only(idx, over, N, epochs):
    w = I.WORKLOADS[idx].scaled(**over)
    X, y = I.train_set(w, N)
    th0 = I.init_params(w).astype(np.float64)
    a = run(w, th0, X, y, epochs)
    worst = worst_layer = 0.0
    for seed in range(6):
        b = run(w, one_ulp(th0, seed), X, y, epochs)
        for e in range(epochs):
            for k in range(w.replicas):
                worst = max(worst, max(rel_err(w.sizes, b[e][k], a[e][k]).values()))
                worst_layer = max(worst_layer, max(layer_err(w.sizes, b[e][k], a[e][k]).values()))
    assert worst >= EPOCH_TOL / 2, worst
    assert worst_layer < EPOCH_TOL / 10, worst_layer


BF16_REDUCED = [(3, dict(replicas=8), 8 * 150 + 3, 2), (3, dict(replicas=6), 6 * 150 + 5, 1)]


@pytest.mark.parametrize("idx,over,N,epochs", BF16_REDUCED)
def test_bf16_reduced_case_elementwise_tensors(idx, over, N, epochs):
    w = I.WORKLOADS[idx].scaled(**over)
    table = BF16_ELEMENTWISE[case_key(idx, over, N, epochs)]
    X, y = I.train_set(w, N)
    th0 = I.init_params(w).astype(np.float64)
    a = run(w, th0, X, y, epochs)
    names = [n for n, _ in zip(["W1", "b1", "W2", "b2", "W3", "b3"], range(2 * w.n_layers))]
    worst = {e: dict.fromkeys(names, 0.0) for e in range(epochs)}
    worst_layer = 0.0
    for seed in range(3):
        b = run(w, one_ulp(th0, seed), X, y, epochs)
        for e in range(epochs):
            for k in range(w.replicas):
                for n, v in rel_err(w.sizes, b[e][k], a[e][k]).items():
                    worst[e][n] = max(worst[e][n], v)
                worst_layer = max(worst_layer, max(layer_err(w.sizes, b[e][k], a[e][k]).values()))
    for e in range(epochs):
        for n in names:
            if n in table[e]:
                assert worst[e][n] < BF16_TOL / 2, (e, n, worst[e])
            else:
                assert worst[e][n] >= BF16_TOL / 2, (e, n, worst[e])
    assert worst_layer < BF16_TOL / 10, worst_layer


def test_bf16_full_size_epoch_is_chaotic_elementwise():
    w = I.WORKLOADS[3]
    o = O.Oracle.from_workload(w)
    X, y = I.train_set(w)
    st, ln = o.shard(w.n_train, 0)
    th0 = I.init_params(w).astype(np.float64)
    # CN 0's epoch from theta0 and from two perturbed starts, side by side
    r = oracle_replicas(o, np.stack([th0, one_ulp(th0, 0), one_ulp(th0, 3)]), [0, 0, 0], X, y, threads=3)
    e = [rel_err(w.sizes, r[i], r[0]) for i in (1, 2)]
    assert all(max(ei[n] for ei in e) >= BF16_TOL / 2 for n in ("W1", "W2", "W3")), e
    lay = [layer_err(w.sizes, r[i], r[0]) for i in (1, 2)]
    assert max(max(li.values()) for li in lay) < BF16_TOL / 5, lay
    assert ln == 3750 and st == 0
