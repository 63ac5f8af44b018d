"""GPU parity of the HIP library against the CPU oracle, through the C ABI.

Every case feeds both sides the same seeded inputs and the same initial parameters, then
compares per-weight relative errors (see tests/parity.py): <= 1e-5 after one step and
<= 1e-3 after full epochs in fp32, <= 2e-2 in bf16-mixed precision; predictions on held-out
data must equal the oracle's argmax except on near-ties.  Cases cover every workload's
shapes at sizes the oracle finishes in seconds (several tiles, ragged last batches and
chunks, uneven slices), the workloads at full size (sampled child networks where the oracle
would take too long), and the edge cases of the method.
"""
import numpy as np
import pytest

import pnn_inputs as I
from oracle import oracle as O
from tests.cases import BF16_ELEMENTWISE, CHUNKED_CASES, EPOCH_CASES, SENSITIVE_FP32_CASES, case_key
from tests.parity import (BF16_TOL, EPOCH_TOL, STEP_TOL, argmax_agrees, assert_close, log, oracle_replicas,
                          rel_err)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2304_09590_amd import pnn as B  # noqa: E402


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def make_net(w, theta0):
    return B.PNN(B.config_from_workload(w), theta0)


def tol_for(w, epoch=False):
    if w.precision == I.BF16_MIXED:
        return BF16_TOL
    return EPOCH_TOL if epoch else STEP_TOL


def close_epoch(w, got, ref, what, elementwise=()):
    """Comparison after whole epochs.  fp32: every weight and bias elementwise at 1e-3.
    bf16-mixed: every layer normwise at 2e-2, and the tensors named in `elementwise` also
    elementwise (rms floor) at 2e-2 -- those whose elementwise divergence the oracle's own
    one-ulp sensitivity keeps below half the bar (tests/cases.py, tests/test_sensitivity.py)."""
    if w.precision != I.BF16_MIXED:
        return assert_close(w.sizes, got, ref, EPOCH_TOL, what)
    worst = assert_close(w.sizes, got, ref, BF16_TOL, what, layerwise=True)
    if elementwise:
        e = {k: v for k, v in rel_err(w.sizes, got, ref).items() if k in elementwise}
        assert max(e.values()) <= BF16_TOL, f"{what}: elementwise {e} exceed {BF16_TOL}"
        worst = max(worst, max(e.values()))
    return worst


def predictions_agree(w, o, theta_oracle_trained, pred_gpu, Xt):
    """Held-out predictions of the GPU-trained network against those of the network the oracle
    trained itself from the same start on the same rows: equal except where the oracle-trained
    network's top two outputs are within the margin (1e-3 in fp32, where trained parameters agree
    to 1e-3 relative; 5e-2 in bf16-mixed)."""
    out = o.forward(np.asarray(theta_oracle_trained, np.float64), Xt)
    n = argmax_agrees(out, pred_gpu, margin=1e-3 if w.precision == I.FP32 else 5e-2)
    log(f"held-out predictions of the oracle-trained network: {n} of {len(Xt)} differ (near-ties)")
    return n


# ------------------------------------------------------------------------------------
# one training step of every workload's net

STEP_CASES = [
    (0, None),
    (1, None),
    (2, None),
    (3, [0, 31, 63]),
    (4, [0, 100, 255]),
]


@pytest.mark.parametrize("idx,ids", STEP_CASES, ids=[I.WORKLOADS[c[0]].name for c in STEP_CASES])
def test_one_step(idx, ids):
    w = I.WORKLOADS[idx]
    K, Bt = w.replicas, w.batch
    N = K * Bt
    log(f"one step: {w.name} N={N}")
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    net.train_epoch(dev(X), dev(y))
    torch.cuda.synchronize()
    o = O.Oracle.from_workload(w)
    ids = list(range(K)) if ids is None else ids
    ref = oracle_replicas(o, np.tile(th0.astype(np.float64), (len(ids), 1)), ids, X, y)
    for i, k in enumerate(ids):
        got = net.get_params(k)
        assert_close(w.sizes, got, ref[i], tol_for(w), f"replica {k}")
        if w.precision == I.FP32:
            # the update itself, relative to its own size
            e = rel_err(w.sizes, got.astype(np.float64) - th0, ref[i] - th0)
            assert max(e.values()) <= 1e-3, e
    net.close()


# ------------------------------------------------------------------------------------
# full epochs at reduced sizes: ragged last batches / chunks, uneven slices, merges



@pytest.mark.parametrize("idx,over,N,epochs", EPOCH_CASES)
def test_epochs(idx, over, N, epochs):
    w = I.WORKLOADS[idx].scaled(**over)
    K = w.replicas
    ew = BF16_ELEMENTWISE.get(case_key(idx, over, N, epochs), {})
    log(f"epochs: {w.name} {over} N={N} epochs={epochs}")
    X, y = I.train_set(w, N)
    Xt, yt = I.test_set(w, 3000)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    log(f"plan: {net.plan}")
    xd, yd = dev(X), dev(y)
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    for e in range(epochs):
        net.train_epoch(xd, yd)
        o.train_epoch(ref, X, y, threads=8)
        for k in range(K):
            close_epoch(w, net.get_params(k), ref[k], f"epoch {e} replica {k}", ew.get(e, ()))
        if w.merge_every_epoch:
            net.merge(broadcast=True)
            m = o.merge(ref)
            ref[:] = m[None, :]
            close_epoch(w, net.get_params(-1), m, f"merged epoch {e}", ew.get(e, ()))
            assert np.array_equal(net.get_params(0), net.get_params(-1))
    if not w.merge_every_epoch:
        net.merge(broadcast=False)
    merged = net.get_params(-1)
    close_epoch(w, merged, o.merge(ref), "merged")
    # predictions with the GPU's merged weights against the oracle's forward of the same weights
    pred = torch.empty(len(yt), dtype=torch.int32, device="cuda")
    out = torch.empty((len(yt), w.sizes[-1]), dtype=torch.float32, device="cuda")
    correct = net.infer(dev(Xt), pred, which=-1, out=out, y=dev(yt), count=True)
    out_ref = o.forward(merged.astype(np.float64), Xt)
    p = pred.cpu().numpy()
    argmax_agrees(out_ref, p, margin=1e-5 if w.precision == I.FP32 else 2e-2)
    assert correct == int((p == yt).sum())
    np.testing.assert_allclose(out.cpu().numpy(), out_ref, rtol=0, atol=1e-5 if w.precision == I.FP32 else 2e-2)
    # and against the network the oracle trained and merged itself
    predictions_agree(w, o, o.merge(ref), p, Xt)
    net.close()


# ------------------------------------------------------------------------------------
# the per-sample chunked plan (B = 1, one hidden layer, where the persistent per-sample kernel
# does not fit): Gram blocks of each chunk of T samples, the chunk's input sums W1 x_t as one
# product, the T sequential steps, and the chunk's rank-T update of W1 as one product



@pytest.mark.parametrize("over,N", CHUNKED_CASES)
def test_chunked_plan_one_step(over, N):
    w = I.WORKLOADS[1].scaled(**over)
    K = w.replicas
    X, y = I.train_set(w, K)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    assert net.plan == "per-sample chunked"
    log(f"chunked one step: {w.name} {over}")
    net.train_epoch(dev(X), dev(y))
    o = O.Oracle.from_workload(w)
    ids = sorted({0, K // 2, K - 1})
    ref = oracle_replicas(o, np.tile(th0.astype(np.float64), (len(ids), 1)), ids, X, y)
    for i, k in enumerate(ids):
        got = net.get_params(k)
        assert_close(w.sizes, got, ref[i], STEP_TOL, f"replica {k}")
        e = rel_err(w.sizes, got.astype(np.float64) - th0, ref[i] - th0)
        assert max(e.values()) <= 1e-3, e
    net.close()


@pytest.mark.parametrize("over,N", CHUNKED_CASES)
def test_chunked_plan_epoch(over, N):
    w = I.WORKLOADS[1].scaled(**over)
    K = w.replicas
    X, y = I.train_set(w, N)
    Xt, yt = I.test_set(w, 2000)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    assert net.plan == "per-sample chunked"
    log(f"chunked epoch: {w.name} {over} N={N}")
    net.train_epoch(dev(X), dev(y))
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    o.train_epoch(ref, X, y, threads=8)
    for k in range(K):
        close_epoch(w, net.get_params(k), ref[k], f"replica {k}")
    net.merge()
    close_epoch(w, net.get_params(-1), o.merge(ref), "merged")
    pred = torch.empty(len(yt), dtype=torch.int32, device="cuda")
    net.infer(dev(Xt), pred)
    predictions_agree(w, o, o.merge(ref), pred.cpu().numpy(), Xt)
    net.close()


# ------------------------------------------------------------------------------------
# the fp32 products on the fp32 matrix instructions (PNN_GEMM=fp32: gemm128_kernel for the
# forward, gemm_kernel for the update) instead of the split-bf16 kernels


@pytest.mark.parametrize("idx,over,N,epochs", [
    (4, dict(replicas=16), 16 * 260 + 7, 2),
    (2, dict(sizes=(784, 192, 10), replicas=4), 4 * 100 + 5, 1),
])
def test_epochs_fp32_matrix_path(idx, over, N, epochs, monkeypatch):
    monkeypatch.setenv("PNN_GEMM", "fp32")
    monkeypatch.setenv("PNN_MB_PLAN", "launch")
    w = I.WORKLOADS[idx].scaled(**over)
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    assert net.plan == "mini-batch"
    log(f"fp32 matrix path: {w.name} {over} N={N}")
    xd, yd = dev(X), dev(y)
    net.profile(True)
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    for e in range(epochs):
        net.train_epoch(xd, yd)
        o.train_epoch(ref, X, y, threads=8)
        for k in range(w.replicas):
            close_epoch(w, net.get_params(k), ref[k], f"epoch {e} replica {k}")
        if w.merge_every_epoch:
            net.merge(broadcast=True)
            ref[:] = o.merge(ref)[None, :]
    names = set(net.profile_read())
    assert names and not any(n.endswith("_x3") for n in names), names
    net.close()


PLAN_CASES = [
    # workload, overrides, plan chosen at init
    (1, {}, "per-sample persistent"),
    (1, dict(replicas=64), "per-sample persistent"),          # 3 launches of 21/21/22 CNs
    (1, dict(sizes=(784, 256, 10)), "per-sample chunked"),
    (2, {}, "mini-batch persistent"),                          # 16 CNs x 16 tiles of 16 neurons
    (2, dict(replicas=20), "mini-batch persistent"),          # 32-neuron tiles
    (2, dict(replicas=40), "mini-batch persistent"),          # 2 launches of 20 CNs
    (2, dict(sizes=(784, 1024, 10)), "mini-batch"),           # 64 tiles of 16 neurons per CN
    (2, dict(batch=33), "mini-batch"),
    (3, dict(replicas=8), "mini-batch"),                      # bf16, two hidden layers
    (4, dict(replicas=4), "mini-batch fused last layer"),
    (4, dict(sizes=(784, 256, 16), acts=(I.TANH, I.SOFTMAX), loss=I.LOSS_XENT), "mini-batch fused last layer"),
    (4, dict(sizes=(784, 192, 10)), "mini-batch"),            # hidden width below 256
    (4, dict(batch=64), "mini-batch"),                        # batch other than 128
]


@pytest.mark.parametrize("idx,over,plan", PLAN_CASES)
def test_plan_selection(idx, over, plan, monkeypatch):
    w = I.WORKLOADS[idx].scaled(**over)
    net = make_net(w, I.init_params(w))
    assert net.plan == plan
    net.close()
    monkeypatch.setenv("PNN_MB_PLAN", "launch")
    net = make_net(w, I.init_params(w))
    assert net.plan == ("mini-batch" if plan in ("mini-batch persistent", "mini-batch fused last layer") else plan)
    net.close()


@pytest.mark.parametrize("idx,over,N,epochs", [
    (2, {}, 16 * 100 + 5, 2),
    (2, dict(sizes=(784, 56, 10), acts=(I.SIGMOID, I.SIGMOID), batch=7, replicas=5), 5 * 40 + 3, 1),
    (4, dict(replicas=4), 4 * 224 + 2, 1),     # the separate last-layer kernel behind the split-bf16 products
])
def test_epochs_launch_plan(idx, over, N, epochs, monkeypatch):
    """The per-layer launch plan on nets that would otherwise get the persistent mini-batch
    kernel or the fused last layer, against the oracle."""
    monkeypatch.setenv("PNN_MB_PLAN", "launch")
    w = I.WORKLOADS[idx].scaled(**over)
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    assert net.plan == "mini-batch"
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    xd, yd = dev(X), dev(y)
    for e in range(epochs):
        net.train_epoch(xd, yd)
        o.train_epoch(ref, X, y, threads=8)
        for k in range(w.replicas):
            close_epoch(w, net.get_params(k), ref[k], f"epoch {e} replica {k}")
    net.close()


def test_deferred_broadcast():
    """Fused last layer with a merge and broadcast after each epoch, nothing read in between: the
    copy of the merged network into the CNs is left to the next epoch's first step, which reads
    the merged slot and writes every CN.  Every CN and the merged network against the oracle
    after each epoch; then a CN read, an evaluation of a CN and a second merge right after a
    deferred merge see the merged network (the copy made on demand)."""
    w = I.WORKLOADS[4].scaled(replicas=16)
    N = 16 * 260 + 7                  # batches 128, 128, 4/5
    X, y = I.train_set(w, N)
    Xt, yt = I.test_set(w, 500)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    assert net.plan == "mini-batch fused last layer"
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    xd, yd = dev(X), dev(y)
    for e in range(3):
        net.train_epoch(xd, yd)
        o.train_epoch(ref, X, y, threads=8)
        net.merge(broadcast=True)
        m = o.merge(ref)
        ref[:] = m[None, :]
    close_epoch(w, net.get_params(-1), m, "merged after three epochs")
    merged = net.get_params(-1)
    # a CN's evaluation first makes the deferred copy; then every CN holds the merged network
    c_cn = net.evaluate(dev(Xt), dev(yt), which=3)
    c_m = net.evaluate(dev(Xt), dev(yt), which=-1)
    assert c_cn == c_m
    for k in range(w.replicas):
        assert np.array_equal(net.get_params(k), merged), k
    # a merge of CNs that all hold the merged network gives it back exactly, with or without a
    # pending copy before it
    net.merge(broadcast=True)
    net.merge(broadcast=False)
    assert np.array_equal(net.get_params(-1), merged)
    assert np.array_equal(net.get_params(5), merged)
    # the allocation-free evaluation of a CN makes a pending copy too
    net.merge(broadcast=True)
    c7, cost7 = net.evaluate_noalloc(dev(Xt), dev(yt), which=7)
    assert c7 == c_m[0] and abs(cost7 - c_m[1]) <= 1e-12 * abs(c_m[1])
    # a weighted merge with broadcast defers the same way: one more epoch from it against the oracle
    wts = np.linspace(1.0, 2.0, w.replicas)
    net.merge_weighted(wts, broadcast=True)
    mw = o.merge_weighted(ref, wts)
    close_epoch(w, net.get_params(-1), mw, "weighted merge")
    net.train_epoch(xd, yd)
    ref[:] = mw[None, :]
    o.train_epoch(ref, X, y, threads=8)
    for k in (0, 9, w.replicas - 1):
        close_epoch(w, net.get_params(k), ref[k], f"epoch after a weighted merge, replica {k}")
    net.close()


def test_misaligned_input_rows_are_rejected():
    """x_dev must be 16-byte aligned (rows are read with 16-byte loads): a view one float into a
    buffer is refused by every call that reads rows, before any device work."""
    w = I.WORKLOADS[2].scaled(replicas=2)
    X, y = I.train_set(w, 2 * 40)
    net = make_net(w, I.init_params(w))
    xb = torch.zeros(X.size + 4, dtype=torch.float32, device="cuda")
    xv = xb[1:1 + X.size].view(X.shape)
    assert xv.data_ptr() % 16 == 4
    yd = dev(y)
    for call in (lambda: net.train_epoch(xv, yd),
                 lambda: net.train_epoch_order(xv, yd, dev(np.arange(len(y), dtype=np.int32))),
                 lambda: net.infer(xv, torch.empty(len(y), dtype=torch.int32, device="cuda")),
                 lambda: net.evaluate(xv, yd)):
        with pytest.raises(B.PnnError) as ei:
            call()
        assert ei.value.status == B.PNN_EINVAL and "aligned" in str(ei.value)
    net.train_epoch(dev(X), yd)  # the handle stays usable
    net.get_params(0)
    net.close()


ABORT_CASES = [
    # workload, overrides, plan, the first call after the failed launch
    (2, dict(replicas=4), "mini-batch persistent", "get_params"),
    (2, dict(replicas=4), "mini-batch persistent", "merge"),
    (1, dict(replicas=3), "per-sample persistent", "merge"),
    (1, dict(replicas=3), "per-sample persistent", "evaluate"),
    (1, dict(replicas=3), "per-sample persistent", "infer"),
    (1, dict(replicas=3), "per-sample persistent", "train_epoch"),
]


@pytest.mark.parametrize("idx,over,plan,first", ABORT_CASES)
def test_persistent_kernel_abort_path(idx, over, plan, first, monkeypatch):
    """Failure handling forced from the host: every wait of the persistent kernel runs into a small
    poll bound (the mini-batch kernel's readers wait for share tags that are never written, the
    per-sample kernel's sequential workgroups for more tiles than exist), the abort flag is raised
    and every workgroup ends.  The next call that consumes the CNs reports the time-out (PNN_EHIP)
    and the handle refuses all further work (PNN_ESTATE); a new handle on the same device then
    trains as the oracle does."""
    w = I.WORKLOADS[idx].scaled(**over)
    K = w.replicas
    N = K * (40 if w.batch > 1 else 70) + 3
    X, y = I.train_set(w, N)
    Xt, yt = I.test_set(w, 100)
    th0 = I.init_params(w)
    monkeypatch.setenv("PNN_SPIN_LIMIT", "2000")
    monkeypatch.setenv("PNN_TEST_STALL_WAITS", "1")
    log(f"abort path: {w.name} {over}, first call {first}")
    net = make_net(w, th0)
    assert net.plan == plan
    xd, yd, xtd, ytd = dev(X), dev(y), dev(Xt), dev(yt)
    net.train_epoch(xd, yd)
    calls = {
        "get_params": lambda: net.get_params(0),
        "merge": lambda: net.merge(),
        "evaluate": lambda: net.evaluate(xtd, ytd),
        "infer": lambda: net.infer(xtd, torch.empty(len(yt), dtype=torch.int32, device="cuda")),
        "train_epoch": lambda: net.train_epoch(xd, yd),
    }
    if first == "train_epoch":
        torch.cuda.synchronize()  # (pnn_train_epoch reads the flag once the failed launch has ended)
    with pytest.raises(B.PnnError) as ei:
        calls[first]()
    assert ei.value.status == B.PNN_EHIP and "timed out" in str(ei.value)
    for name, call in calls.items():
        with pytest.raises(B.PnnError) as ei:
            call()
        assert ei.value.status == B.PNN_ESTATE, name
    net.close()
    monkeypatch.delenv("PNN_TEST_STALL_WAITS")
    monkeypatch.delenv("PNN_SPIN_LIMIT")
    net = make_net(w, th0)
    net.train_epoch(xd, yd)
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    o.train_epoch(ref, X, y, threads=4)
    for k in range(K):
        close_epoch(w, net.get_params(k), ref[k], f"replica {k} after the aborted handle")
    net.close()


@pytest.mark.parametrize("over,N", [(dict(sizes=(784, 64, 10), acts=(1, 0), replicas=3), 302),
                                     (dict(replicas=2), 2 * 150 + 7),
                                     # 32-row tiles (40 CNs fit one launch with them)
                                     (dict(replicas=40), 40 * 70 + 3),
                                     # 16-row tiles, the CNs in three launches sharing the flags
                                     (dict(replicas=60), 60 * 70 + 3)])
def test_per_sample_tiles_out_of_order(over, N, monkeypatch):
    """Ordering forced from the host: the upper half of every CN's tile workgroups start a few
    milliseconds late, so that the others publish Q_0 and Q_1 (the input sums of the first two
    chunks) before they publish anything.  The sequential workgroup must still wait for every
    tile's share of each Q (one readiness counter per chunk parity).  Over two epochs both runs
    match the oracle at the epoch tolerance.  (They need not agree bit for bit: Q joins the next
    chunk's accumulated input sums as soon as it is complete, between folds whose number
    depends on timing.)  With a single counter the first rows would start from stale input
    sums, errors of order 0.1 and more."""
    w = I.WORKLOADS[1].scaled(**over)
    K = w.replicas
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    xd, yd = dev(X), dev(y)
    got = {}
    for delay in (0, 2000):
        if delay:
            monkeypatch.setenv("PNN_TEST_TILE_DELAY", str(delay))
        log(f"tiles out of order: {w.name} {over} N={N} delay {delay}")
        net = make_net(w, th0)
        assert net.plan == "per-sample persistent"
        for _ in range(2):
            net.train_epoch(xd, yd)
        got[delay] = [net.get_params(k) for k in range(K)]
        net.close()
    monkeypatch.delenv("PNN_TEST_TILE_DELAY")
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    for _ in range(2):
        o.train_epoch(ref, X, y, threads=4)
    for k in range(K):
        close_epoch(w, got[0][k], ref[k], f"replica {k}")
        close_epoch(w, got[2000][k], ref[k], f"replica {k}, late tiles")


def test_per_sample_many_cns_flag_reset():
    """More CNs than one workgroup of the flag-reset kernel covers (3 K counters > 256): every
    epoch starts with every CN's readiness counters at zero, so the second epoch matches the
    oracle too."""
    w = I.WORKLOADS[0].scaled(replicas=90)
    K = w.replicas
    N = K * 150 + 5  # three chunks of input sums per CN
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    log(f"many CNs, per-sample: {w.name} K={K} N={N}")
    net = make_net(w, th0)
    log(f"plan: {net.plan}")
    assert net.plan == "per-sample persistent"
    xd, yd = dev(X), dev(y)
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    for e in range(2):
        net.train_epoch(xd, yd)
        o.train_epoch(ref, X, y, threads=8)
        for k in (0, 1, K // 2, K - 2, K - 1):
            close_epoch(w, net.get_params(k), ref[k], f"epoch {e} replica {k}")
    net.close()


# ------------------------------------------------------------------------------------
# step-by-step trajectory: before every step the oracle restarts from the GPU's state

def step_rows(N, K, Bt, s):
    """Data rows of batch step s of every CN (an epoch over them is exactly that step)."""
    o = O.Oracle((8, 2), (O.SIGMOID,), O.LOSS_MSE, replicas=K)
    rows = []
    for k in range(K):
        st, ln = o.shard(N, k)
        rows.append(np.arange(st + s * Bt, st + min(ln, (s + 1) * Bt)))
    return rows


@pytest.mark.parametrize("idx,over,N", [
    (3, dict(replicas=8), 8 * 150 + 3),
    (4, dict(replicas=4), 4 * 300 + 3),
    (2, dict(replicas=4), 4 * 70 + 2),
])
def test_stepwise_trajectory(idx, over, N):
    w = I.WORKLOADS[idx].scaled(**over)
    K, Bt = w.replicas, w.batch
    log(f"trajectory: {w.name} {over} N={N}")
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    o = O.Oracle.from_workload(w)
    nsteps = -(-(-(-N // K)) // Bt)
    for s in range(nsteps):
        rows = step_rows(N, K, Bt, s)
        if min(len(r) for r in rows) == 0:
            break
        before = np.stack([net.get_params(k) for k in range(K)]).astype(np.float64)
        # one step of every CN: each CN gets exactly its own rows of this step
        idxs = np.concatenate(rows)
        if len(set(len(r) for r in rows)) == 1:
            net.train_epoch(dev(X[idxs]), dev(y[idxs]))
            for k in range(K):
                ref = before[k].copy()[None, :]
                one = O.Oracle.from_workload(w, replicas=1)
                one.train_epoch(ref, X[rows[k]], y[rows[k]])
                assert_close(w.sizes, net.get_params(k), ref[0], tol_for(w), f"step {s} replica {k}")
        else:
            break  # uneven last batches are covered by the epoch tests
    net.close()


# ------------------------------------------------------------------------------------
# full-size workloads in the launch configuration of the benchmark

def _full(w, ids_per_epoch, threads=16):
    K = w.replicas
    X, y = I.train_set(w)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    xd, yd = dev(X), dev(y)
    o = O.Oracle.from_workload(w)
    start = np.tile(th0.astype(np.float64), (K, 1)) if not w.merge_every_epoch else None
    state = {k: th0.astype(np.float64) for k in (ids_per_epoch if ids_per_epoch else range(K))}
    for e in range(w.epochs):
        log(f"full {w.name}: epoch {e}")
        if w.merge_every_epoch:
            begin = net.get_params(-1).astype(np.float64)
        net.train_epoch(xd, yd)
        torch.cuda.synchronize()
        ids = list(state.keys())
        starts = np.stack([begin if w.merge_every_epoch else state[k] for k in ids])
        ref = oracle_replicas(o, starts, ids, X, y, threads=threads)
        for i, k in enumerate(ids):
            state[k] = ref[i]
            close_epoch(w, net.get_params(k), ref[i], f"epoch {e} replica {k}")
        if w.merge_every_epoch:
            reps = np.stack([net.get_params(k) for k in range(K)]).astype(np.float64)
            net.merge(broadcast=True)
            m = net.get_params(-1)
            assert_close(w.sizes, m, o.merge(reps), 2e-7, f"merge epoch {e}")
    if not w.merge_every_epoch:
        reps = np.stack([net.get_params(k) for k in range(K)]).astype(np.float64)
        net.merge(broadcast=False)
        assert_close(w.sizes, net.get_params(-1), o.merge(reps), 2e-7, "merge")
    Xt, yt = I.test_set(w)
    pred = torch.empty(len(yt), dtype=torch.int32, device="cuda")
    correct = net.infer(dev(Xt), pred, y=dev(yt), count=True)
    out_ref = o.forward(net.get_params(-1).astype(np.float64), Xt)
    argmax_agrees(out_ref, pred.cpu().numpy(), margin=1e-5 if w.precision == I.FP32 else 2e-2)
    if not w.merge_every_epoch and len(state) == K:
        # every CN was trained by the oracle on its own from theta0: its merged network
        predictions_agree(w, o, o.merge(np.stack([state[k] for k in range(K)])), pred.cpu().numpy(), Xt)
    log(f"full {w.name}: merged accuracy {correct / len(yt):.4f}")
    # clearly above chance (10 classes); the workloads with few, small steps (the 256-CN one
    # takes 38 steps of eta = 0.02) are far from converged after their epochs
    assert correct / len(yt) > 0.2
    net.close()
    del start


def test_full_workload0():
    w = I.WORKLOADS[0]
    _full(w, [0], threads=1)


def test_full_workload1_all_replicas():
    w = I.WORKLOADS[1]
    _full(w, list(range(w.replicas)), threads=4)


def test_full_workload2_all_replicas():
    w = I.WORKLOADS[2]
    _full(w, list(range(w.replicas)))


def test_full_workload3_sampled():
    _full(I.WORKLOADS[3], [0, 9, 18, 27, 36, 45, 54, 63])


def test_full_workload4_sampled():
    # every sixteenth CN and both sides of the slice-length boundary (CNs 191 / 192)
    _full(I.WORKLOADS[4], sorted(set(range(0, 256, 16)) | {191, 192, 255}))


# ------------------------------------------------------------------------------------
# merge, inference and handle behaviour

def test_merge_identities():
    w = I.WORKLOADS[2].scaled(replicas=5)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    net.merge()
    assert np.array_equal(net.get_params(-1), th0)  # identical replicas: identity, bitwise
    P = th0.size
    for k in range(5):
        net.set_params(k, np.full(P, float(k), np.float32))
    net.merge(broadcast=False)
    assert np.all(net.get_params(-1) == 2.0)  # (K - 1) / 2 exactly
    assert np.all(net.get_params(3) == 3.0)
    rng = np.random.default_rng(3)
    reps = rng.standard_normal((5, P)).astype(np.float32)
    for k in range(5):
        net.set_params(k, reps[k])
    net.merge(broadcast=True)
    ref = reps.astype(np.float64).mean(axis=0)
    m = net.get_params(-1)
    assert np.max(np.abs(m - ref) / np.maximum(np.abs(ref), 1e-3)) <= 2e-7
    for k in range(5):
        assert np.array_equal(net.get_params(k), m)
    net.close()


def test_replica_inference_and_edges():
    w = I.WORKLOADS[1].scaled(replicas=2)
    X, y = I.train_set(w, 400)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    net.train_epoch(dev(X), dev(y))
    o = O.Oracle.from_workload(w)
    Xt, yt = I.test_set(w, 9000)  # crosses the 8192-row inference chunk
    for which in (0, 1, -1):
        pred = torch.empty(len(yt), dtype=torch.int32, device="cuda")
        c = net.infer(dev(Xt), pred, which=which, y=dev(yt), count=True)
        p = pred.cpu().numpy()
        argmax_agrees(o.forward(net.get_params(which).astype(np.float64), Xt), p)
        assert c == int((p == yt).sum())
    empty = torch.empty((0, 784), dtype=torch.float32, device="cuda")
    assert net.infer(empty, torch.empty(0, dtype=torch.int32, device="cuda"), y=dev(np.zeros(0, np.int32)),
                     count=True) == 0
    with pytest.raises(B.PnnError) as ei:
        net.infer(dev(Xt), pred, which=2)
    assert ei.value.status == B.PNN_EINVAL
    with pytest.raises(B.PnnError) as ei:
        net.train_epoch(dev(X[:1]), dev(y[:1]))  # N < K
    assert ei.value.status == B.PNN_ESHAPE
    net.close()


@pytest.mark.parametrize("idx", [1, 2, 3])
def test_zero_lr_and_determinism_and_resume(idx):
    w = I.WORKLOADS[idx].scaled(replicas=4)
    X, y = I.train_set(w, 4 * 3 * w.batch + 5)
    th0 = I.init_params(w)
    xd, yd = dev(X), dev(y)
    # eta = 0 leaves every parameter unchanged
    z = B.PNN(B.config_from_workload(w, lr=0.0), th0)
    z.train_epoch(xd, yd)
    assert np.array_equal(z.get_params(2), th0)
    z.close()
    # two runs are bitwise identical; a run resumed from a checkpoint equals the uninterrupted one
    runs = []
    for _ in range(2):
        n = make_net(w, th0)
        n.train_epoch(xd, yd)
        n.train_epoch(xd, yd)
        runs.append(np.stack([n.get_params(k) for k in range(4)]))
        n.close()
    assert np.array_equal(runs[0], runs[1])
    a = make_net(w, th0)
    a.train_epoch(xd, yd)
    ck = [a.get_params(k) for k in range(4)]
    a.close()
    b = make_net(w, np.zeros_like(th0))
    for k in range(4):
        b.set_params(k, ck[k])
    b.train_epoch(xd, yd)
    assert np.array_equal(np.stack([b.get_params(k) for k in range(4)]), runs[0])
    b.close()


# ------------------------------------------------------------------------------------
# evaluation of the merged network and of single CNs: correct count and mean cost


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4])
def test_eval_accuracy_and_cost(idx):
    w = I.WORKLOADS[idx].scaled(replicas=min(4, I.WORKLOADS[idx].replicas))
    K = w.replicas
    X, y = I.train_set(w, K * 3 * w.batch + 7)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    net.train_epoch(dev(X), dev(y))
    net.merge()
    o = O.Oracle.from_workload(w)
    Xt, yt = I.test_set(w, 9000 if idx == 1 else 1500)  # (9000 crosses the 8192-row inference chunk)
    bf = w.precision == I.BF16_MIXED
    for which in (-1, 0, K - 1):
        th = net.get_params(which).astype(np.float64)
        correct, cost = net.evaluate(dev(Xt), dev(yt), which=which)
        log(f"eval {w.name} which={which}: correct {correct}, cost {cost:.6f}")
        out = o.forward(th, Xt)
        ref_correct = int((np.argmax(out, axis=1) == yt).sum())
        srt = np.sort(out, axis=1)
        ties = int((srt[:, -1] - srt[:, -2] <= (1e-4 if bf else 1e-5)).sum())
        assert abs(correct - ref_correct) <= ties, (correct, ref_correct, ties)
        ref_cost = o.cost(th, Xt, yt)
        assert np.isfinite(cost)
        assert abs(cost - ref_cost) <= (1e-3 if bf else 1e-5) * abs(ref_cost), (cost, ref_cost)
        # the same rows through pnn_infer count the same
        pred = torch.empty(len(yt), dtype=torch.int32, device="cuda")
        assert net.infer(dev(Xt), pred, which=which, y=dev(yt), count=True) == correct
    empty_x = torch.empty((0, w.sizes[0]), dtype=torch.float32, device="cuda")
    assert net.evaluate(empty_x, dev(np.zeros(0, np.int32))) == (0, 0.0)
    with pytest.raises(B.PnnError) as ei:
        net.evaluate(dev(Xt), dev(yt), which=K)
    assert ei.value.status == B.PNN_EINVAL
    net.close()


# ------------------------------------------------------------------------------------
# nets whose training amplifies rounding differences to the size of the epoch bar (tanh hidden
# layer, sigmoid outputs with the cross-entropy error; tests/test_sensitivity.py): whole epochs
# normwise per layer, and every step elementwise with the oracle restarting from the GPU's state


@pytest.mark.parametrize("idx,over,N,epochs", SENSITIVE_FP32_CASES)
def test_sensitive_epochs_normwise(idx, over, N, epochs):
    w = I.WORKLOADS[idx].scaled(**over)
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    for e in range(epochs):
        net.train_epoch(dev(X), dev(y))
        o.train_epoch(ref, X, y, threads=8)
        for k in range(w.replicas):
            assert_close(w.sizes, net.get_params(k), ref[k], EPOCH_TOL, f"epoch {e} replica {k}", layerwise=True)
    net.close()



def test_per_sample_stepwise_tanh_xent():
    w = I.WORKLOADS[1].scaled(sizes=(784, 64, 10), acts=(I.TANH, I.SIGMOID), loss=I.LOSS_XENT, replicas=3)
    K, S = w.replicas, 24
    X, y = I.train_set(w, K * S)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    o = O.Oracle.from_workload(w)
    prev = np.tile(th0.astype(np.float64), (K, 1))
    for s in range(S):
        Xs, ys = X[s * K:(s + 1) * K], y[s * K:(s + 1) * K]  # one sample per CN
        net.train_epoch(dev(Xs), dev(ys))
        ref = oracle_replicas(o, prev, list(range(K)), Xs, ys)
        got = np.stack([net.get_params(k) for k in range(K)])
        for k in range(K):
            assert_close(w.sizes, got[k], ref[k], STEP_TOL, f"step {s} replica {k}")
        prev = got.astype(np.float64)
    net.close()



# ------------------------------------------------------------------------------------
# weighted combination


@pytest.mark.parametrize("idx", [2, 3])
def test_weighted_merge(idx):
    w = I.WORKLOADS[idx].scaled(replicas=4)
    K = w.replicas
    X, y = I.train_set(w, K * 2 * w.batch + 3)
    th0 = I.init_params(w)
    net = make_net(w, th0)
    net.train_epoch(dev(X), dev(y))
    cns = np.stack([net.get_params(k) for k in range(K)]).astype(np.float64)
    o = O.Oracle.from_workload(w)
    wts = np.array([0.5, 1.0, 2.0, 0.25])
    net.merge_weighted(wts)
    got = net.get_params(-1)
    ref = o.merge_weighted(cns, wts).astype(np.float32)
    np.testing.assert_allclose(got, ref, rtol=1.2e-7, atol=0)
    # the merged network's bf16 copy follows: its evaluation matches the oracle's on those weights
    Xt, yt = I.test_set(w, 1000)
    _, cost = net.evaluate(dev(Xt), dev(yt))
    ref_cost = o.cost(got.astype(np.float64), Xt, yt)
    assert abs(cost - ref_cost) <= (1e-3 if w.precision == I.BF16_MIXED else 1e-5) * abs(ref_cost)
    # equal weights: the plain average, bitwise
    net.merge()
    plain = net.get_params(-1)
    net.merge_weighted(np.full(K, 3.0))
    assert np.array_equal(net.get_params(-1), plain)
    # broadcast: every CN continues from the weighted mean
    net.merge_weighted(wts, broadcast=True)
    m = net.get_params(-1)
    for k in range(K):
        assert np.array_equal(net.get_params(k), m)
    for bad in ([-1.0, 1.0, 1.0, 1.0], [0.0, 0.0, 0.0, 0.0], [1.0, float("nan"), 1.0, 1.0]):
        with pytest.raises(B.PnnError) as ei:
            net.merge_weighted(np.array(bad))
        assert ei.value.status == B.PNN_EINVAL
    net.close()


# ------------------------------------------------------------------------------------
# epochs over a caller-given order (seeded per-epoch shuffling)


@pytest.mark.parametrize("idx,K", [(1, 3), (2, 4)])
def test_train_epoch_order(idx, K):
    w = I.WORKLOADS[idx].scaled(replicas=K)
    N = K * (70 if w.batch == 1 else 3 * w.batch) + 2
    X, y = I.train_set(w, N)
    th0 = I.init_params(w)
    a = make_net(w, th0)
    b = make_net(w, th0)
    o = O.Oracle.from_workload(w)
    ref = o.replicate(th0)
    xd, yd = dev(X), dev(y)
    for epoch in range(2):
        # a per-CN shuffle: each slice permuted within its own range, seeded per epoch
        rng = np.random.Generator(np.random.PCG64(1000 + epoch))
        order = np.concatenate([s + rng.permutation(n) for s, n in (o.shard(N, k) for k in range(K))]).astype(np.int32)
        a.train_epoch_order(xd, yd, dev(order))
        b.train_epoch(dev(X[order]), dev(y[order]))
        o.train_epoch(ref, X[order], y[order], threads=K)
    for k in range(K):
        assert np.array_equal(a.get_params(k), b.get_params(k))
        assert_close(w.sizes, a.get_params(k), ref[k], EPOCH_TOL, f"replica {k}")
    # entries outside [0, N) select row 0
    bad = np.arange(N, dtype=np.int32)
    bad[1], bad[N - 1] = -5, N + 3
    fix = bad.copy()
    fix[1] = fix[N - 1] = 0
    a.train_epoch_order(xd, yd, dev(bad))
    b.train_epoch(dev(X[fix]), dev(y[fix]))
    assert np.array_equal(a.get_params(0), b.get_params(0))
    a.close()
    b.close()
