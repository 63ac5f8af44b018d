"""Host-side checks of bench.py's pricing of the kernels (CPU only).

The per-launch work that bench.py divides by measured kernel times must add up to the
method's own operation count: the matrix kernels of a mini-batch step together perform the
multiply-adds of the forward pass, the hidden errors and the weight gradients (eq. (2), (11),
(12)) of every sample once per epoch, and the per-sample kernel is priced at one read and
one write of every parameter plus the input row per step.
"""
import pytest

import bench
import pnn_inputs as I

MINIBATCH = [i for i, w in enumerate(I.WORKLOADS) if w.batch > 1]


def test_per_sample_effective_bytes():
    w = I.WORKLOADS[1]
    f, b = bench.kernel_work(w, "psgd_persistent", 1, w.n_train, 1)
    assert b == w.n_train * (8.0 * w.param_count() + 4.0 * w.sizes[0])
    assert f == w.n_train * bench.method_flops_per_sample(w)


@pytest.mark.parametrize("idx", MINIBATCH)
def test_minibatch_kernels_cover_the_method(idx):
    w = I.WORKLOADS[idx]
    s, N, E = w.sizes, w.n_train, w.epochs
    total = 0.0
    for name in ("fwd_gemm", "bwd_gemm", "upd_gemm", "tail"):
        f, _ = bench.kernel_work(w, name, 1, N, E)
        total += f
    weights = sum(s[l] * s[l + 1] for l in range(len(s) - 1))
    behind = sum(s[l] * s[l + 1] for l in range(1, len(s) - 1))
    assert total == pytest.approx(N * E * (4.0 * weights + 2.0 * behind), rel=1e-12)


@pytest.mark.parametrize("idx", MINIBATCH)
def test_minibatch_bytes_cover_every_weight_pass(idx):
    # each batch step of each CN reads every operand weight at least once and rewrites the
    # fp32 master of every weight
    w = I.WORKLOADS[idx]
    s, K = w.sizes, w.replicas
    bsteps = -(-(-(-w.n_train // K)) // w.batch) * w.epochs
    total = sum(bench.kernel_work(w, n, 1, w.n_train, w.epochs)[1] for n in ("fwd_gemm", "bwd_gemm", "upd_gemm", "tail"))
    weights = sum(s[l] * s[l + 1] for l in range(len(s) - 1))
    assert total >= K * bsteps * weights * 8.0


def test_fused_last_layer_kernels_cover_the_method():
    # plan "mini-batch fused last layer" (784-1024-10, K = 256, B = 128): the forward, out_err and
    # update kernels together carry the last layer's multiply-adds that the separate kernel
    # would (the output errors' own flops aside), and its weight and activation passes
    w = I.WORKLOADS[4]
    s, K, N, E = w.sizes, w.replicas, w.n_train, w.epochs
    fused = sum(bench.kernel_work(w, n, 1, N, E, True)[0] for n in ("fwd_gemm", "upd_gemm"))
    plain = sum(bench.kernel_work(w, n, 1, N, E)[0] for n in ("fwd_gemm", "bwd_gemm", "upd_gemm", "tail"))
    assert fused == pytest.approx(plain, rel=1e-12)
    bsteps = -(-(-(-N // K)) // w.batch) * E
    b = sum(bench.kernel_work(w, n, 1, N, E, True)[1] for n in ("fwd_gemm", "out_err", "upd_gemm"))
    weights = sum(s[l] * s[l + 1] for l in range(len(s) - 1))
    assert b >= K * bsteps * weights * 8.0
    assert bench.kernel_work(w, "out_err", 1, N, E)[0] == N * E * s[-1]


def test_persistent_minibatch_effective_bytes():
    # one launch = one epoch: every batch step of every CN would read and write every parameter
    # once in a streaming implementation, and every input row is read once
    w = I.WORKLOADS[2]
    K, N = w.replicas, w.n_train
    bsteps = -(-(-(-N // K)) // w.batch)
    f, b = bench.kernel_work(w, "mb_persistent", 1, N, w.epochs)
    assert b == K * bsteps * 8.0 * w.param_count() + N * 4.0 * w.sizes[0]
    assert f == N * bench.method_flops_per_sample(w)
    # the ragged last batch counts as a step: 3750 rows per CN in batches of 32
    assert bsteps == 118
    # below the fp32 ridge (19.7 flop/B): bench.py prices it against HBM
    assert f / b < 19.7


def test_unpriced_kernels():
    w = I.WORKLOADS[2]
    assert bench.kernel_work(w, "fwd_reduce", 1, w.n_train, 1) is None


def test_more_than_one_gpu_is_refused():
    # one GPU only: bench.py --gpus N with N > 1 exits with a message before touching a device
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_merge_bytes_follow_the_deferred_broadcast():
    """The merge writes the K copies of the merged network itself except with the last layer
    fused, where the next epoch's first step writes them (the copy made on demand is priced as
    the broadcast)."""
    w = I.WORKLOADS[4]
    K, P = w.replicas, w.param_count()
    assert w.merge_every_epoch
    _, b_plain = bench.kernel_work(w, "merge", 1, w.n_train, 1, False)
    _, b_fused = bench.kernel_work(w, "merge", 1, w.n_train, 1, True)
    assert b_plain == (2 * K * P + P) * 4.0
    assert b_fused == (K * P + P) * 4.0
    assert bench.kernel_work(w, "broadcast", 1, w.n_train, 1, True)[1] == (K * P + P) * 4.0
