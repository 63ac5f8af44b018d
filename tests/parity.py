"""Helpers of the GPU parity tests: run the library through its C ABI and the oracle on the
same seeded inputs, and compare.

Tolerance (the per-weight relative error): for every weight and bias tensor t,
    err(t) = max_i |gpu_i - ref_i| / max(|ref_i|, rms(ref_t))
The rms floor keeps near-zero entries (biases start at 0) from turning rounding noise into
large relative errors.  Bars: 1e-5 after one training step and 1e-3 after full epochs in
fp32; 2e-2 per step in bf16-mixed precision.

Where the method amplifies rounding differences to the size of a bar, that bar would measure
the amplification rather than the implementation; tests/test_sensitivity.py measures, for every
parity case, how far the oracle moves from its own run when its start moves by one fp32 ulp.
Where that reaches half a bar for some tensor (bf16-mixed training over several steps; fp32
nets with a tanh hidden layer under sigmoid outputs with the cross-entropy error), whole epochs
are compared normwise per layer, W_l and b_l together:
    err(l) = ||gpu_l - ref_l||_2 / ||ref_l||_2,
the tensors that stay below half the bar elementwise (tests/cases.py) are still compared
elementwise, and every single step of those nets is held elementwise by tests that restart the
oracle from the GPU's state before each step.
"""
from __future__ import annotations

import os
import sys
import threading
from typing import Dict, List, Sequence

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import pnn_inputs as I  # noqa: E402
from oracle import oracle as O  # noqa: E402

STEP_TOL = 1e-5
EPOCH_TOL = 1e-3
BF16_TOL = 2e-2


def log(msg: str) -> None:
    print(msg, flush=True)


def split(sizes: Sequence[int], theta: np.ndarray):
    out, o = [], 0
    for l in range(len(sizes) - 1):
        nw = sizes[l + 1] * sizes[l]
        out.append((f"W{l + 1}", theta[o:o + nw]))
        o += nw
        out.append((f"b{l + 1}", theta[o:o + sizes[l + 1]]))
        o += sizes[l + 1]
    return out


def rel_err(sizes, got: np.ndarray, ref: np.ndarray) -> Dict[str, float]:
    res = {}
    for (name, g), (_, r) in zip(split(sizes, np.asarray(got, np.float64)), split(sizes, np.asarray(ref, np.float64))):
        floor = max(float(np.sqrt(np.mean(r * r))), 1e-30)
        res[name] = float(np.max(np.abs(g - r) / np.maximum(np.abs(r), floor)))
    return res


def layer_err(sizes, got: np.ndarray, ref: np.ndarray) -> Dict[str, float]:
    g = split(sizes, np.asarray(got, np.float64))
    r = split(sizes, np.asarray(ref, np.float64))
    res = {}
    for l in range(len(sizes) - 1):
        gl = np.concatenate([g[2 * l][1], g[2 * l + 1][1]])
        rl = np.concatenate([r[2 * l][1], r[2 * l + 1][1]])
        res[f"layer{l + 1}"] = float(np.linalg.norm(gl - rl) / max(np.linalg.norm(rl), 1e-30))
    return res


def assert_close(sizes, got, ref, tol, what="", layerwise=False):
    e = layer_err(sizes, got, ref) if layerwise else rel_err(sizes, got, ref)
    worst = max(e.values())
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU parameters"
    assert worst <= tol, f"{what}: relative error {e} exceeds {tol}"
    return worst


def oracle_replicas(o: O.Oracle, thetas: np.ndarray, ids: Sequence[int], X, y, threads: int = 8) -> np.ndarray:
    """Train the listed CNs for one epoch (thetas[i] is the start of CN ids[i]), in threads."""
    thetas = np.ascontiguousarray(thetas, dtype=np.float64).copy()
    groups: List[List[int]] = [[] for _ in range(max(1, min(threads, len(ids))))]
    for i in range(len(ids)):
        groups[i % len(groups)].append(i)

    def work(g):
        sub = thetas[g].copy()
        o.train_replicas(sub, [ids[i] for i in g], X, y)
        thetas[g] = sub

    ts = [threading.Thread(target=work, args=(g,)) for g in groups if g]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    return thetas


def argmax_agrees(out_ref: np.ndarray, pred_gpu: np.ndarray, margin: float = 1e-5):
    """GPU predictions equal the oracle's argmax except where the oracle's top two outputs are
    within `margin` (then either of the tied classes is accepted).  With a single output the
    prediction is that output's index, 0."""
    if out_ref.shape[1] < 2:
        assert (pred_gpu == 0).all(), "a single-output network predicts class 0"
        return 0
    top = np.argmax(out_ref, axis=1)
    srt = np.sort(out_ref, axis=1)
    gap = srt[:, -1] - srt[:, -2]
    diff = pred_gpu != top
    if not diff.any():
        return 0
    idx = np.nonzero(diff)[0]
    ok = (gap[idx] <= margin) & (out_ref[idx, pred_gpu[idx]] >= srt[idx, -1] - margin)
    assert ok.all(), f"{(~ok).sum()} predictions differ from the oracle outside ties (rows {idx[~ok][:10]})"
    return len(idx)
