#!/usr/bin/env python3
"""Hand derivation of one bf16-mixed training step of a 2-2-2 net (sigmoid hidden layer, softmax
output with the cross-entropy error), written out scalar by scalar from the paper's equations
(section "Fundamentals": forward eq. (2)-(3) and (5), output error eq. (10), hidden error
eq. (11), updates eq. (12)-(13)) with the bf16 rounding points of the mixed-precision reading:
the input x, the weights used as operands (a bf16 copy of the fp32 master), the hidden
activation a1 and the errors d2 and d1 are rounded to bfloat16 (nearest, ties to even) where
they enter products; biases, the sigmoid and softmax arithmetic and the master update are exact.

Independent of the oracle and of the GPU library: exact rational arithmetic (fractions), the two
exponentials from Python's math.exp, and its own bf16 rounding (the rational value scaled to an
integer significand of 8 bits and rounded half to even).  Besides the values of that reading it
lists what the step gives when one rounding point is moved or dropped, so that a test can show
that each point changes the result.

Writes worked_2_2_2_sigmoid_softmax_bf16.json next to this file.
"""
import json
import math
import os
import struct
from fractions import Fraction as F


def f32(v: float) -> F:
    """The float32 value nearest to v (the inputs are stored in fp32), as an exact rational."""
    return F(struct.unpack("<f", struct.pack("<f", v))[0])


def bf16(q: F) -> F:
    """Round a rational to bfloat16: 8 significant bits, nearest, ties to even."""
    if q == 0:
        return q
    s = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if F(2) ** e > a:
        e -= 1
    # 2^e <= a < 2^(e+1): the significand a / 2^(e-7) lies in [128, 256)
    m = a / F(2) ** (e - 7)
    n = math.floor(m)
    r = m - n
    if r > F(1, 2) or (r == F(1, 2) and n % 2 == 1):
        n += 1
    return s * n * F(2) ** (e - 7)


def sigmoid(z: F) -> F:
    return F(1) / (F(1) + F(math.exp(-float(z))))


def step(x, W1, b1, W2, b2, label, lr, rx=True, rw=True, ra=True, rd2=True, rd1=True,
         d1_round_before_deriv=False, deriv_from_unrounded=False):
    """One per-sample step; the flags move or drop single rounding points (for the variants)."""
    R = lambda v, on: bf16(v) if on else v
    xb = [R(v, rx) for v in x]
    W1b = [[R(v, rw) for v in row] for row in W1]
    W2b = [[R(v, rw) for v in row] for row in W2]
    z1 = [W1b[k][0] * xb[0] + W1b[k][1] * xb[1] + b1[k] for k in range(2)]
    a1 = [sigmoid(z) for z in z1]
    a1b = [R(v, ra) for v in a1]
    z2 = [W2b[k][0] * a1b[0] + W2b[k][1] * a1b[1] + b2[k] for k in range(2)]
    m = max(z2)
    ex = [F(math.exp(float(z - m))) for z in z2]
    a2 = [v / (ex[0] + ex[1]) for v in ex]
    e = [F(1) if k == label else F(0) for k in range(2)]
    d2 = [a2[k] - e[k] for k in range(2)]
    d2b = [R(v, rd2) for v in d2]
    s = [W2b[0][j] * d2b[0] + W2b[1][j] * d2b[1] for j in range(2)]
    aa = a1 if deriv_from_unrounded else a1b
    deriv = [v * (1 - v) for v in aa]
    if d1_round_before_deriv:
        d1 = [R(s[j], rd1) * deriv[j] for j in range(2)]
        d1b = d1
    else:
        d1 = [s[j] * deriv[j] for j in range(2)]
        d1b = [R(v, rd1) for v in d1]
    W2n = [[W2[k][j] - lr * d2b[k] * a1b[j] for j in range(2)] for k in range(2)]
    b2n = [b2[k] - lr * d2b[k] for k in range(2)]
    W1n = [[W1[j][i] - lr * d1b[j] * xb[i] for i in range(2)] for j in range(2)]
    b1n = [b1[j] - lr * d1b[j] for j in range(2)]
    return dict(xb=xb, W1b=W1b, W2b=W2b, z1=z1, a1=a1, a1b=a1b, z2=z2, a2=a2, d2=d2, d2b=d2b, s=s, deriv=deriv,
                d1=d1, d1b=d1b, W1_new=W1n, b1_new=b1n, W2_new=W2n, b2_new=b2n)


def as_float(v):
    if isinstance(v, list):
        return [as_float(u) for u in v]
    return float(v)


def main():
    x = [f32(0.9), f32(0.3)]
    W1 = [[f32(0.1), f32(-0.2)], [f32(0.3), f32(0.4)]]
    b1 = [f32(0.13), f32(0.09)]
    W2 = [[f32(0.5), f32(-0.6)], [f32(-0.3), f32(0.8)]]
    b2 = [f32(0.2), f32(-0.1)]
    label, lr = 0, F(1, 2)
    ref = step(x, W1, b1, W2, b2, label, lr)
    variants = {
        "x_not_rounded": dict(rx=False),
        "weights_not_rounded": dict(rw=False),
        "a1_not_rounded": dict(ra=False),
        "d2_not_rounded": dict(rd2=False),
        "d1_not_rounded": dict(rd1=False),
        "d1_rounded_before_deriv": dict(d1_round_before_deriv=True),
        "deriv_from_unrounded_a1": dict(deriv_from_unrounded=True),
    }
    out = {
        "source": "Hand-derived (tests/golden/derive_bf16_step.py: exact rationals, math.exp, its own "
                  "bf16 rounding) from eq. (2)-(3), (5), (10), (11), (12)-(13) of section Fundamentals, "
                  "with the bf16-mixed rounding points: x, the operand copy of the weights, a1, d2 and d1 "
                  "rounded to bfloat16 (nearest even) where they enter products; d1 = round(s * a1b (1 - a1b)) "
                  "with s = W2b^T d2b; biases, activations, softmax and the master update exact. "
                  "Inputs are the float32 values nearest to the decimals 0.9, 0.3, 0.1, ...",
        "sizes": [2, 2, 2],
        "acts": ["sigmoid", "softmax"],
        "loss": "xent",
        "precision": "bf16_mixed",
        "x": as_float(x), "label": label, "lr": float(lr),
        "W1": as_float(W1), "b1": as_float(b1), "W2": as_float(W2), "b2": as_float(b2),
    }
    for k, v in ref.items():
        out[k] = as_float(v)
    out["variants"] = {}
    for name, flags in variants.items():
        r = step(x, W1, b1, W2, b2, label, lr, **flags)
        out["variants"][name] = {k: as_float(r[k]) for k in ("W1_new", "b1_new", "W2_new", "b2_new")}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "worked_2_2_2_sigmoid_softmax_bf16.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(path)


if __name__ == "__main__":
    main()
