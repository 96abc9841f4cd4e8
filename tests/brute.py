"""Pure-Python brute force used to pin the CPU oracle on tiny inputs.

Nothing here shares code with the oracle: elements are decoded with
``struct`` (IEEE binary16), the sign of each element-wise product is read off
the IEEE product itself (its sign is the XOR of the operand signs, zeros
included), the Eq. (2) decision is taken in exact rational arithmetic, and the
gated MLP of Eq. (1) is summed element by element in exact rationals.
"""

from __future__ import annotations

import math
import struct
from fractions import Fraction

import numpy as np


def f16(bits: int) -> float:
    """Value of an IEEE binary16 bit pattern."""
    return struct.unpack("<e", struct.pack("<H", int(bits) & 0xFFFF))[0]


def product_is_negative(wb: int, xb: int) -> bool:
    """Sign of the IEEE product ``w * x`` (finite operands)."""
    return math.copysign(1.0, f16(wb) * f16(xb)) < 0


def n_neg(w_row, x_row) -> int:
    """Number of element-wise products with a negative sign."""
    return sum(1 for wb, xb in zip(w_row, x_row) if product_is_negative(wb, xb))


def alpha_value(alpha) -> Fraction | None:
    """Exact value of the float32 ``alpha`` the library receives (None = +inf)."""
    a = float(np.float32(alpha))
    if math.isinf(a):
        return None
    return Fraction(a)


def predicted_active(nneg: int, d: int, alpha) -> bool:
    """Eq. (2) with the inequality taken literally: the row is sparse iff
    ``alpha * N_pos < N_neg``; the row is kept otherwise."""
    a = alpha_value(alpha)
    if a is None:
        return True
    return not (a * (d - nneg) < nneg)


def predict(w_gate, x, alpha):
    """``(mask, active[b][k])`` for lists of bit patterns ``w_gate[k][d]`` and
    ``x[b][d]``."""
    d = len(x[0])
    act = [[predicted_active(n_neg(row, xt), d, alpha) for row in w_gate] for xt in x]
    mask = [int(any(act[t][i] for t in range(len(x)))) for i in range(len(w_gate))]
    return mask, act


def mlp(w_gate, w_up, w_down, x, mask):
    """Exact Eq. (1) over the kept rows.  ``w_down`` is ``[d][k]``.
    Returns ``(y[b][d], g[b][k], h3[b][k])`` as Fractions (g, h3 are 0 on
    dropped rows)."""
    k, d = len(w_gate), len(w_gate[0])
    ys, gs, hs = [], [], []
    for xt in x:
        X = [Fraction(f16(v)) for v in xt]
        g_t = [Fraction(0)] * k
        h3_t = [Fraction(0)] * k
        for i in range(k):
            if not mask[i]:
                continue
            g = sum((Fraction(f16(w_gate[i][j])) * X[j] for j in range(d)), Fraction(0))
            u = sum((Fraction(f16(w_up[i][j])) * X[j] for j in range(d)), Fraction(0))
            g_t[i] = g
            h3_t[i] = max(g, Fraction(0)) * u
        y_t = [sum((h3_t[i] * Fraction(f16(w_down[c][i])) for i in range(k)), Fraction(0))
               for c in range(d)]
        ys.append(y_t); gs.append(g_t); hs.append(h3_t)
    return ys, gs, hs


def relu_mlp(w_fc1, w_down, x, mask):
    """Exact non-gated ReLU MLP over the kept rows (``w_down`` is
    ``[d][k]``).  Returns ``(y[b][d], h[b][k])`` as Fractions."""
    k, d = len(w_fc1), len(w_fc1[0])
    ys, hs = [], []
    for xt in x:
        X = [Fraction(f16(v)) for v in xt]
        h_t = [Fraction(0)] * k
        for i in range(k):
            if mask[i]:
                g = sum((Fraction(f16(w_fc1[i][j])) * X[j] for j in range(d)), Fraction(0))
                h_t[i] = max(g, Fraction(0))
        ys.append([sum((h_t[i] * Fraction(f16(w_down[c][i])) for i in range(k)), Fraction(0))
                   for c in range(d)])
        hs.append(h_t)
    return ys, hs


def gate_positive(w_gate, x):
    """Exact ``X . W_gate,i > 0`` for every token and row."""
    out = []
    for xt in x:
        X = [Fraction(f16(v)) for v in xt]
        out.append([sum((Fraction(f16(w)) * X[j] for j, w in enumerate(row)), Fraction(0)) > 0
                    for row in w_gate])
    return out


def fp16_bits(value: float) -> int:
    """Bit pattern of the fp16 nearest to ``value``."""
    return struct.unpack("<H", struct.pack("<e", value))[0]


def decode_fp16_by_fields(bits: int) -> float:
    """Binary16 decoded from its fields (sign, 5-bit exponent, 10-bit
    fraction); NaN/Inf patterns return None."""
    s = (bits >> 15) & 1
    e = (bits >> 10) & 0x1F
    f = bits & 0x3FF
    if e == 0x1F:
        return None
    if e == 0:
        v = f * 2.0 ** -24
    else:
        v = (1024 + f) * 2.0 ** (e - 25)
    return -v if s else v
