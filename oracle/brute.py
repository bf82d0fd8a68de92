"""Pure-Python brute-force twin of the oracle, for tiny inputs.

TEST INFRASTRUCTURE ONLY (see ``oracle/ternary.py``).  No numpy: plain
loops over Python lists, ``math.fsum`` for exact sums, ``fractions.Fraction``
for exact comparisons and ``struct`` for float32 rounding.  It re-derives each
step of the quantizer of Sec. 3.1 in a different formulation from the
vectorized oracle, so agreement between the two pins both:

* the scale is the exactly rounded mean absolute value of the group, rounded
  once more to float32;
* the code is zero exactly when the float32 quotient |w| / (s + eps) rounds to
  at most one half.  Round-to-nearest-even of a real quotient v gives a float32
  <= 1/2 iff v <= 1/2 + 2**-25 (the midpoint between 1/2 and the next float32,
  1/2 + 2**-24, rounds to the even 1/2).  Half-to-even rounding then sends
  1/2 to 0 and everything in (1/2, 1] to 1, so the code is
  sign(w) * [|w| > (s + eps) * (1/2 + 2**-25)], evaluated exactly with
  rationals.  A zero divisor (all-zero group at eps = 0) gives +-inf -> +-1
  for non-zero w and 0 for w = 0.
"""

from __future__ import annotations

import math
import struct
from fractions import Fraction

_HALF_PLUS = Fraction(1, 2) + Fraction(1, 2 ** 25)


def f32(x: float) -> float:
    """Round a Python float to the nearest float32 (ties to even)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def scales(W, g):
    """Per-row, per-group float32 scales: fl32(fsum|w| / g)."""
    out = []
    for row in W:
        K = len(row)
        assert K % g == 0
        out.append([f32(math.fsum(abs(f32(w)) for w in row[j:j + g]) / g)
                    for j in range(0, K, g)])
    return out


def codes(W, s32, g, eps):
    """Codes in {-1, 0, 1} by the exact threshold formulation above."""
    eps32 = f32(eps)
    out = []
    for row, srow in zip(W, s32):
        qrow = []
        for k, w in enumerate(row):
            w = f32(w)
            d = f32(srow[k // g] + eps32)
            if w == 0.0:
                qrow.append(0)
            elif d == 0.0:
                qrow.append(1 if w > 0 else -1)
            elif Fraction(abs(w)) > Fraction(d) * _HALF_PLUS:
                qrow.append(1 if w > 0 else -1)
            else:
                qrow.append(0)
        out.append(qrow)
    return out


def pack_row(qrow):
    """One row of codes -> list of bytes, element by element from the format:
    element e of word w sits at bit 2*(e//2) + 16*(e%2), two's complement."""
    K = len(qrow)
    assert K % 16 == 0
    out = []
    for w0 in range(0, K, 16):
        word = 0
        for e in range(16):
            two_bit = {0: 0, 1: 1, -1: 3}[qrow[w0 + e]]
            word |= two_bit << (2 * (e // 2) + 16 * (e % 2))
        out.extend(word.to_bytes(4, "little"))
    return out


def gemm(X, q, s, g):
    """Y[m][n] = sum_k X[m][k] * s[n][k//g] * q[n][k], exact-rounded fsum."""
    return [[math.fsum(X[m][k] * s[n][k // g] * q[n][k] for k in range(len(X[m])))
             for n in range(len(q))] for m in range(len(X))]


def gemm_dx(dY, q, s, g):
    """dX[m][k] = sum_n dY[m][n] * s[n][k//g] * q[n][k]."""
    N, K = len(q), len(q[0])
    return [[math.fsum(dY[m][n] * s[n][k // g] * q[n][k] for n in range(N))
             for k in range(K)] for m in range(len(dY))]


def gemm_dw(dY, X):
    """dW[n][k] = sum_m dY[m][n] * X[m][k]."""
    M, N, K = len(dY), len(dY[0]), len(X[0])
    return [[math.fsum(dY[m][n] * X[m][k] for m in range(M)) for k in range(K)]
            for n in range(N)]


def codes_thresh(W, s32, g, eps, row_mult):
    """Codes with a per-row threshold multiplier m: the divisor is
    fl32(fl32(m * s) + eps), decided by the same exact comparison as `codes`."""
    tau = [[f32(f32(m) * s) for s in srow] for srow, m in zip(s32, row_mult)]
    return codes(W, tau, g, eps)


def group_code_dot(q, d, g):
    """sum of q * d over each group, exactly (Fractions), returned as floats."""
    out = []
    for qrow, drow in zip(q, d):
        out.append([float(sum(Fraction(int(qq)) * Fraction(dd)
                              for qq, dd in zip(qrow[j:j + g], drow[j:j + g])))
                    for j in range(0, len(qrow), g)])
    return out


def f16(x):
    """Round a real number (float or Fraction) to IEEE binary16, ties to even,
    from the format's definition: 11 significant bits, exponents down to -14
    with subnormals spaced 2**-24 below that, largest finite 65504, and
    everything from 65520 (the midpoint to 2**16) up rounding to infinity."""
    a = abs(Fraction(x))
    neg = x < 0
    if a == 0:
        return -0.0 if neg else 0.0
    if a >= 65520:
        return float("-inf") if neg else float("inf")
    e = a.numerator.bit_length() - a.denominator.bit_length()  # floor(log2 a) or one above
    if Fraction(2) ** e > a:
        e -= 1
    e = max(e, -14)
    spacing = Fraction(2) ** (e - 10)
    m = a / spacing
    r = math.floor(m)
    if m - r > Fraction(1, 2) or (m - r == Fraction(1, 2) and r % 2 == 1):
        r += 1
    v = float(r * spacing)
    return -v if neg else v


def gemv(x, q, s16, g):
    """y[b][n] = sum_k x[b][k] * s16[n][k//g] * q[n][k] (decode product with
    float16 scales given as their values), exact-rounded fsum."""
    return [[math.fsum(xb[k] * s16[n][k // g] * q[n][k] for k in range(len(xb)))
             for n in range(len(q))] for xb in x]


def dense_gemv(x, W):
    """y[b][n] = sum_k x[b][k] * W[n][k], exact-rounded fsum (float values)."""
    return [[math.fsum(xb[k] * W[n][k] for k in range(len(xb))) for n in range(len(W))]
            for xb in x]


def mixer_step(zxbcdt, conv_state, ssm_state, conv_w, conv_b, dt_bias, A_log, D, norm_w,
               eps, headdim, d_state):
    """One Mamba-2 mixer decode step in plain loops over lists (a second
    formulation of ``oracle/mamba.py``): per token, the convolution window of
    each channel, the per-head decay and input terms, the per-element state
    recurrence, the readout, the gate and the root-mean-square scale."""
    nheads = len(A_log)
    d_inner = nheads * headdim
    conv_dim = d_inner + 2 * d_state
    sp = lambda v: v if v > 20 else math.log1p(math.exp(v))
    si = lambda v: v / (1.0 + math.exp(-v))
    outs, conv_new, ssm_new = [], [], []
    for b, row in enumerate(zxbcdt):
        z = row[:d_inner]
        xbc = row[d_inner:d_inner + conv_dim]
        dt = row[d_inner + conv_dim:]
        u, cs = [], []
        for c in range(conv_dim):
            win = list(conv_state[b][c][1:]) + [xbc[c]]
            cs.append(win)
            u.append(si(math.fsum(win[t] * conv_w[c][t] for t in range(len(win))) + conv_b[c]))
        conv_new.append(cs)
        Bv, Cv = u[d_inner:d_inner + d_state], u[d_inner + d_state:]
        y, st_b = [], []
        for h in range(nheads):
            d = sp(dt[h] + dt_bias[h])
            a = math.exp(-d * math.exp(A_log[h]))
            st_h = []
            for p in range(headdim):
                xv = u[h * headdim + p]
                new = [a * ssm_state[b][h][p][n] + d * xv * Bv[n] for n in range(d_state)]
                st_h.append(new)
                y.append(math.fsum(new[n] * Cv[n] for n in range(d_state)) + D[h] * xv)
            st_b.append(st_h)
        ssm_new.append(st_b)
        g = [y[i] * si(z[i]) for i in range(d_inner)]
        r = 1.0 / math.sqrt(math.fsum(v * v for v in g) / d_inner + eps)
        outs.append([g[i] * r * norm_w[i] for i in range(d_inner)])
    return outs, conv_new, ssm_new
