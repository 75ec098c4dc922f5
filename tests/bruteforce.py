"""Exact reference arithmetic for pinning the oracle on tiny inputs.

Python integers and fractions.Fraction only: no fixed-width integers, no
shifts and no floating point after the scale derivation, so a wrong sign,
a dropped term or an off-by-one in the oracle's int64 code shows up here.
"""
from fractions import Fraction
import math


def floor_half_up(x: Fraction) -> int:
    """Nearest integer, ties toward +infinity."""
    return math.floor(x + Fraction(1, 2))


def requant_exact(c: int, M0: int, sh: int) -> int:
    """c * M0 / 2^sh rounded half up, as an exact rational."""
    if sh >= 1:
        return floor_half_up(Fraction(c * M0, 2 ** sh))
    return c * M0 * 2 ** (-sh)


def sat(v: int, bits: int) -> int:
    lo, hi = -(2 ** (bits - 1)), 2 ** (bits - 1) - 1
    return max(lo, min(hi, v))


def qlinear_exact(A, W, zp_a, bias_q, M0, sh, zp_y, out_bits, zp_w=None):
    """Y from nested lists: A [M][K], W [N][K], per-column bias_q/M0/sh and
    optional per-column weight zero-points zp_w."""
    M, N = len(A), len(W)
    Y = [[0] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            zw = 0 if zp_w is None else zp_w[n]
            c = sum((A[m][k] - zp_a) * (W[n][k] - zw) for k in range(len(A[m])))
            c = sat(c + bias_q[n], 32)
            r = requant_exact(c, M0[n], sh[n])
            Y[m][n] = sat(r + zp_y, out_bits)
    return Y
