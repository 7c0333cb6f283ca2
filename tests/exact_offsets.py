"""Exact-arithmetic filter offsets, independent of both the oracle and the kernels.

Used only by tests to pin the offset rule of Definition 1, Eq. (2):
    dh(k) = floor(-(k - pad) sin theta),   dw(k) = floor((k - pad) cos theta).

sin and cos are evaluated to 60 significant digits with Python's decimal
module (pi from Machin's formula, Taylor series after reduction to
[0, 45] degrees).  A product that agrees with an integer to 40 digits is that
integer exactly (for the angles used here the products are algebraic numbers
of low degree, which cannot lie that close to an integer without being one),
so the floor below is the exact-real-arithmetic floor.

The operation's documented reading of Eq. (2) treats a product that lies
within 1e-9 of an integer as that integer (angles given in float32 degrees can
sit a hair away from 0, 30, 90 ... degrees, where plain floating point cannot
decide the floor).  `exact_offsets(..., snap=True)` applies that reading to the
exact values; `snap=False` gives the pure real-arithmetic floor.
"""
from __future__ import annotations

from decimal import Decimal, localcontext

_PREC = 60


def _atan_inv(n: int) -> Decimal:
    # atan(1/n) = sum (-1)^i / ((2i+1) n^(2i+1))
    x = Decimal(1) / n
    x2 = x * x
    term = x
    total = Decimal(0)
    i = 0
    eps = Decimal(10) ** (-(_PREC + 5))
    while abs(term) > eps:
        total += term / (2 * i + 1) if i % 2 == 0 else -term / (2 * i + 1)
        term *= x2
        i += 1
    return total


def _pi() -> Decimal:
    with localcontext() as ctx:
        ctx.prec = _PREC + 10
        return 16 * _atan_inv(5) - 4 * _atan_inv(239)


def _sin_cos_rad(t: Decimal):
    s = Decimal(0)
    c = Decimal(0)
    term = Decimal(1)  # t^n / n!
    n = 0
    eps = Decimal(10) ** (-(_PREC + 5))
    while True:
        if n % 4 == 0:
            c += term
        elif n % 4 == 1:
            s += term
        elif n % 4 == 2:
            c -= term
        else:
            s -= term
        n += 1
        term = term * t / n
        if abs(term) < eps and n > 4:
            break
    return s, c


def sin_cos_deg(theta_deg) -> tuple[Decimal, Decimal]:
    """(sin, cos) of an angle in degrees; theta_deg may be a float (taken exactly) or a Decimal."""
    with localcontext() as ctx:
        ctx.prec = _PREC + 10
        d = Decimal(theta_deg) % 360
        if d < 0:
            d += 360
        # reduce to [0, 90) by quadrant, then to [0, 45] by complement
        quad = int(d // 90)
        r = d - 90 * quad
        pi = _pi()
        if r <= 45:
            s, c = _sin_cos_rad(r * pi / 180)
        else:
            c, s = _sin_cos_rad((90 - r) * pi / 180)
        for _ in range(quad):  # rotate by +90 degrees: (s, c) -> (c, -s)
            s, c = c, -s
        return +s, +c


SNAP = Decimal("1e-9")


def exact_floor(v: Decimal, snap: bool = True) -> int:
    with localcontext() as ctx:
        ctx.prec = _PREC + 10
        r = v.to_integral_value()
        if abs(v - r) < (SNAP if snap else Decimal(10) ** -40):
            return int(r)
        return int(v.to_integral_value(rounding="ROUND_FLOOR"))


def exact_offsets(theta_deg, K: int, pad: int | None = None, snap: bool = True):
    """Exact (dh, dw) lists for taps k = 0 .. K-1."""
    pad = K // 2 if pad is None else pad
    s, c = sin_cos_deg(theta_deg)
    dh, dw = [], []
    with localcontext() as ctx:
        ctx.prec = _PREC + 10
        for k in range(K):
            j = k - pad
            dh.append(exact_floor(-j * s, snap))
            dw.append(exact_floor(j * c, snap))
    return dh, dw


def min_distance_to_integer(theta_deg, K: int, pad: int | None = None) -> float:
    """Smallest non-zero distance of a product (k - pad) * sin/cos to an integer (conditioning aid)."""
    pad = K // 2 if pad is None else pad
    s, c = sin_cos_deg(theta_deg)
    best = 1.0
    for k in range(K):
        j = k - pad
        for v in (-j * s, j * c):
            d = abs(v - v.to_integral_value())
            if d > Decimal(10) ** -40:
                best = min(best, float(d))
    return best
