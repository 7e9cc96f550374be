"""Interval arithmetic that encloses fp32 evaluation (a test helper).

An ``Iv`` holds arrays of lower and upper bounds (float64).  Each operation
forms the exact real range of the operation over its input intervals (the
endpoint arithmetic runs in float64 and is widened outwards by one float64 ulp
per operation, so the range is enclosed), then encloses its rounding to fp32:
round-to-nearest-even is monotone, so every fp32 result of a point inside the
inputs lies in [round-down-to-fp32(lo), round-up-to-fp32(hi)].  ``fma`` is the
exact product-sum rounded once, as fmaf.  Division requires a denominator
interval that excludes zero.  Evaluating a function's fp32 operation sequence
on intervals therefore encloses every value the fp32 function takes on the
input box (dependencies between operands are ignored, which only widens)."""
from __future__ import annotations

import numpy as np

F32 = np.float32
_INF = np.inf


def _down64(x):
    return np.nextafter(x, -_INF)


def _up64(x):
    return np.nextafter(x, _INF)


def _round_down32(x):
    """Largest fp32 value <= x (elementwise, x float64)."""
    x = np.atleast_1d(np.asarray(x, dtype=np.float64))
    f = x.astype(np.float32).astype(np.float64)
    over = f > x
    f[over] = np.nextafter(f[over].astype(np.float32), np.float32(-np.inf)).astype(np.float64)
    return f


def _round_up32(x):
    x = np.atleast_1d(np.asarray(x, dtype=np.float64))
    f = x.astype(np.float32).astype(np.float64)
    under = f < x
    f[under] = np.nextafter(f[under].astype(np.float32), np.float32(np.inf)).astype(np.float64)
    return f


class Iv:
    __slots__ = ("lo", "hi")

    def __init__(self, lo, hi=None):
        lo = np.asarray(lo, dtype=np.float64)
        hi = lo if hi is None else np.asarray(hi, dtype=np.float64)
        self.lo, self.hi = np.broadcast_arrays(lo, hi)
        self.lo, self.hi = self.lo.copy(), self.hi.copy()

    @staticmethod
    def f32(lo, hi):
        """fp32 enclosure of the real range [lo, hi]."""
        return Iv(_round_down32(_down64(lo)), _round_up32(_up64(hi)))

    def __neg__(self):
        return Iv(-self.hi, -self.lo)

    def __add__(self, o):
        o = _iv(o)
        return Iv.f32(self.lo + o.lo, self.hi + o.hi)

    def __sub__(self, o):
        return self + (-_iv(o))

    def _prod(self, o):
        c = np.stack([self.lo * o.lo, self.lo * o.hi, self.hi * o.lo, self.hi * o.hi])
        return c.min(axis=0), c.max(axis=0)

    def __mul__(self, o):
        o = _iv(o)
        lo, hi = self._prod(o)
        return Iv.f32(lo, hi)

    def square(self):
        """x * x with both operands the same value: the range of x^2."""
        a, b = np.abs(self.lo), np.abs(self.hi)
        hi = np.maximum(a, b) ** 2
        lo = np.where((self.lo <= 0) & (self.hi >= 0), 0.0, np.minimum(a, b) ** 2)
        return Iv.f32(lo, hi)

    def __truediv__(self, o):
        o = _iv(o)
        if np.any((o.lo <= 0) & (o.hi >= 0)):
            raise ZeroDivisionError("denominator interval contains zero")
        c = np.stack([self.lo / o.lo, self.lo / o.hi, self.hi / o.lo, self.hi / o.hi])
        return Iv.f32(c.min(axis=0), c.max(axis=0))

    def abs_max(self):
        return np.maximum(np.abs(self.lo), np.abs(self.hi))

    def contains(self, x):
        x = np.asarray(x, dtype=np.float64)
        return (self.lo <= x) & (x <= self.hi)


def _iv(v):
    return v if isinstance(v, Iv) else Iv(np.float64(F32(v)))


def fma(a, b, c):
    """fp32 enclosure of fmaf(a, b, c): the exact product-sum, rounded once."""
    a, b, c = _iv(a), _iv(b), _iv(c)
    lo, hi = a._prod(b)
    return Iv.f32(_down64(lo) + c.lo, _up64(hi) + c.hi)
