"""Skewed embedding-ID draws (host side).

The paper motivates GBA's per-ID handling by the skew of ID occurrences in
recommendation data (Fig. 4 and Insight 2 of Sec. 2).  The stand-in here is a
truncated Zipf law P(rank = k) proportional to k**-s over ranks 1..n, drawn
by rejection-inversion (W. Hoermann and G. Derflinger, "Rejection-inversion to
generate variates from monotone discrete distributions", ACM TOMACS 6(3),
1996), so no table over n ranks is needed.  Ranks are then spread over the
table by the bijection r -> (a r + b) mod n, gcd(a, n) = 1, so hot rows are
not adjacent in memory.

The uniforms come from the counter generator (stream STREAM_ZIPF, index
``j * 64 + attempt``), so occurrence j's ID depends only on the seed and j.
"""
from __future__ import annotations

import math

import numpy as np

from . import counter

MAX_ATTEMPTS = 64
BIJECTION_A = 2654435761      # prime; stepped up when it shares a factor with n
BIJECTION_B = 1442695040888963407


def _helper1(t):
    """log1p(t) / t, continuous at t = 0."""
    t = np.asarray(t, dtype=np.float64)
    small = np.abs(t) < 1e-8
    safe = np.where(small, 1.0, t)
    return np.where(small, 1.0 - t * (0.5 - t / 3.0), np.log1p(safe) / safe)


def _helper2(t):
    """expm1(t) / t, continuous at t = 0."""
    t = np.asarray(t, dtype=np.float64)
    small = np.abs(t) < 1e-8
    safe = np.where(small, 1.0, t)
    return np.where(small, 1.0 + t * 0.5 * (1.0 + t / 3.0), np.expm1(safe) / safe)


class ZipfRejectionInversion:
    """Draw ranks in 1..n with P(k) proportional to k**-s (s > 0)."""

    def __init__(self, n: int, s: float):
        if n < 1 or s <= 0:
            raise ValueError("need n >= 1 and s > 0")
        self.n = int(n)
        self.s = float(s)
        self.h_x1 = float(self._H(1.5)) - 1.0
        self.h_n = float(self._H(self.n + 0.5))
        self.sq = 2.0 - float(self._H_inv(self._H(2.5) - self._h(2.0)))

    def _h(self, x):
        return np.exp(-self.s * np.log(x))

    def _H(self, x):
        # integral of x**-s from 1 to x, up to a constant: (x^(1-s) - 1) / (1 - s)
        lx = np.log(x)
        return _helper2((1.0 - self.s) * lx) * lx

    def _H_inv(self, y):
        t = np.maximum(y * (1.0 - self.s), -1.0)
        return np.exp(_helper1(t) * y)

    def ranks(self, seed: int, j: np.ndarray) -> np.ndarray:
        """Rank (1-based) of each occurrence index j; deterministic in (seed, j)."""
        j = np.asarray(j, dtype=np.int64)
        out = np.zeros(j.shape, dtype=np.int64)
        todo = np.arange(j.size)
        for attempt in range(MAX_ATTEMPTS):
            if todo.size == 0:
                break
            ctr = j[todo].astype(np.uint64) * np.uint64(MAX_ATTEMPTS) + np.uint64(attempt)
            v = 1.0 - counter.uniform01(seed, counter.STREAM_ZIPF, ctr)      # in (0, 1]
            u = self.h_n + v * (self.h_x1 - self.h_n)
            x = self._H_inv(u)
            k = np.clip(np.floor(x + 0.5), 1, self.n)
            ok = (k - x <= self.sq) | (u >= self._H(k + 0.5) - self._h(k))
            out[todo[ok]] = k[ok].astype(np.int64)
            todo = todo[~ok]
        # The acceptance rate is above 0.9 for every law used here, so reaching
        # this point has probability below 1e-60 per draw; rank 1 keeps it total.
        out[todo] = 1
        return out


def bijection_multiplier(n: int) -> int:
    a = BIJECTION_A % n if n > 1 else 1
    if a == 0:
        a = 1
    while math.gcd(a, n) != 1:
        a += 1
    return a


def rank_to_row(rank0: np.ndarray, n: int) -> np.ndarray:
    """Map 0-based ranks to rows in [0, n) by r -> (a r + b) mod n."""
    a = bijection_multiplier(n)
    b = BIJECTION_B % n
    r = np.asarray(rank0, dtype=np.int64)
    # a < 2**32 and r < 2**31 keep the product inside int64 only for small n;
    # use Python-int-safe modular arithmetic via two 32-bit halves.
    lo = (r & 0xFFFF) * a
    hi = ((r >> 16) * a) % n
    return ((hi * 65536) % n + lo % n + b) % n
