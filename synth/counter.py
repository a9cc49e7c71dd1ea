"""Counter-based random values shared by the test inputs of both sides.

Every synthetic value is a pure function of (seed, stream, index): the
``n``-th output of a SplitMix64 generator (Steele, Lea and Flood, "Fast
splittable pseudorandom number generators", OOPSLA 2014) whose state starts at
``seed``, with ``n = (stream << 40) + index``.  The n-th output of SplitMix64 is
``mix(seed + (n + 1) * 0x9E3779B97F4A7C15)`` with the published finaliser
``mix``.  Because the value depends only on the counter, the same bits can be
produced on the host (this file, numpy uint64 arithmetic that wraps modulo
2**64) and on the device (``synth/gen.hip``), chunk by chunk and in any order.

The maps from 64-bit words to values are chosen so that one IEEE operation at
most turns an integer into the float, hence both sides round identically:

* ``param``      (u24 - 2**23) * 2**-27          uniform in [-1/16, 1/16)
* ``accum``      (u24 + 2**22) * 2**-26          in [1/16, 5/16)   (warm Adagrad state)
* ``adam_m``     (u24 - 2**23) * 2**-33          about +-1e-3
* ``adam_v``     (u24 + 2**22) * 2**-40          in [2**-18, 5 * 2**-18)
* ``grad``       f32(S - 131070) * f32(scale), S = sum of the four 16-bit
                 fields of the word (Irwin-Hall of order 4: a bounded
                 stand-in for a normal law; sd of S - 131070 is 37837.2)
* ``dyadic``     (top byte - 128) * 2**-8        exact-sum test values

where u24 is the top 24 bits of the word.  Nothing here computes any step of
the aggregation method; it only draws inputs.
"""
from __future__ import annotations

import numpy as np

GOLDEN_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# Standard deviation of (sum of four uniform 16-bit integers) - 131070.
IRWIN_HALL4_SD = float(np.sqrt(4.0 * (65536.0 ** 2 - 1.0) / 12.0))

# Value kinds: the integer codes are shared with the device generator.
KIND_PARAM = 0
KIND_ACCUM = 1
KIND_ADAM_M = 2
KIND_ADAM_V = 3
KIND_GRAD = 4
KIND_DYADIC = 5

# Stream ids (< 2**24).  Per-contribution arrays add the contribution index.
STREAM_DENSE_PARAM = 1
STREAM_DENSE_SLOT1 = 2
STREAM_DENSE_SLOT2 = 3
STREAM_TABLE = 4
STREAM_TABLE_SLOT1 = 5
STREAM_TABLE_SLOT2 = 6
STREAM_ROWS = 8
STREAM_ZIPF = 9
STREAM_STALENESS = 10
STREAM_TAGS = 11
STREAM_DENSE_GRAD_BASE = 1 << 16     # + m, m < 65536

_INDEX_BITS = 40


def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def words(seed: int, stream: int, index) -> np.ndarray:
    """SplitMix64 output number (stream << 40) + index, as uint64 (vectorised)."""
    if not (0 <= stream < (1 << 24)):
        raise ValueError("stream out of range")
    idx = np.asarray(index, dtype=np.uint64)
    ctr = (np.uint64(stream) << np.uint64(_INDEX_BITS)) + idx
    with np.errstate(over="ignore"):
        state = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + (ctr + np.uint64(1)) * GOLDEN_GAMMA
        return _mix(state)


def words_range(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    return words(seed, stream, np.arange(start, start + count, dtype=np.uint64))


def grad_scale(sigma: float) -> np.float32:
    """The one fp32 constant that maps centred Irwin-Hall integers to gradients."""
    return np.float32(sigma / IRWIN_HALL4_SD)


def to_values(w: np.ndarray, kind: int, scale: float = 0.0) -> np.ndarray:
    """Map 64-bit words to float32 values of the given kind (see module doc)."""
    w = np.asarray(w, dtype=np.uint64)
    if kind == KIND_GRAD:
        m16 = np.uint64(0xFFFF)
        s = ((w & m16) + ((w >> np.uint64(16)) & m16) + ((w >> np.uint64(32)) & m16)
             + (w >> np.uint64(48))).astype(np.int64) - 131070
        return s.astype(np.float32) * np.float32(scale)
    if kind == KIND_DYADIC:
        return ((w >> np.uint64(56)).astype(np.int64) - 128).astype(np.float32) * np.float32(2.0 ** -8)
    u24 = (w >> np.uint64(40)).astype(np.int64)
    if kind == KIND_PARAM:
        return ((u24 - (1 << 23)).astype(np.float64) * 2.0 ** -27).astype(np.float32)
    if kind == KIND_ACCUM:
        return ((u24 + (1 << 22)).astype(np.float64) * 2.0 ** -26).astype(np.float32)
    if kind == KIND_ADAM_M:
        return ((u24 - (1 << 23)).astype(np.float64) * 2.0 ** -33).astype(np.float32)
    if kind == KIND_ADAM_V:
        return ((u24 + (1 << 22)).astype(np.float64) * 2.0 ** -40).astype(np.float32)
    raise ValueError(f"unknown kind {kind}")


def values(seed: int, stream: int, index, kind: int, scale: float = 0.0) -> np.ndarray:
    return to_values(words(seed, stream, index), kind, scale)


def values_range(seed: int, stream: int, start: int, count: int, kind: int,
                 scale: float = 0.0) -> np.ndarray:
    return to_values(words_range(seed, stream, start, count), kind, scale)


def uniform01(seed: int, stream: int, index) -> np.ndarray:
    """Doubles in [0, 1) from the top 53 bits of each word."""
    w = words(seed, stream, index)
    return (w >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def ctz64(w: np.ndarray, cap: int = 64) -> np.ndarray:
    """Count of trailing zero bits of each word (64 for a zero word), capped."""
    w = np.asarray(w, dtype=np.uint64).copy()
    out = np.zeros(w.shape, dtype=np.int64)
    live = np.ones(w.shape, dtype=bool)
    for _ in range(min(cap, 64)):
        bit = (w & np.uint64(1)) == np.uint64(0)
        live &= bit
        out += live
        w >>= np.uint64(1)
    return np.minimum(out, cap)
