"""Comparison rules for the parity tests.

Integers, IDs, offsets, counts, tags and token weights must match bit for
bit.  A float result x passes against the oracle's r when
    |x - r| <= 1e-5 * max(|r|, mu)
where mu is the oracle's magnitude companion of r (the same expression with
every term taken in absolute value).  For a sum this is the relative error of
1e-5 measured against the sum of magnitudes, the quantity that bounds the
rounding error of any summation order (Higham, Accuracy and Stability of
Numerical Algorithms, 2nd ed., Sec. 4.2); where nothing cancels, mu = |r| and
the rule is a plain relative error of 1e-5.
"""
import numpy as np

RTOL = 1e-5


def assert_exact(got, ref, name):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} != {ref.shape}"
    bad = got != ref
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{name}: {int(bad.sum())} of {bad.size} differ; first at {tuple(i)}: "
                             f"got {got[tuple(i)]} want {ref[tuple(i)]}")


def assert_rule_t(got, ref, mu=None, name="", rtol=RTOL):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} != {ref.shape}"
    mag = np.abs(ref) if mu is None else np.maximum(np.abs(ref), np.asarray(mu, np.float64))
    bound = rtol * mag + 1e-30
    err = np.abs(got - ref)
    bad = ~(err <= bound)
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{name}: {int(bad.sum())} of {bad.size} outside the 1e-5 rule; first at {i}: "
                             f"got {got[i]!r} want {ref[i]!r} (bound {bound[i]:.3g})")
