"""The float32 optimiser updates stay inside the comparison rule.

Every optimiser update (dense and table rows, separate and fused calls)
computes Adagrad (Duchi et al. 2011) and Adam (Kingma and Ba 2015), the
optimisers Table 1 names, in float32 with the hardware square root and
reciprocal, each within 1 ulp of the exact value:
  Adagrad: a' = a + g*g, p' = p - (lr g) * rcp(sqrt(a') + eps);
  Adam:    m' = b1 m + (1 - b1) g, v' = b2 v + (1 - b2) g*g,
           p' = p - (lr m' / bc1) * rcp(sqrt(v' / bc2) + eps),
with lr, eps, b1, b2 and the constants 1 - b1, 1 - b2, 1 / bc1 and 1 / bc2
rounded once to float32.  This emulates that arithmetic in numpy, with every
rounding of the square root and the reciprocal pushed one ulp either way, and
checks the result against the oracle under the parity rule with the oracle's
magnitude companions: the error is a few 1e-7 of the companion, far inside
1e-5, also where p' or m' cancels to almost nothing.  (CPU only: no device
code runs here.)"""
import itertools
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from oracle import gba_oracle as oracle  # noqa: E402
from compare import assert_rule_t  # noqa: E402

F = np.float32


def _ulp_shift(x, k):
    """x moved k ulps (k in -1, 0, 1) in float32."""
    if k == 0:
        return x
    return np.nextafter(x, np.full_like(x, np.inf if k > 0 else -np.inf))


def _row_adagrad_f32(p, a, g, lr, eps, ks, kr):
    p, a, g = F(p), F(a), F(g)
    an = (a + g * g).astype(F)
    s = _ulp_shift(np.sqrt(an).astype(F), ks)
    den = (s + F(eps)).astype(F)
    r = _ulp_shift((F(1.0) / den).astype(F), kr)
    step = ((F(lr) * g).astype(F) * r).astype(F)
    return (p - step).astype(F), an


def _cases(n=20000, seed=11):
    rng = np.random.default_rng(seed)
    p = rng.uniform(-1.0, 1.0, n).astype(F)
    a = rng.uniform(0.0, 2.0, n).astype(F)
    g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-6, 1, n)).astype(F)
    lr, eps = 0.01, 1e-8
    # a quarter of the cases cancel: p is set to the step itself, nudged by
    # a few float32 ulps, so p' is a small remainder of two equal terms
    step = lr * g.astype(np.float64) / (np.sqrt(a.astype(np.float64) + g.astype(np.float64) ** 2) + eps)
    c = rng.random(n) < 0.25
    p[c] = (step[c] * (1.0 + rng.integers(-4, 5, c.sum()) * 2.0 ** -24)).astype(F)
    # zero gradients and zero accumulators
    g[:50] = 0.0
    a[50:100] = 0.0
    return p, a, g, lr, eps


def test_row_adagrad_f32_within_rule_with_companion():
    p, a, g, lr, eps = _cases()
    ref_p, ref_a = oracle.adagrad(p, a, g, lr, eps)
    mu_p, mu_a = oracle.adagrad_magnitude(p, a, g, np.abs(g), lr, eps)
    for ks, kr in itertools.product((-1, 0, 1), repeat=2):
        got_p, got_a = _row_adagrad_f32(p, a, g, lr, eps, ks, kr)
        assert_rule_t(got_p, ref_p, mu_p, f"p' (sqrt {ks:+d} ulp, rcp {kr:+d} ulp)")
        assert_rule_t(got_a, ref_a, mu_a, "a'")


def test_row_adagrad_f32_error_is_far_inside_the_rule():
    """The worst error over the cases, in units of |p| + |step|, is below
    1e-6 (a tenth of the rule), so rows whose gradient carries its own
    rounding error still pass."""
    p, a, g, lr, eps = _cases(seed=12)
    ref_p, _ = oracle.adagrad(p, a, g, lr, eps)
    step = lr * np.abs(g.astype(np.float64)) / (np.sqrt(a.astype(np.float64) + g.astype(np.float64) ** 2) + eps)
    scale = np.abs(p.astype(np.float64)) + step + 1e-30
    worst = 0.0
    for ks, kr in itertools.product((-1, 0, 1), repeat=2):
        got_p, _ = _row_adagrad_f32(p, a, g, lr, eps, ks, kr)
        worst = max(worst, float(np.max(np.abs(got_p.astype(np.float64) - ref_p.astype(np.float64)) / scale)))
    assert worst < 1e-6, worst


def test_row_adagrad_plain_rule_would_fail_on_cancellation():
    """Pins the need for the companion: without it (mu = |p'|) the cancelling
    cases exceed the plain relative rule, so the tests must pass mu."""
    p, a, g, lr, eps = _cases(seed=13)
    ref_p, _ = oracle.adagrad(p, a, g, lr, eps)
    got_p, _ = _row_adagrad_f32(p, a, g, lr, eps, 1, 1)
    err = np.abs(got_p.astype(np.float64) - ref_p.astype(np.float64))
    assert np.any(err > 1e-5 * np.abs(ref_p.astype(np.float64)) + 1e-30)


def _row_adam_f32(p, m, v, g, lr, b1, b2, eps, t, ks, kr):
    p, m, v, g = F(p), F(m), F(v), F(g)
    bc1, bc2 = 1.0 - b1 ** t, 1.0 - b2 ** t
    mn = (F(b1) * m + F(1.0 - b1) * g).astype(F)
    vn = (F(b2) * v + F(1.0 - b2) * (g * g).astype(F)).astype(F)
    s = _ulp_shift(np.sqrt((vn * F(1.0 / bc2)).astype(F)).astype(F), ks)
    den = (s + F(eps)).astype(F)
    r = _ulp_shift((F(1.0) / den).astype(F), kr)
    step = ((F(lr) * (mn * F(1.0 / bc1)).astype(F)).astype(F) * r).astype(F)
    return (p - step).astype(F), mn, vn


def test_row_adam_f32_within_rule_with_companion():
    rng = np.random.default_rng(21)
    n = 20000
    p = rng.uniform(-1.0, 1.0, n).astype(F)
    m = (rng.standard_normal(n) * 1e-3).astype(F)
    v = (rng.uniform(0.0, 1.0, n) * 1e-6).astype(F)
    g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-6, 0, n)).astype(F)
    lr, b1, b2, eps, t = 1e-3, 0.9, 0.999, 1e-8, 7
    # cancelling first moments: b1 m = -(1 - b1) g to a few ulps
    c = rng.random(n) < 0.25
    m[c] = (-(1.0 - b1) * g[c].astype(np.float64) / b1 * (1.0 + rng.integers(-4, 5, c.sum()) * 2.0 ** -24)).astype(F)
    g[:50] = 0.0
    v[50:100] = 0.0
    ref = oracle.adam(p, m, v, g, lr, b1, b2, eps, t)
    mu = oracle.adam_magnitude(p, m, v, g, np.abs(g), lr, b1, b2, eps, t)
    for ks, kr in itertools.product((-1, 0, 1), repeat=2):
        got = _row_adam_f32(p, m, v, g, lr, b1, b2, eps, t, ks, kr)
        for x, r, u, what in zip(got, ref, mu, ("p'", "m'", "v'")):
            assert_rule_t(x, r, u, f"{what} (sqrt {ks:+d} ulp, rcp {kr:+d} ulp)")
