"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each checks it against a
value worked by hand (tests/golden/hand_example.json), a brute-force
computation organised differently (per sample and slot, no sorting, no
dedup), an invariant the paper states (Sec. 3.1: data staleness is zero in
synchronous training and GBA keeps the global batch of synchronous training;
Eq. 1 excludes gradients past the threshold), or a closed form of the
optimiser rules.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from synth import counter, workload
from synth.configs import BY_NAME

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_example.json")


def _frac(x):
    return float(Fraction(x))


@pytest.fixture(scope="module")
def hand():
    with open(GOLDEN) as f:
        return json.load(f)


def _hand_inputs(h):
    grads = np.array(h["dense_grads"], np.float32)
    ids = np.array(h["ids"], np.int64)
    rows = np.array(h["rows"], np.float32)
    off = np.array(h["offsets"], np.int64)
    tag = np.full(16, -7, np.int32)            # rows never touched keep their odd value
    for r, t in h["tag_before"].items():
        tag[int(r)] = t
    return grads, ids, rows, off, tag


# ---------------------------------------------------------------- hand example
@pytest.mark.parametrize("case", ["iota1", "iota0"])
def test_hand_example_weights_and_dense(hand, case):
    c = hand["cases"][case]
    w, s, nex = oracle.token_weights(hand["tokens"], hand["step"], c["iota"])
    assert list(s) == c["staleness"]
    assert list(w) == c["w"]
    assert nex == c["num_excluded"]
    grads, *_ = _hand_inputs(hand)
    g = oracle.aggregate_dense(grads, w)
    np.testing.assert_array_equal(g, np.array([_frac(x) for x in c["g_bar"]], np.float32))


@pytest.mark.parametrize("case", ["iota1", "iota0"])
@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_hand_example_sparse(hand, case, decay):
    c = hand["cases"][case]
    grads, ids, rows, off, tag = _hand_inputs(hand)
    w, _, _ = oracle.token_weights(hand["tokens"], hand["step"], c["iota"])
    out = oracle.aggregate_sparse(ids, rows, off, w, hand["tokens"], hand["step"], c["iota"],
                                  tag=tag, decay=decay)
    assert list(out["unique_ids"]) == hand["unique_ids"]
    assert list(out["seg_offsets"]) == hand["seg_offsets"]
    assert list(out["contrib_count"]) == hand["contrib_count"]
    assert list(out["active_count"]) == c[decay]["active_count"]
    np.testing.assert_array_equal(out["agg"][:, 0], np.array([_frac(x) for x in c[decay]["agg"]], np.float32))
    if decay == "id_tag":
        after = out["new_tag"]
        for r, t in c["id_tag"]["tag_after"].items():
            assert after[int(r)] == t
        untouched = np.setdiff1d(np.arange(16), [2, 7, 9])
        assert np.all(after[untouched] == -7)


def test_hand_example_adagrad(hand):
    c = hand["cases"]["iota1"]
    a = c["adagrad"]
    grads, ids, rows, off, tag = _hand_inputs(hand)
    w, _, _ = oracle.token_weights(hand["tokens"], hand["step"], c["iota"])
    g = oracle.aggregate_dense(grads, w)
    p, acc = oracle.adagrad(np.array(a["dense_param_before"], np.float32),
                            np.array(a["dense_accum_before"], np.float32), g, a["lr"], a["eps"])
    np.testing.assert_allclose(p, [_frac(x) for x in a["dense_param_after"]], rtol=2e-7)
    np.testing.assert_allclose(acc, [_frac(x) for x in a["dense_accum_after"]], rtol=2e-7)
    # rows, through the whole-step composition
    tr = a["token_rows"]
    table = {int(r): v for r, v in tr["param_before"].items()}
    accum = {int(r): v for r, v in tr["accum_before"].items()}
    res = oracle.gba_step(hand["tokens"], hand["step"], c["iota"], grads, ids, rows, off,
                          np.array(a["dense_param_before"], np.float32),
                          [np.array(a["dense_accum_before"], np.float32)],
                          lambda rr: np.array([[table[int(r)]] for r in rr], np.float32),
                          lambda k, rr: np.array([[accum[int(r)]] for r in rr], np.float32),
                          "adagrad", dict(lr=a["lr"], eps=a["eps"]))
    got = {int(r): (res["table_rows"][i, 0], res["table_slot_rows"][0][i, 0])
           for i, r in enumerate(res["active_ids"])}
    for r in (2, 7):
        assert got[r][0] == np.float32(_frac(tr["param_after"][str(r)]))
        assert got[r][1] == np.float32(_frac(tr["accum_after"][str(r)]))
    assert 9 not in got                       # inactive row: not updated


# ------------------------------------------------------------------ Eq. 1
def test_eq1_sync_mode_keeps_everything():
    """Sec. 3.1: data staleness is zero in synchronous training, so every
    gradient passes the tolerance function whatever the threshold."""
    for iota in (0, 1, 5):
        w, s, nex = oracle.token_weights(np.full(9, 42), 42, iota)
        assert np.all(s == 0) and np.all(w == 1) and nex == 0


def test_eq1_threshold_is_monotone_and_bsp_limit():
    """Raising iota never excludes more; iota >= max staleness excludes nothing
    (the BSP limit, Sec. 4.1); iota = -1 would exclude everything."""
    rng = np.random.default_rng(3)
    tok = 100 - rng.integers(0, 12, 64)
    prev = -1
    for iota in range(0, 13):
        _, _, nex = oracle.token_weights(tok, 100, iota)
        assert prev == -1 or nex <= prev
        prev = nex
    assert oracle.token_weights(tok, 100, 11)[2] == 0
    assert oracle.token_weights(tok, 100, -1)[2] == 64


def test_eq1_future_token_is_error():
    with pytest.raises(ValueError):
        oracle.token_weights([3, 6], 5, 2)


# ------------------------------------------------------- brute force (sparse)
def _brute_sparse(ids, rows, offsets, w, tokens, iota, tag, decay, norm, R):
    """Accumulate every (contribution, slot) into a full R x D array and a
    K x R 'seen' table, with plain loops: no sort, no dedup."""
    K = len(offsets) - 1
    D = rows.shape[1]
    acc = [[Fraction(0)] * D for _ in range(R)]
    seen = [[False] * R for _ in range(K)]
    active = [[False] * R for _ in range(K)]
    for m in range(K):
        for j in range(offsets[m], offsets[m + 1]):
            r = int(ids[j])
            seen[m][r] = True
            if decay == "token":
                wt = float(w[m])
            else:
                st = int(tag[r]) - int(tokens[m]) + 1
                wt = 1.0 if (st if st > 0 else 0) <= iota else 0.0
            if wt != 0:
                active[m][r] = True
                for d in range(D):
                    acc[r][d] += Fraction(float(rows[j][d])) * Fraction(wt)
    out = {}
    for r in range(R):
        c = sum(seen[m][r] for m in range(K))
        if c == 0:
            continue
        W = sum(active[m][r] for m in range(K))
        div = c if norm == "per_id_count" else K
        out[r] = (c, W, [float(a / div) for a in acc[r]])
    return out


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("decay", ["token", "id_tag"])
@pytest.mark.parametrize("norm", ["per_id_count", "by_k"])
def test_sparse_matches_brute_force(seed, decay, norm):
    rng = np.random.default_rng(seed)
    K, R, D = int(rng.integers(1, 8)), int(rng.integers(1, 40)), int(rng.integers(1, 5))
    sizes = rng.integers(0, 12, K)                    # empty contributions included
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    ids = rng.integers(0, R, N).astype(np.int64)
    rows = (rng.integers(-128, 128, (N, D)) * 2.0 ** -8).astype(np.float32)   # dyadic: exact sums
    step, iota = 20, int(rng.integers(0, 4))
    tokens = step - rng.integers(0, 6, K)
    tag = rng.integers(-1, step, R).astype(np.int32)
    w, _, _ = oracle.token_weights(tokens, step, iota)
    got = oracle.aggregate_sparse(ids, rows, off, w, tokens, step, iota, tag, decay, norm)
    ref = _brute_sparse(ids, rows, off, w, tokens, iota, tag, decay, norm, R)
    assert list(got["unique_ids"]) == sorted(ref)
    counts = np.bincount(ids, minlength=R)
    assert list(np.diff(got["seg_offsets"])) == [int(counts[r]) for r in sorted(ref)]
    for i, r in enumerate(got["unique_ids"]):
        c, W, vals = ref[int(r)]
        assert got["contrib_count"][i] == c
        assert got["active_count"][i] == W
        np.testing.assert_array_equal(got["agg"][i], np.array(vals, np.float32))
    if decay == "id_tag":
        act = [r for r in ref if ref[r][1] > 0]
        exp_tag = tag.copy()
        exp_tag[act] = step
        np.testing.assert_array_equal(got["new_tag"], exp_tag)


def test_dedup_special_cases():
    # one ID repeated N times across 3 contributions
    off = np.array([0, 5, 5, 9], np.int64)
    u, so, c = oracle.dedup(np.full(9, 17), off)
    assert list(u) == [17] and list(so) == [0, 9] and list(c) == [2]
    # all IDs distinct
    ids = np.array([9, 3, 14, 0, 7, 2], np.int64)
    u, so, c = oracle.dedup(ids, np.array([0, 2, 6], np.int64))
    assert list(u) == sorted(ids) and list(so) == list(range(7)) and np.all(c == 1)
    # nothing at all
    u, so, c = oracle.dedup(np.zeros(0, np.int64), np.array([0, 0], np.int64))
    assert u.size == 0 and list(so) == [0] and c.size == 0


# ------------------------------------------------- sync-mode invariant (Sec. 3.1)
def test_sync_invariant_equals_global_batch_gradient():
    """With every token fresh (staleness 0) and K local batches of B samples,
    the GBA aggregate equals the synchronous gradient of the global batch of
    K * B samples (Sec. 3.1: G_a = B_a M = G_s).  The reference here is the
    mean over all K * B per-sample gradients, computed without contributions."""
    rng = np.random.default_rng(11)
    K, B, L, P, R, D = 6, 5, 3, 7, 13, 4
    per_dense = rng.normal(size=(K, B, P))
    per_ids = rng.integers(0, R, (K, B, L))
    per_rows = rng.normal(size=(K, B, L, D))
    # local gradient of contribution m = mean over its B samples
    grads = [per_dense[m].mean(axis=0).astype(np.float32) for m in range(K)]
    ids = per_ids.reshape(-1).astype(np.int64)
    rows = (per_rows / B).reshape(-1, D).astype(np.float32)
    off = np.arange(K + 1, dtype=np.int64) * B * L
    tokens = np.full(K, 9)
    w, _, nex = oracle.token_weights(tokens, 9, iota=0)
    assert nex == 0
    g = oracle.aggregate_dense(grads, w)
    sync_dense = per_dense.reshape(K * B, P).mean(axis=0)
    np.testing.assert_allclose(g, sync_dense, rtol=2e-6, atol=1e-7)
    sp = oracle.aggregate_sparse(ids, rows, off, w, tokens, 9, 0, norm="by_k")
    sync_rows = np.zeros((R, D))
    for k in range(K):
        for b in range(B):
            for l in range(L):
                sync_rows[per_ids[k, b, l]] += per_rows[k, b, l]
    sync_rows /= K * B
    np.testing.assert_allclose(sp["agg"], sync_rows[sp["unique_ids"]], rtol=2e-6, atol=1e-7)
    assert np.all(sp["active_count"] == sp["contrib_count"])


# ------------------------------------------------ threshold invariant (Eq. 1)
@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_excluded_contributions_never_reach_the_result(decay):
    """A contribution past the threshold is excluded (Eq. 1): filling it with
    NaN changes nothing, while its IDs still count in c_r."""
    w_ = BY_NAME["c0"].scaled(K=5, B=4, L=3, R=50, D=4, P=33)
    hs = workload.host_step(w_, seed=5, staleness=[0, 4, 1, 7, 2])
    w, _, nex = oracle.token_weights(hs.tokens, hs.step, 2)
    assert nex == 2
    clean = oracle.aggregate_dense(hs.grads, w)
    sp_clean = oracle.aggregate_sparse(hs.ids, hs.rows, hs.offsets, w, hs.tokens, hs.step, 2,
                                       hs.tags, decay)
    grads, rows = hs.grads.copy(), hs.rows.copy()
    grads[w == 0] = np.nan
    weights = oracle.row_weights(w, hs.tokens, oracle.contribution_of_occurrence(hs.offsets),
                                 hs.ids, 2, decay, hs.tags)
    rows[weights == 0] = np.nan
    dirty = oracle.aggregate_dense(grads, w)
    sp_dirty = oracle.aggregate_sparse(hs.ids, rows, hs.offsets, w, hs.tokens, hs.step, 2,
                                       hs.tags, decay)
    assert np.all(np.isfinite(dirty)) and np.all(np.isfinite(sp_dirty["agg"]))
    np.testing.assert_array_equal(clean, dirty)
    for k in ("unique_ids", "seg_offsets", "contrib_count", "active_count", "agg"):
        np.testing.assert_array_equal(sp_clean[k], sp_dirty[k])
    # the stale contributions' IDs are still counted in c_r
    m_of_j = oracle.contribution_of_occurrence(hs.offsets)
    stale_ids = np.unique(hs.ids[w[m_of_j] == 0])
    assert np.any(sp_clean["contrib_count"][np.searchsorted(sp_clean["unique_ids"], stale_ids)] >
                  sp_clean["active_count"][np.searchsorted(sp_clean["unique_ids"], stale_ids)])


def test_id_tag_weights_dominate_token_weights():
    """Per-ID staleness never exceeds the token staleness (a row cannot have
    been updated more often than the dense vector), so every contribution that
    the token rule keeps is kept per ID; tags only move forward to k."""
    w_ = BY_NAME["c0"].scaled(K=8, B=16, L=4, R=300, D=4, P=8)
    hs = workload.host_step(w_, seed=9)
    for iota in range(0, 4):
        w, _, _ = oracle.token_weights(hs.tokens, hs.step, iota)
        a = oracle.aggregate_sparse(hs.ids, hs.rows, hs.offsets, w, hs.tokens, hs.step, iota,
                                    hs.tags, "token")
        b = oracle.aggregate_sparse(hs.ids, hs.rows, hs.offsets, w, hs.tokens, hs.step, iota,
                                    hs.tags, "id_tag")
        assert np.all(b["active_count"] >= a["active_count"])
        assert np.all(b["new_tag"] >= hs.tags)
        changed = np.nonzero(b["new_tag"] != hs.tags)[0]
        assert np.all(b["new_tag"][changed] == hs.step)
        assert np.all(np.isin(changed, b["unique_ids"]))


# ----------------------------------------------------- arrival-order invariance
def test_order_of_arrival_does_not_matter():
    """Permuting the buffer (with each gradient keeping its token) leaves the
    step unchanged; dyadic values make float sums exact, so bitwise."""
    w_ = BY_NAME["c0"].scaled(K=7, B=8, L=5, R=90, D=4, P=50)
    hs = workload.host_step(w_, seed=21, value_kind=counter.KIND_DYADIC)
    perm = np.random.default_rng(0).permutation(w_.K)
    n = np.diff(hs.offsets)
    off_p = np.concatenate([[0], np.cumsum(n[perm])]).astype(np.int64)
    ids_p = np.concatenate([hs.ids[hs.offsets[m]:hs.offsets[m + 1]] for m in perm])
    rows_p = np.concatenate([hs.rows[hs.offsets[m]:hs.offsets[m + 1]] for m in perm])
    for decay in ("token", "id_tag"):
        w, _, _ = oracle.token_weights(hs.tokens, hs.step, 1)
        wp, _, _ = oracle.token_weights(hs.tokens[perm], hs.step, 1)
        np.testing.assert_array_equal(oracle.aggregate_dense(hs.grads, w),
                                      oracle.aggregate_dense(hs.grads[perm], wp))
        a = oracle.aggregate_sparse(hs.ids, hs.rows, hs.offsets, w, hs.tokens, hs.step, 1, hs.tags, decay)
        b = oracle.aggregate_sparse(ids_p, rows_p, off_p, wp, hs.tokens[perm], hs.step, 1, hs.tags, decay)
        for k in ("unique_ids", "seg_offsets", "contrib_count", "active_count", "agg"):
            np.testing.assert_array_equal(a[k], b[k])


# ------------------------------------------------------- optimiser closed forms
def test_adagrad_constant_gradient_closed_form():
    """From a zero accumulator, T steps of a constant gradient g give
    a_T = T g^2 and p_T = p_0 - lr sign(g) sum_{t<=T} 1/sqrt(t) (eps = 0)."""
    g = np.array([0.25, -2.0, 3.0], np.float32)
    p = np.array([1.0, 0.5, -1.0], np.float32)
    a = np.zeros(3, np.float32)
    lr, T = 0.1, 9
    for _ in range(T):
        p, a = oracle.adagrad(p, a, g, lr, 0.0)
    harm = sum(1.0 / np.sqrt(t) for t in range(1, T + 1))
    np.testing.assert_allclose(a, T * g.astype(np.float64) ** 2, rtol=1e-7)
    np.testing.assert_allclose(p, np.array([1.0, 0.5, -1.0]) - lr * np.sign(g) * harm, rtol=1e-6)


def test_adagrad_epsilon_sits_outside_the_root():
    # a = 0, g = 3, eps = 1: update lr * 3 / (3 + 1)
    p, a = oracle.adagrad(np.float32([0.0]), np.float32([0.0]), np.float32([3.0]), 1.0, 1.0)
    assert p[0] == np.float32(-0.75) and a[0] == 9.0


def test_adam_first_step_closed_form():
    """Kingma and Ba: from m = v = 0 at t = 1, the bias-corrected moments are
    g and g^2, so the step is lr g / (|g| + eps)."""
    g = np.array([0.5, -4.0, 1e-3], np.float32)
    z = np.zeros(3, np.float32)
    lr, eps = 0.01, 0.5
    p, m, v = oracle.adam(z, z, z, g, lr, 0.9, 0.999, eps, 1)
    np.testing.assert_allclose(p, -lr * g / (np.abs(g) + eps), rtol=1e-6)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-6)
    np.testing.assert_allclose(v, 0.001 * g.astype(np.float64) ** 2, rtol=1e-6)


def test_adam_constant_gradient_closed_form():
    """With a constant gradient the bias-corrected moments stay g and g^2 at
    every t, so after T steps p_T = p_0 - T lr g / (|g| + eps)."""
    g = np.array([0.5, -2.0], np.float32)
    p = np.array([1.0, 1.0], np.float32)
    m = np.zeros(2, np.float32)
    v = np.zeros(2, np.float32)
    lr, eps, T = 1e-3, 0.25, 12
    for t in range(1, T + 1):
        p, m, v = oracle.adam(p, m, v, g, lr, 0.9, 0.999, eps, t)
    np.testing.assert_allclose(p, 1.0 - T * lr * g / (np.abs(g) + eps), rtol=1e-6)


# ------------------------------------------------------------------ App. B
@pytest.mark.parametrize("seed", range(6))
def test_early_sum_equals_exact_rational_mean(seed):
    """Folding dyadic contributions in as they arrive, in any grouping, gives
    the exact weighted sum / K (computed here in rational arithmetic)."""
    rng = np.random.default_rng(seed)
    K, P = int(rng.integers(1, 12)), int(rng.integers(1, 9))
    grads = [counter.values_range(seed, 700 + m, 0, P, counter.KIND_DYADIC) for m in range(K)]
    w = (rng.random(K) < 0.7).astype(np.float32)
    run = np.zeros(P, np.float64)
    cuts = np.sort(rng.choice(np.arange(1, K), size=min(K - 1, int(rng.integers(0, 4))), replace=False)) \
        if K > 1 else np.zeros(0, int)
    for lo, hi in zip(np.r_[0, cuts], np.r_[cuts, K]):
        oracle.accumulate_dense(run, grads[lo:hi], w[lo:hi])
    got = oracle.finalize_dense(run, K)
    for i in range(P):
        exact = sum(Fraction(float(w[m])) * Fraction(float(grads[m][i])) for m in range(K)) / K
        assert got[i] == np.float32(float(exact)), (i, got[i], exact)


def test_early_sum_is_bitwise_the_one_shot_sum_and_skips_excluded():
    """Arrival order is buffer order, so the running sum is the one-shot sum
    bit for bit (non-dyadic values too); an excluded gradient is never read."""
    rng = np.random.default_rng(3)
    K, P = 37, 1001
    grads = [counter.values_range(9, 800 + m, 0, P, counter.KIND_GRAD, counter.grad_scale(1e-2)) for m in range(K)]
    tokens = 50 - rng.integers(0, 6, K)
    w, _, _ = oracle.token_weights(tokens, 50, 3)
    poisoned = [g if w[m] != 0 else np.full(P, np.nan, np.float32) for m, g in enumerate(grads)]
    run = np.zeros(P, np.float64)
    for lo in range(0, K, 5):
        oracle.accumulate_dense(run, poisoned[lo:lo + 5], w[lo:lo + 5])
    assert np.array_equal(oracle.finalize_dense(run, K), oracle.aggregate_dense(grads, w))


# ------------------------------------------------- Sec. 3.1, Alg. 2 pull side
def test_token_list_gives_m_batches_per_value_in_ascending_order():
    """Sec. 3.1: tokens start from zero, M consecutive batches share each
    value, and the list ascends; with Q batches there are ceil(Q / M)
    distinct values."""
    for M in (1, 3, 4, 64):
        Q = 10 * M + 3
        toks = [oracle.token_of_batch(i, M) for i in range(Q)]
        assert toks[0] == 0 and all(b - a in (0, 1) for a, b in zip(toks, toks[1:]))
        values, counts = np.unique(toks, return_counts=True)
        assert values.size == -(-Q // M)
        assert np.all(counts[:-1] == M) and counts[-1] == Q - M * (values.size - 1)


@pytest.mark.parametrize("n,R", [(1, 5), (50, 7), (1000, 100_000), (500, 1)])
def test_pull_rows_reconstructs_the_request(n, R):
    """Looking rows up once per distinct ID loses nothing: rows[inverse] is
    the plain per-position lookup, and the distinct IDs are sorted and unique."""
    rng = np.random.default_rng(n)
    ids = rng.integers(0, R, n).astype(np.int64)
    table = rng.standard_normal((R, 4)).astype(np.float32)
    u, inv, rows = oracle.pull_rows(ids, table)
    assert np.all(np.diff(u) > 0)
    assert np.array_equal(u[inv], ids)
    assert np.array_equal(rows[inv], table[ids])
    assert set(u.tolist()) == set(ids.tolist())


# ---------------------------------------------- storage keyed by 64-bit IDs
@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_results_follow_the_id_not_its_value(decay):
    """Renaming the IDs by any injective map (as an ID -> row index does)
    renames the outputs and changes nothing else: per-ID sums, c_r, W_r and
    tags travel with the ID."""
    rng = np.random.default_rng(11)
    K, R, D = 5, 300, 4
    sizes = rng.integers(0, 60, K)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    ids = rng.integers(0, R, N).astype(np.int64)
    rows = counter.values_range(4, counter.STREAM_ROWS, 0, N * D, counter.KIND_DYADIC).reshape(N, D)
    tokens = 40 - rng.integers(0, 5, K)
    w, _, _ = oracle.token_weights(tokens, 40, 2)
    tag = rng.integers(-1, 40, R).astype(np.int64)
    perm = rng.permutation(R)          # the renaming: ID r becomes perm[r]
    tag2 = np.empty(R, np.int64)
    tag2[perm] = tag
    a = oracle.aggregate_sparse(ids, rows, off, w, tokens, 40, 2, tag.copy(), decay)
    b = oracle.aggregate_sparse(perm[ids], rows, off, w, tokens, 40, 2, tag2.copy(), decay)
    order = np.argsort(perm[a["unique_ids"]])
    assert np.array_equal(b["unique_ids"], perm[a["unique_ids"]][order])
    for k in ("contrib_count", "active_count", "agg"):
        assert np.array_equal(b[k], a[k][order]), k
    if decay == "id_tag":
        assert np.array_equal(b["new_tag"][perm], a["new_tag"])


# ------------------------------------------- magnitude companions of the float rule
# The comparison rule passes a float x against the oracle's r when
# |x - r| <= 1e-5 max(|r|, mu).  mu comes from the oracle's *_magnitude
# functions and agg_mu; these pins check them against a second worked example
# (tests/golden/magnitudes.json, mixed signs so that mu != |r| where a sum
# cancels), against brute-force sums of absolute terms in exact arithmetic,
# and against the error they must cover.
MAG = os.path.join(os.path.dirname(__file__), "golden", "magnitudes.json")


@pytest.fixture(scope="module")
def mag():
    with open(MAG) as f:
        return json.load(f)


def _fr(v):
    return np.array([float(Fraction(x)) for x in v])


def _mag_inputs(m):
    grads = np.array(m["dense_grads"], np.float32)
    ids = np.array(m["ids"], np.int64)
    rows = np.array(m["rows"], np.float32)
    off = np.array(m["offsets"], np.int64)
    tag = np.full(16, -7, np.int32)
    for r, t in m["tag_before"].items():
        tag[int(r)] = t
    w, _, _ = oracle.token_weights(m["tokens"], m["step"], m["iota"])
    return grads, ids, rows, off, tag, w


def test_magnitude_of_the_dense_sum(mag):
    grads, _, _, _, _, w = _mag_inputs(mag)
    assert list(w) == mag["w"]
    np.testing.assert_array_equal(oracle.aggregate_dense(grads, w), _fr(mag["g_bar"]).astype(np.float32))
    # the stale contribution's 100s must not count: (|1| + |-3|) / 3 and (|-6| + |2|) / 3
    np.testing.assert_array_equal(oracle.aggregate_dense_magnitude(grads, w), _fr(mag["g_bar_mu"]))


@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_magnitude_of_the_row_sums(mag, decay):
    _, ids, rows, off, tag, w = _mag_inputs(mag)
    out = oracle.aggregate_sparse(ids, rows, off, w, mag["tokens"], mag["step"], mag["iota"], tag=tag, decay=decay)
    assert list(out["unique_ids"]) == mag["unique_ids"]
    assert list(out["contrib_count"]) == mag["contrib_count"]
    assert list(out["active_count"]) == mag[decay]["active_count"]
    np.testing.assert_array_equal(out["agg"][:, 0], _fr(mag[decay]["agg"]).astype(np.float32))
    np.testing.assert_array_equal(out["agg_mu"][:, 0], _fr(mag[decay]["agg_mu"]))


def test_magnitudes_of_adagrad(mag):
    grads, ids, rows, off, tag, w = _mag_inputs(mag)
    a = mag["adagrad"]
    lr, eps = float(Fraction(a["lr"])), float(a["eps"])
    g = oracle.aggregate_dense(grads, w)
    gmu = oracle.aggregate_dense_magnitude(grads, w)
    d = a["dense"]
    p0, a0 = _fr(d["param_before"]).astype(np.float32), _fr(d["accum_before"]).astype(np.float32)
    p1, a1 = oracle.adagrad(p0, a0, g, lr, eps)
    np.testing.assert_allclose(p1, _fr(d["param_after"]), rtol=1e-6)
    np.testing.assert_allclose(a1, _fr(d["accum_after"]), rtol=1e-6)
    mu_p, mu_a = oracle.adagrad_magnitude(p0, a0, g, gmu, lr, eps)
    np.testing.assert_allclose(mu_p, _fr(d["mu_param"]), rtol=1e-6)
    np.testing.assert_allclose(mu_a, _fr(d["mu_accum"]), rtol=1e-6)
    # table rows, with the row means and their companions
    sp = oracle.aggregate_sparse(ids, rows, off, w, mag["tokens"], mag["step"], mag["iota"])
    tr = a["token_rows"]
    assert list(sp["unique_ids"]) == tr["ids"]
    E0, A0 = _fr(tr["param_before"]).astype(np.float32)[:, None], _fr(tr["accum_before"]).astype(np.float32)[:, None]
    E1, A1 = oracle.adagrad(E0, A0, sp["agg"], lr, eps)
    np.testing.assert_allclose(E1[:, 0], _fr(tr["param_after"]), rtol=1e-6)
    np.testing.assert_allclose(A1[:, 0], _fr(tr["accum_after"]), rtol=1e-6)
    mu_p, mu_a = oracle.adagrad_magnitude(E0, A0, sp["agg"], sp["agg_mu"], lr, eps)
    np.testing.assert_allclose(mu_p[:, 0], _fr(tr["mu_param"]), rtol=1e-6)
    np.testing.assert_allclose(mu_a[:, 0], _fr(tr["mu_accum"]), rtol=1e-6)


def test_magnitudes_of_adam(mag):
    grads, _, _, _, _, w = _mag_inputs(mag)
    a = mag["adam"]
    lr, b1, b2 = (float(Fraction(a[k])) for k in ("lr", "beta1", "beta2"))
    eps, t = float(a["eps"]), a["t"]
    g = oracle.aggregate_dense(grads, w)
    gmu = oracle.aggregate_dense_magnitude(grads, w)
    d = a["dense"]
    p0, m0, v0 = (_fr(d[k]).astype(np.float32) for k in ("param_before", "m_before", "v_before"))
    p1, m1, v1 = oracle.adam(p0, m0, v0, g, lr, b1, b2, eps, t)
    np.testing.assert_allclose(p1, _fr(d["param_after"]), rtol=1e-6)
    np.testing.assert_allclose(m1, _fr(d["m_after"]), rtol=1e-6)
    np.testing.assert_allclose(v1, _fr(d["v_after"]), rtol=1e-6)
    mu_p, mu_m, mu_v = oracle.adam_magnitude(p0, m0, v0, g, gmu, lr, b1, b2, eps, t)
    np.testing.assert_allclose(mu_p, _fr(d["mu_param"]), rtol=1e-6)
    np.testing.assert_allclose(mu_m, _fr(d["mu_m"]), rtol=1e-6)
    np.testing.assert_allclose(mu_v, _fr(d["mu_v"]), rtol=1e-6)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("decay", ["token", "id_tag"])
@pytest.mark.parametrize("norm", ["per_id_count", "by_k"])
def test_magnitudes_are_sums_of_absolute_terms(seed, decay, norm):
    """Brute force in exact rational arithmetic, organised per contribution and
    occurrence: mu of the dense sum is sum over kept m of |w_m g_m| / K, and mu
    of a row mean is sum over its kept occurrences of |w x| / c_r (or / K).
    Dyadic inputs make the oracle's float64 sums exact, so after the one
    correctly rounded division both sides agree bit for bit."""
    rng = np.random.default_rng(4000 + seed)
    K, P, D, R = int(rng.integers(1, 6)), int(rng.integers(1, 7)), int(rng.integers(1, 4)), int(rng.integers(1, 9))
    step, iota = 20, int(rng.integers(0, 4))
    tokens = step - rng.integers(0, 6, K)
    w, _, _ = oracle.token_weights(tokens, step, iota)
    w = (w * rng.choice([1.0, 0.5, 0.75, 0.25], K)).astype(np.float32)    # fractional policies (token mode)
    grads = (rng.integers(-64, 65, (K, P)) / 8).astype(np.float32)
    sizes = rng.integers(0, 5, K)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    ids = rng.integers(0, R, N).astype(np.int64)
    rows = (rng.integers(-64, 65, (N, D)) / 16).astype(np.float32)
    tag = rng.integers(-1, step, R).astype(np.int32)

    F = Fraction
    want = [sum((abs(F(float(w[m])) * F(float(grads[m, i]))) for m in range(K) if w[m] != 0), F(0)) / K
            for i in range(P)]
    np.testing.assert_array_equal(oracle.aggregate_dense_magnitude(grads, w), np.array([float(x) for x in want]))

    if N == 0:
        return
    seen, total = {}, {}
    for m in range(K):
        for j in range(int(off[m]), int(off[m + 1])):
            r = int(ids[j])
            seen.setdefault(r, set()).add(m)
            if decay == "token":
                wt = F(float(w[m]))
            else:
                wt = F(1) if max(0, int(tag[r]) - int(tokens[m]) + 1) <= iota else F(0)
            acc = total.setdefault(r, [F(0)] * D)
            if wt != 0:
                for d_ in range(D):
                    acc[d_] += abs(wt * F(float(rows[j, d_])))
    out = oracle.aggregate_sparse(ids, rows, off, w, tokens, step, iota, tag=tag, decay=decay, norm=norm)
    keys = sorted(total)
    assert list(out["unique_ids"]) == keys
    for u, r in enumerate(keys):
        div = len(seen[r]) if norm == "per_id_count" else K
        np.testing.assert_array_equal(out["agg_mu"][u], np.array([float(x / div) for x in total[r]]))


def test_rule_t_rejects_an_error_of_twice_the_bound():
    from compare import assert_rule_t
    ref = np.array([1.0, -2.0, 1e-3, 0.0])
    mu = np.array([3.0, 2.0, 10.0, 4.0])
    assert_rule_t(ref + 0.9e-5 * mu, ref, mu, "inside")
    assert_rule_t(ref - 0.9e-5 * mu, ref, mu, "inside")
    for i in range(ref.size):
        bad = ref.copy()
        bad[i] += 2e-5 * mu[i]
        with pytest.raises(AssertionError):
            assert_rule_t(bad, ref, mu, "outside")
    # without a companion the bound is relative to |r|
    with pytest.raises(AssertionError):
        assert_rule_t(np.array([1.0 + 2e-5]), np.array([1.0]), None, "relative")
    assert_rule_t(np.array([1.0 + 0.5e-5]), np.array([1.0]), None, "relative")
    with pytest.raises(AssertionError):
        assert_rule_t(np.array([np.nan]), np.array([1.0]), None, "nan")


@pytest.mark.parametrize("seed", range(4))
def test_optimiser_magnitudes_cover_the_gradient_tolerance(seed):
    """A gradient that is itself within 1e-5 mu_g of the oracle's moves each
    optimiser output by at most 1e-5 of that output's companion: the companions
    carry the tolerance of their input through the update.  State values are
    those of a warm parameter server (the generator's accumulator and moment
    ranges), and mu_g runs up to 20 |g| (cancelling sums)."""
    rng = np.random.default_rng(77 + seed)
    n = 20000
    g = rng.normal(0.0, 1e-2, n).astype(np.float32)
    gmu = np.abs(g.astype(np.float64)) * rng.uniform(1.0, 20.0, n)
    delta = rng.uniform(-0.99, 0.99, n) * 1e-5 * gmu
    g2 = (g.astype(np.float64) + delta).astype(np.float32)
    p = rng.uniform(-1 / 16, 1 / 16, n).astype(np.float32)
    lr, eps = 0.01, 1e-8
    a = rng.uniform(1 / 16, 5 / 16, n).astype(np.float32)
    mu_p, mu_a = oracle.adagrad_magnitude(p, a, g, gmu, lr, eps)
    for x, y, mu in zip(oracle.adagrad(p, a, g, lr, eps), oracle.adagrad(p, a, g2, lr, eps), (mu_p, mu_a)):
        assert np.all(np.abs(y.astype(np.float64) - x) <= 1e-5 * mu)
    m = rng.uniform(-1e-3, 1e-3, n).astype(np.float32)
    v = rng.uniform(2.0 ** -18, 5 * 2.0 ** -18, n).astype(np.float32)
    b1, b2, t = 0.9, 0.999, 1001
    mu_p, mu_m, mu_v = oracle.adam_magnitude(p, m, v, g, gmu, 1e-3, b1, b2, eps, t)
    for x, y, mu in zip(oracle.adam(p, m, v, g, 1e-3, b1, b2, eps, t), oracle.adam(p, m, v, g2, 1e-3, b1, b2, eps, t),
                        (mu_p, mu_m, mu_v)):
        assert np.all(np.abs(y.astype(np.float64) - x) <= 1e-5 * mu)
