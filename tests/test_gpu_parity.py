"""Parity of every C-ABI entry point with the CPU oracle, on seeded inputs
at sizes that span several tiles and ragged tails, plus the degenerate
cases of the method (empty contributions, a single hot ID, all IDs
distinct, every contribution excluded, nothing at all)."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2205_11048_amd as gba
from compare import assert_exact, assert_rule_t
from paper_2205_11048_amd.step import GBAStep
from synth import counter, workload
from synth import device as sdev
from synth.configs import BY_NAME

pytestmark = pytest.mark.gpu
DEV = "cuda"


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


# ------------------------------------------------------------------ Eq. 1
@pytest.mark.parametrize("K", [1, 2, 63, 64, 65, 1000, 4096])
def test_token_weights(K):
    rng = np.random.default_rng(K)
    step, iota = 777, int(rng.integers(0, 6))
    tokens = step - rng.integers(0, 12, K)
    w = torch.empty(K, dtype=torch.float32, device=DEV)
    s = torch.empty(K, dtype=torch.int64, device=DEV)
    nex = torch.zeros(1, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    gba.gba_token_weights(dev(tokens), step, iota, w, s, nex, err)
    rw, rs, rn = oracle.token_weights(tokens, step, iota)
    assert_exact(host(w), rw, "w")
    assert_exact(host(s), rs, "staleness")
    assert int(host(nex)[0]) == rn
    assert int(host(err)[0]) == 0


def test_future_token_is_reported():
    tokens = np.array([5, 9, 4], np.int64)
    w = torch.empty(3, dtype=torch.float32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    gba.gba_token_weights(dev(tokens), 6, 2, w, err=err)
    assert int(host(err)[0]) & gba.DERR_FUTURE_TOKEN
    assert host(w)[1] == 0.0


# ------------------------------------------------------------ dense, Alg. 2
@pytest.mark.parametrize("K,P", [(1, 1), (3, 5), (4, 65536), (37, 100003), (256, 4099), (9, 3)])
def test_aggregate_dense(K, P):
    rng = np.random.default_rng(K * 1000 + P)
    grads = [counter.values_range(17, counter.STREAM_DENSE_GRAD_BASE + m, 0, P, counter.KIND_GRAD,
                                  counter.grad_scale(1e-2)) for m in range(K)]
    tokens = 50 - rng.integers(0, 6, K)
    w, _, _ = oracle.token_weights(tokens, 50, 3)
    ref = oracle.aggregate_dense(grads, w)
    poisoned = [g.copy() if w[m] != 0 else np.full(P, np.nan, np.float32) for m, g in enumerate(grads)]
    g_dev = [dev(g) for g in poisoned]
    out = torch.empty(P, dtype=torch.float32, device=DEV)
    gba.gba_aggregate_dense(gba.pointer_table(g_dev), dev(w), P, out)
    got = host(out)
    assert_rule_t(got, ref, oracle.aggregate_dense_magnitude(grads, w), "g_bar")
    assert_exact(got, ref, "g_bar (float64 accumulation in buffer order is exact)")


def test_aggregate_dense_launched_in_rounds():
    """More block steps than two rounds of the blocks the GPU holds at once
    (each step covers 32,768 elements): the reduction is launched one round at
    a time, and every element, the ragged tail included, is still summed once."""
    K, P = 3, 3 * 256 * 32768 + 3      # three rounds of 256 one-block compute units
    rng = np.random.default_rng(29)
    grads = [rng.random(P, dtype=np.float32) - np.float32(0.5) for _ in range(K)]
    w = np.array([1.0, 0.0, 1.0], np.float32)
    ref = oracle.aggregate_dense(grads, w)
    out = torch.empty(P, dtype=torch.float32, device=DEV)
    gba.gba_aggregate_dense(gba.pointer_table([dev(g) for g in grads]), dev(w), P, out)
    assert_exact(host(out), ref, "g_bar")
    steps = -(-(P // 4) // 8192)
    assert 1 < gba.gba_aggregate_dense_launches(P, K) <= steps
    assert gba.gba_aggregate_dense_launches(100_000, K) == 1
    assert gba.gba_aggregate_dense_launches(0, K) == 0


def test_aggregate_dense_unaligned_and_fractional_weights():
    K, P = 5, 1001
    base = [dev(counter.values_range(3, 100 + m, 0, P + 1, counter.KIND_GRAD, counter.grad_scale(1e-2)))
            for m in range(K)]
    views = [b[1:] for b in base]                  # 4-byte offset: no 16-byte loads possible
    w = np.array([1.0, 0.5, 0.0, 0.25, 1.0], np.float32)
    out = torch.empty(P, dtype=torch.float32, device=DEV)
    gba.gba_aggregate_dense(gba.pointer_table(views), dev(w), P, out)
    ref = oracle.aggregate_dense([host(v) for v in views], w)
    assert_exact(host(out), ref, "g_bar")


def test_aggregate_dense_all_excluded():
    K, P = 4, 777
    g_dev = [torch.full((P,), float("nan"), device=DEV) for _ in range(K)]
    out = torch.full((P,), 7.0, device=DEV)
    gba.gba_aggregate_dense(gba.pointer_table(g_dev), torch.zeros(K, device=DEV), P, out)
    assert_exact(host(out), np.zeros(P, np.float32), "g_bar")


# ----------------------------------------------------------- sparse, Alg. 2
def _run_sparse(ids, rows, offsets, w, tokens, step, iota, R, tag=None, decay="token", norm="per_id_count",
                plan=None):
    """plan: None calls gba_aggregate_sparse (automatic sort plan), else
    gba_aggregate_sparse_plan with that plan."""
    N, D = rows.shape
    K = len(offsets) - 1
    cap = max(N, 1)
    out = dict(unique_ids=torch.full((cap,), -5, dtype=torch.int64, device=DEV),
               seg_offsets=torch.full((cap + 1,), -5, dtype=torch.int64, device=DEV),
               contrib_count=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
               active_count=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
               agg=torch.full((cap, D), float("nan"), dtype=torch.float32, device=DEV),
               num_unique=torch.full((1,), -5, dtype=torch.int64, device=DEV))
    wsb = (gba.gba_aggregate_sparse_workspace_size(N, K, D, R) if plan is None
           else gba.gba_aggregate_sparse_plan_workspace_size(N, K, D, R, plan))
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    tag_d = dev(tag) if tag is not None else None
    args = (dev(ids), dev(rows.reshape(N, D)) if N else torch.empty((0, D), device=DEV),
            dev(offsets), R, dev(w), dev(tokens), step, iota, tag_d,
            gba.DECAY_ID_TAG if decay == "id_tag" else gba.DECAY_TOKEN,
            gba.NORM_BY_K if norm == "by_k" else gba.NORM_PER_ID_COUNT,
            out["unique_ids"], out["seg_offsets"], out["contrib_count"],
            out["active_count"], out["agg"], out["num_unique"], ws)
    if plan is None:
        gba.gba_aggregate_sparse(*args, err)
    else:
        gba.gba_aggregate_sparse_plan(*args, plan, err)
    res = {k: host(v) for k, v in out.items()}
    res["err"] = int(host(err)[0])
    res["tag"] = host(tag_d) if tag_d is not None else None
    return res


def _check_sparse(res, ids, rows, offsets, w, tokens, step, iota, tag=None, decay="token",
                  norm="per_id_count", expect_exact=False):
    ref = oracle.aggregate_sparse(ids, rows, offsets, w, tokens, step, iota, tag, decay, norm)
    U = ref["num_unique"]
    assert res["err"] == 0
    assert int(res["num_unique"][0]) == U
    assert_exact(res["unique_ids"][:U], ref["unique_ids"], "unique_ids")
    assert_exact(res["seg_offsets"][:U + 1], ref["seg_offsets"], "seg_offsets")
    assert_exact(res["contrib_count"][:U], ref["contrib_count"], "contrib_count")
    assert_exact(res["active_count"][:U], ref["active_count"], "active_count")
    assert_rule_t(res["agg"][:U], ref["agg"], ref["agg_mu"], "agg")
    if expect_exact:
        assert_exact(res["agg"][:U], ref["agg"], "agg (dyadic inputs)")
    if decay == "id_tag":
        assert_exact(res["tag"], ref["new_tag"], "tag")
    return ref


def _case(K, sizes, R, D, seed, zipf_s=1.1, kind=counter.KIND_GRAD, step=1000, stale_hi=5):
    rng = np.random.default_rng(seed)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    from synth.zipf import ZipfRejectionInversion, rank_to_row
    ids = rank_to_row(ZipfRejectionInversion(R, zipf_s).ranks(seed, np.arange(N)) - 1, R) if N else \
        np.zeros(0, np.int64)
    rows = counter.values_range(seed, counter.STREAM_ROWS, 0, N * D, kind,
                                counter.grad_scale(1e-2)).reshape(N, D)
    tokens = step - rng.integers(0, stale_hi + 1, K)
    tag = workload.tag_values(seed, np.arange(R), step) if R <= 50_000_000 else None
    return ids.astype(np.int64), rows, off, tokens, tag


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
@pytest.mark.parametrize("D", [4, 8, 12, 16, 20, 32, 64, 128, 256])
@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_sparse_widths(D, decay, plan):
    K = 7
    sizes = np.array([900, 0, 1733, 17, 1200, 0, 611])
    ids, rows, off, tokens, tag = _case(K, sizes, 3000, D, seed=D)
    w, _, _ = oracle.token_weights(tokens, 1000, 2)
    res = _run_sparse(ids, rows, off, w, tokens, 1000, 2, 3000, tag, decay, plan=plan)
    _check_sparse(res, ids, rows, off, w, tokens, 1000, 2, tag, decay)


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
@pytest.mark.parametrize("norm", ["per_id_count", "by_k"])
@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_sparse_c0_full_size(norm, decay, plan):
    c = BY_NAME["c0"]
    hs = workload.host_step(c, value_kind=counter.KIND_DYADIC)
    w, _, _ = oracle.token_weights(hs.tokens, hs.step, c.iota)
    res = _run_sparse(hs.ids, hs.rows, hs.offsets, w, hs.tokens, hs.step, c.iota, c.R, hs.tags, decay, norm,
                      plan=plan)
    _check_sparse(res, hs.ids, hs.rows, hs.offsets, w, hs.tokens, hs.step, c.iota, hs.tags, decay, norm,
                  expect_exact=True)


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
@pytest.mark.parametrize("D", [4, 32, 256])
def test_sparse_one_hot_id_spans_many_blocks(D, plan):
    """One ID holds most occurrences, so its segment crosses many blocks and
    the per-block partial sums must be joined."""
    K, n = 6, 40_000
    rng = np.random.default_rng(D)
    N = K * n
    ids = np.where(rng.random(N) < 0.7, 4242, rng.integers(0, 10_000, N)).astype(np.int64)
    ids[: n // 2] = 4242                           # a long run inside the first contribution
    off = np.arange(K + 1, dtype=np.int64) * n
    rows = counter.values_range(9, counter.STREAM_ROWS, 0, N * D, counter.KIND_DYADIC).reshape(N, D)
    tokens = 100 - np.array([0, 1, 4, 0, 2, 7])
    w, _, _ = oracle.token_weights(tokens, 100, 3)
    res = _run_sparse(ids, rows, off, w, tokens, 100, 3, 10_000, plan=plan)
    _check_sparse(res, ids, rows, off, w, tokens, 100, 3, expect_exact=True)


@pytest.mark.parametrize("D,tile,short", [(4, 8192, 8), (32, 1024, 8), (256, 128, 4)])
def test_sparse_fixup_chain_lengths(D, tile, short):
    """Segments that run on past their head's row-pass tile by exactly the
    chain length the fix-up sums in one lane group (`short` later tiles), and by
    one and two more, which the whole block sums.  Under 2^23 occurrences a
    row-pass tile holds 32 positions per lane group (4 waves, 64 / (D / 4)
    groups per wave)."""
    K = 3
    nA = short * tile + 1                  # head at position 0, ends at the first position of tile `short`
    nB = (short + 1) * tile                # head in tile `short`, runs on over short + 1 later tiles
    nC = (short + 2) * tile
    rng = np.random.default_rng(D)
    ids = rng.permutation(np.repeat(np.array([5, 9, 13], np.int64), [nA, nB, nC]))
    N = ids.size
    cut = np.sort(rng.choice(np.arange(1, N), K - 1, replace=False))
    off = np.concatenate([[0], cut, [N]]).astype(np.int64)
    rows = counter.values_range(11, counter.STREAM_ROWS, 0, N * D, counter.KIND_DYADIC).reshape(N, D)
    tokens = np.array([50, 49, 47])
    w, _, _ = oracle.token_weights(tokens, 50, 2)
    res = _run_sparse(ids, rows, off, w, tokens, 50, 2, 20)
    ref = _check_sparse(res, ids, rows, off, w, tokens, 50, 2, expect_exact=True)
    assert list(ref["seg_offsets"]) == [0, nA, nA + nB, N]


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
def test_sparse_single_id_everywhere(plan):
    """Every occurrence holds one ID (with the hot-key plan: no cold key at all)."""
    K, n, D = 3, 50_000, 16
    ids = np.full(K * n, 7, np.int64)
    off = np.arange(K + 1, dtype=np.int64) * n
    rows = counter.values_range(4, counter.STREAM_ROWS, 0, K * n * D, counter.KIND_DYADIC).reshape(-1, D)
    tokens = np.array([10, 10, 3])
    w, _, _ = oracle.token_weights(tokens, 10, 2)
    res = _run_sparse(ids, rows, off, w, tokens, 10, 2, 8, plan=plan)
    ref = _check_sparse(res, ids, rows, off, w, tokens, 10, 2, expect_exact=True)
    assert ref["num_unique"] == 1 and list(ref["contrib_count"]) == [3] and list(ref["active_count"]) == [2]


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
def test_sparse_all_distinct(plan):
    """All IDs distinct (with the hot-key plan: no hot ID at all)."""
    K, D, R = 4, 32, 1 << 20
    rng = np.random.default_rng(1)
    ids = rng.permutation(R)[:9999].astype(np.int64)
    off = np.array([0, 2500, 5000, 7500, 9999], np.int64)
    rows = counter.values_range(5, counter.STREAM_ROWS, 0, 9999 * D, counter.KIND_GRAD,
                                counter.grad_scale(1e-2)).reshape(-1, D)
    tokens = np.array([9, 9, 8, 1])
    w, _, _ = oracle.token_weights(tokens, 9, 3)
    res = _run_sparse(ids, rows, off, w, tokens, 9, 3, R, plan=plan)
    ref = _check_sparse(res, ids, rows, off, w, tokens, 9, 3)
    assert ref["num_unique"] == 9999 and np.all(ref["contrib_count"] == 1)


# ID ranges whose key widths select every plan of the ID sort: one to four
# 8-bit digit passes with a first (narrowest) digit of 1, 2, 5 or 8 bits
# (R = 200: 8; 1000: 2+8; 5000: 5+8; 70,000: 1+8+8; 2^21: 5+8+8; 2^26:
# 2+8+8+8; 2^29 - 3: 5+8+8+8; 2^31 + 5: 8+8+8+8).  18,411 occurrences span
# several sort tiles and a ragged last one; dyadic rows make every sum exact,
# so any misplaced key shows.
@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
@pytest.mark.parametrize("R", [200, 1000, 5000, 70_000, 1 << 21, 1 << 26, (1 << 29) - 3, (1 << 31) + 5])
def test_sparse_sort_digit_plans(R, plan):
    K, D = 3, 4
    sizes = np.array([7000, 5000, 6411])
    ids, rows, off, tokens, _ = _case(K, sizes, R, D, seed=R % 997, zipf_s=1.05, kind=counter.KIND_DYADIC)
    assert ids.max() >= R // 2   # the top digit is exercised
    w, _, _ = oracle.token_weights(tokens, 1000, 3)
    res = _run_sparse(ids, rows, off, w, tokens, 1000, 3, R, plan=plan)
    _check_sparse(res, ids, rows, off, w, tokens, 1000, 3, expect_exact=True)


@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_sparse_hot_ids_crowded_in_one_bucket(decay):
    """The hot-key plan with the hot IDs close together in value (rows numbered
    in order of first appearance), so they share one lookup bucket."""
    K, D, R = 6, 16, 1 << 24
    rng = np.random.default_rng(12)
    sizes = np.array([40_000, 0, 25_000, 33_000, 1, 20_000])
    N = int(sizes.sum())
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ids = rng.integers(0, R, N)
    hot = rng.random(N) < 0.6
    ids[hot] = rng.integers(0, 200, int(hot.sum()))
    ids = ids.astype(np.int64)
    rows = counter.values_range(12, counter.STREAM_ROWS, 0, N * D, counter.KIND_DYADIC).reshape(N, D)
    tokens = 1000 - rng.integers(0, 5, K)
    tag = workload.tag_values(12, np.arange(R), 1000)
    w, _, _ = oracle.token_weights(tokens, 1000, 2)
    res = _run_sparse(ids, rows, off, w, tokens, 1000, 2, R, tag, decay, plan=gba.SORT_HOT)
    _check_sparse(res, ids, rows, off, w, tokens, 1000, 2, tag, decay, expect_exact=True)


@pytest.mark.parametrize("K", [256, 300])
@pytest.mark.parametrize("D", [16, 32])
@pytest.mark.parametrize("norm", ["per_id_count", "by_k"])
def test_sparse_means_for_every_count(K, D, norm):
    """ID r lies in contributions 0..r, so the per-ID counts c_r run through
    1..K (through the table of reciprocals when K <= 256, past it when K = 300);
    dyadic rows make the sums exact, so the means match only if every quotient
    is correctly rounded."""
    ids_l, sizes = [], []
    for m in range(K):
        r = np.arange(m, K, dtype=np.int64)
        dup = r[(r + m) % 7 == 0]                 # some IDs twice in one contribution
        part = np.concatenate([r, dup])
        np.random.default_rng(m).shuffle(part)
        ids_l.append(part)
        sizes.append(part.size)
    ids = np.concatenate(ids_l)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = ids.size
    rows = counter.values_range(41, counter.STREAM_ROWS, 0, N * D, counter.KIND_DYADIC, 1.0).reshape(N, D)
    step, iota = 1000, 3
    tokens = step - (np.arange(K) % 6)            # contributions with staleness 4 and 5 are excluded
    w, _, _ = oracle.token_weights(tokens, step, iota)
    for plan in (None, gba.SORT_HOT):
        res = _run_sparse(ids, rows, off, w, tokens, step, iota, K, norm=norm, plan=plan)
        ref = _check_sparse(res, ids, rows, off, w, tokens, step, iota, norm=norm, expect_exact=True)
        assert_exact(ref["contrib_count"], np.arange(1, K + 1, dtype=np.int32), "c_r = r + 1")


def test_sparse_empty():
    K, D = 3, 8
    off = np.zeros(K + 1, np.int64)
    res = _run_sparse(np.zeros(0, np.int64), np.zeros((0, D), np.float32), off, np.ones(K, np.float32),
                      np.array([1, 1, 1]), 1, 0, 100)
    assert int(res["num_unique"][0]) == 0 and int(res["seg_offsets"][0]) == 0 and res["err"] == 0


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
def test_sparse_all_excluded(plan):
    K, sizes, R, D = 5, np.array([300, 200, 0, 50, 450]), 500, 16
    ids, rows, off, tokens, tag = _case(K, sizes, R, D, seed=77, stale_hi=0)
    tokens = tokens - 10                                     # every contribution too stale
    w, _, nex = oracle.token_weights(tokens, 1000, 2)
    assert nex == K
    res = _run_sparse(ids, rows, off, w, tokens, 1000, 2, R, plan=plan)
    ref = _check_sparse(res, ids, rows, off, w, tokens, 1000, 2)
    assert np.all(ref["active_count"] == 0) and np.all(res["agg"][:ref["num_unique"]] == 0)


def test_sparse_table_of_one_row_and_full_32bit_ids():
    K, D = 2, 4
    off = np.array([0, 3000, 7000], np.int64)
    rows = counter.values_range(6, counter.STREAM_ROWS, 0, 7000 * D, counter.KIND_DYADIC).reshape(-1, D)
    tokens = np.array([4, 4])
    w = np.ones(K, np.float32)
    ids = np.zeros(7000, np.int64)
    res = _run_sparse(ids, rows, off, w, tokens, 4, 0, 1)
    _check_sparse(res, ids, rows, off, w, tokens, 4, 0, expect_exact=True)
    R = 1 << 32
    rng = np.random.default_rng(2)
    ids = np.concatenate([rng.integers(0, R, 6000), np.full(1000, R - 1)]).astype(np.int64)
    res = _run_sparse(ids, rows, off, w, tokens, 4, 0, R)
    _check_sparse(res, ids, rows, off, w, tokens, 4, 0, expect_exact=True)


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
def test_sparse_many_small_contributions(plan):
    """4096 tiny contributions: hot IDs run through many of them, and their
    contributions cross the chunks of the hot-key plan."""
    K, D, R = 4096, 8, 5000
    rng = np.random.default_rng(3)
    sizes = rng.integers(0, 6, K)
    ids, rows, off, tokens, tag = _case(K, sizes, R, D, seed=3)
    w, _, _ = oracle.token_weights(tokens, 1000, 3)
    for decay in ("token", "id_tag"):
        res = _run_sparse(ids, rows, off, w, tokens, 1000, 3, R, tag, decay, plan=plan)
        _check_sparse(res, ids, rows, off, w, tokens, 1000, 3, tag, decay)


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
def test_sparse_device_errors(plan):
    K, D, R = 2, 4, 1000
    off = np.array([0, 3, 6], np.int64)
    rows = np.ones((6, D), np.float32)
    ids = np.array([1, 2, 3000, 4, 5, 6], np.int64)         # 3000 is outside [0, R)
    res = _run_sparse(ids, rows, off, np.ones(K, np.float32), np.array([1, 1]), 1, 0, R, plan=plan)
    assert res["err"] & gba.DERR_ID_RANGE
    ids = np.array([1, 2, 3, 4, 5, 6], np.int64)
    res = _run_sparse(ids, rows, np.array([0, 4, 3], np.int64), np.ones(K, np.float32),
                      np.array([1, 1]), 1, 0, R, plan=plan)
    assert res["err"] & gba.DERR_OFFSETS


def test_host_checks_enqueue_nothing():
    with pytest.raises(gba.GBAError):
        gba.gba_aggregate_sparse_workspace_size(10, 2, 6, 100)      # D not a multiple of 4
    with pytest.raises(gba.GBAError):
        gba.gba_aggregate_sparse_workspace_size(10, 0, 8, 100)      # K = 0
    ws = torch.empty(16, dtype=torch.uint8, device=DEV)
    z64 = torch.zeros(8, dtype=torch.int64, device=DEV)
    z32 = torch.zeros(8, dtype=torch.int32, device=DEV)
    with pytest.raises(gba.GBAError):                                  # workspace too small
        gba.gba_aggregate_sparse(z64, torch.zeros((8, 4), device=DEV), torch.tensor([0, 8], device=DEV),
                                 100, torch.ones(1, device=DEV), z64[:1], 0, 0, None, 0, 0, z64,
                                 torch.zeros(9, dtype=torch.int64, device=DEV), z32, z32,
                                 torch.zeros((8, 4), device=DEV), z64[:1], ws)


# ------------------------------------------------------------ optimisers
def dev_at(x, offset):
    """Device copy of x that starts `offset` floats into its allocation."""
    buf = torch.zeros(x.size + offset, dtype=torch.float32, device=DEV)
    view = buf[offset:]
    view.copy_(torch.from_numpy(np.ascontiguousarray(x)))
    return view


@pytest.mark.parametrize("n,offset", [(1, 0), (5, 0), (100_003, 0), (100_003, 1), (64, 3)])
def test_apply_dense_adagrad(n, offset):
    p = counter.values_range(1, 1, 0, n, counter.KIND_PARAM)
    a = counter.values_range(1, 2, 0, n, counter.KIND_ACCUM)
    g = counter.values_range(1, 3, 0, n, counter.KIND_GRAD, counter.grad_scale(1e-2))
    pd, ad = dev_at(p, offset), dev(a)
    gba.gba_apply_adagrad(pd, ad, dev(g), 0.01, 1e-8)
    rp, ra = oracle.adagrad(p, a, g, 0.01, 1e-8)
    mp, ma = oracle.adagrad_magnitude(p, a, g, np.abs(g), 0.01, 1e-8)
    assert_rule_t(host(pd), rp, mp, "param")
    assert_rule_t(host(ad), ra, ma, "accum")


@pytest.mark.parametrize("n,offset", [(1, 0), (7, 0), (100_003, 0), (100_003, 2), (64, 1)])
def test_apply_dense_adam(n, offset):
    p = counter.values_range(2, 1, 0, n, counter.KIND_PARAM)
    m = counter.values_range(2, 2, 0, n, counter.KIND_ADAM_M)
    v = counter.values_range(2, 3, 0, n, counter.KIND_ADAM_V)
    g = counter.values_range(2, 4, 0, n, counter.KIND_GRAD, counter.grad_scale(1e-2))
    pd, md, vd = dev(p), dev(m), dev_at(v, offset)
    gba.gba_apply_adam(pd, md, vd, dev(g), 1e-3, 0.9, 0.999, 1e-8, 1001)
    rp, rm, rv = oracle.adam(p, m, v, g, 1e-3, 0.9, 0.999, 1e-8, 1001)
    mp, mm, mv = oracle.adam_magnitude(p, m, v, g, np.abs(g), 1e-3, 0.9, 0.999, 1e-8, 1001)
    assert_rule_t(host(pd), rp, mp, "param")
    assert_rule_t(host(md), rm, mm, "m")
    assert_rule_t(host(vd), rv, mv, "v")


@pytest.mark.parametrize("opt", ["adagrad", "adam"])
@pytest.mark.parametrize("D", [4, 16, 24, 64, 256])
def test_apply_rows(opt, D):
    R, n = 3000, 1200
    rng = np.random.default_rng(D)
    rows = rng.permutation(R)[:n].astype(np.int64)
    active = (rng.random(n) < 0.8).astype(np.int32)
    count = 1000                                     # entries past the count are ignored
    table = counter.values_range(3, counter.STREAM_TABLE, 0, R * D, counter.KIND_PARAM).reshape(R, D)
    s1 = counter.values_range(3, 5, 0, R * D, counter.KIND_ACCUM if opt == "adagrad" else counter.KIND_ADAM_M).reshape(R, D)
    s2 = counter.values_range(3, 6, 0, R * D, counter.KIND_ADAM_V).reshape(R, D)
    g = counter.values_range(3, 7, 0, n * D, counter.KIND_GRAD, counter.grad_scale(1e-2)).reshape(n, D)
    td, s1d, s2d = dev(table), dev(s1), dev(s2)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    num = torch.tensor([count], dtype=torch.int64, device=DEV)
    if opt == "adagrad":
        gba.gba_apply_adagrad(td, s1d, dev(g), 0.01, 1e-8, rows=dev(rows), active=dev(active), num_rows=num,
                              R=R, err=err)
    else:
        gba.gba_apply_adam(td, s1d, s2d, dev(g), 1e-3, 0.9, 0.999, 1e-8, 7, rows=dev(rows), active=dev(active),
                           num_rows=num, R=R, err=err)
    upd = np.zeros(R, bool)
    sel = np.nonzero(active[:count] > 0)[0]
    upd[rows[sel]] = True
    et, e1, e2 = table.copy(), s1.copy(), s2.copy()
    mt, m1 = None, None
    if opt == "adagrad":
        et[rows[sel]], e1[rows[sel]] = oracle.adagrad(table[rows[sel]], s1[rows[sel]], g[sel], 0.01, 1e-8)
        mt, m1 = np.abs(table).astype(np.float64), np.abs(s1).astype(np.float64)
        mt[rows[sel]], m1[rows[sel]] = oracle.adagrad_magnitude(table[rows[sel]], s1[rows[sel]], g[sel],
                                                                np.abs(g[sel]), 0.01, 1e-8)
    else:
        et[rows[sel]], e1[rows[sel]], e2[rows[sel]] = oracle.adam(table[rows[sel]], s1[rows[sel]], s2[rows[sel]],
                                                                  g[sel], 1e-3, 0.9, 0.999, 1e-8, 7)
        mt, m1, m2 = (np.abs(x).astype(np.float64) for x in (table, s1, s2))
        mt[rows[sel]], m1[rows[sel]], m2[rows[sel]] = oracle.adam_magnitude(
            table[rows[sel]], s1[rows[sel]], s2[rows[sel]], g[sel], np.abs(g[sel]), 1e-3, 0.9, 0.999, 1e-8, 7)
    gt, g1, g2 = host(td), host(s1d), host(s2d)
    assert_exact(gt[~upd], table[~upd], "untouched rows")
    assert_exact(g1[~upd], s1[~upd], "untouched state")
    assert_rule_t(gt, et, mt, "table")
    assert_rule_t(g1, e1, m1, "slot1")
    if opt == "adam":
        assert_rule_t(g2, e2, m2, "slot2")
    assert int(host(err)[0]) == 0


def test_apply_rows_out_of_range_is_reported():
    R, D = 10, 4
    td = torch.zeros((R, D), device=DEV)
    ad = torch.ones((R, D), device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    gba.gba_apply_adagrad(td, ad, torch.ones((2, D), device=DEV), 0.1, 0.0,
                          rows=torch.tensor([3, 10], device=DEV), num_rows=torch.tensor([2], device=DEV),
                          R=R, err=err)
    assert int(host(err)[0]) & gba.DERR_ROW_RANGE
    t = host(td)
    assert np.all(t[3] != 0) and np.all(np.delete(t, 3, axis=0) == 0)


# ------------------------------------------------------------ whole step
@pytest.mark.parametrize("fused", [(True, True), (False, False), (True, False), (False, True)])
@pytest.mark.parametrize("D", [16, 32])
@pytest.mark.parametrize("decay", ["token", "id_tag"])
@pytest.mark.parametrize("opt", ["adagrad", "adam"])
def test_full_step_small(decay, opt, D, fused):
    """The whole step against the oracle, with the dense and the sparse calls
    each fused or separate; D = 32 takes the row pass that applies the rows
    itself, D = 16 the aggregation followed by the row apply."""
    fused_dense, fused_sparse = fused
    c = BY_NAME["c0"].scaled(optimizer=opt, lr=0.01 if opt == "adagrad" else 1e-3, D=D)
    hs = workload.host_step(c)
    stepper = GBAStep(c.K, c.N, c.D, c.R, c.P)
    grads = [dev(g) for g in hs.grads]
    param, table = dev(hs.param), dev(hs.table)
    dslots = [dev(s) for s in hs.dense_slots]
    tslots = [dev(s) for s in hs.table_slots]
    tag = dev(hs.tags)
    stepper.run(tokens=dev(hs.tokens), step=hs.step, iota=c.iota, grads=grads, ids=dev(hs.ids),
                rows=dev(hs.rows), offsets=dev(hs.offsets), param=param, dense_slots=dslots, table=table,
                table_slots=tslots, optimizer=opt, lr=c.lr, eps=c.eps, t=c.adam_t, tag=tag,
                decay=gba.DECAY_ID_TAG if decay == "id_tag" else gba.DECAY_TOKEN, fused_dense=fused_dense,
                fused_sparse=fused_sparse)
    hp = dict(lr=c.lr, eps=c.eps, beta1=c.beta1, beta2=c.beta2)
    ref = oracle.gba_step(hs.tokens, hs.step, c.iota, hs.grads, hs.ids, hs.rows, hs.offsets, hs.param,
                          hs.dense_slots, lambda r: hs.table[r], lambda k, r: hs.table_slots[k][r], opt, hp,
                          tag=hs.tags, decay=decay, t=c.adam_t, magnitudes=True)
    assert int(host(stepper.err)[0]) == 0
    assert_exact(host(stepper.w), ref["w"], "w")
    assert int(host(stepper.num_excluded)[0]) == ref["num_excluded"]
    assert_exact(host(stepper.g_bar), ref["g_bar"], "g_bar")
    assert_rule_t(host(param), ref["param"], ref["param_mu"], "param")
    for k, (s, mu) in enumerate(zip(ref["dense_slots"], ref["dense_slots_mu"])):
        assert_rule_t(host(dslots[k]), s, mu, f"dense slot {k}")
    t_after = host(table)
    act = ref["active_ids"]
    assert_rule_t(t_after[act], ref["table_rows"], ref["table_rows_mu"], "table rows")
    untouched = np.ones(c.R, bool)
    untouched[act] = False
    assert_exact(t_after[untouched], hs.table[untouched], "untouched rows")
    for k, (s, mu) in enumerate(zip(ref["table_slot_rows"], ref["table_slot_rows_mu"])):
        assert_rule_t(host(tslots[k])[act], s, mu, f"table slot {k}")
    if decay == "id_tag":
        assert_exact(host(tag), ref["sparse"]["new_tag"], "tag")


@pytest.mark.parametrize("iota", [np.iinfo(np.int64).max, -1])
@pytest.mark.parametrize("decay", ["token", "id_tag"])
@pytest.mark.parametrize("opt", ["adagrad", "adam"])
def test_eq1_limits_through_the_step(opt, decay, iota):
    """Eq. 1 at its two limits, through the weights and the whole fused step
    (as the benchmark launches it): a threshold above every staleness keeps
    every contribution (the bulk-synchronous limit: every weight 1 and W_r =
    c_r for every ID, in both decay modes), and iota = -1 excludes every
    contribution (no row is applied or re-tagged; the dense update still runs,
    with a zero gradient)."""
    c = BY_NAME["c0"].scaled(optimizer=opt, lr=0.01 if opt == "adagrad" else 1e-3, D=32)
    hs = workload.host_step(c)
    stepper = GBAStep(c.K, c.N, c.D, c.R, c.P)
    grads = [dev(g) for g in hs.grads]
    param, table = dev(hs.param), dev(hs.table)
    dslots = [dev(s) for s in hs.dense_slots]
    tslots = [dev(s) for s in hs.table_slots]
    tag = dev(hs.tags)
    stepper.run(tokens=dev(hs.tokens), step=hs.step, iota=int(iota), grads=grads, ids=dev(hs.ids),
                rows=dev(hs.rows), offsets=dev(hs.offsets), param=param, dense_slots=dslots, table=table,
                table_slots=tslots, optimizer=opt, lr=c.lr, eps=c.eps, t=c.adam_t, tag=tag,
                decay=gba.DECAY_ID_TAG if decay == "id_tag" else gba.DECAY_TOKEN, keep_agg=True)
    hp = dict(lr=c.lr, eps=c.eps, beta1=c.beta1, beta2=c.beta2)
    ref = oracle.gba_step(hs.tokens, hs.step, int(iota), hs.grads, hs.ids, hs.rows, hs.offsets, hs.param,
                          hs.dense_slots, lambda r: hs.table[r], lambda k, r: hs.table_slots[k][r], opt, hp,
                          tag=hs.tags, decay=decay, t=c.adam_t, magnitudes=True)
    keep_all = iota > 0
    assert int(host(stepper.err)[0]) == 0
    assert_exact(host(stepper.w), ref["w"], "w")
    assert_exact(ref["w"], np.full(c.K, 1.0 if keep_all else 0.0, np.float32), "oracle w at the limit")
    assert int(host(stepper.num_excluded)[0]) == ref["num_excluded"] == (0 if keep_all else c.K)
    assert_exact(host(stepper.g_bar), ref["g_bar"], "g_bar")
    assert_rule_t(host(param), ref["param"], ref["param_mu"], "param")
    for k, (s, mu) in enumerate(zip(ref["dense_slots"], ref["dense_slots_mu"])):
        assert_rule_t(host(dslots[k]), s, mu, f"dense slot {k}")
    sp = ref["sparse"]
    U = int(host(stepper.num_unique)[0])
    assert U == sp["num_unique"]
    W = host(stepper.active_count)[:U]
    assert_exact(W, sp["active_count"], "W_r")
    assert_exact(W, sp["contrib_count"] if keep_all else np.zeros(U, np.int32), "W_r at the limit")
    assert_rule_t(host(stepper.agg)[:U], sp["agg"], sp["agg_mu"], "agg")
    t_after = host(table)
    act = ref["active_ids"]
    assert act.size == (U if keep_all else 0)
    if act.size:
        assert_rule_t(t_after[act], ref["table_rows"], ref["table_rows_mu"], "table rows")
        for k, (s, mu) in enumerate(zip(ref["table_slot_rows"], ref["table_slot_rows_mu"])):
            assert_rule_t(host(tslots[k])[act], s, mu, f"table slot {k}")
    untouched = np.ones(c.R, bool)
    untouched[act] = False
    assert_exact(t_after[untouched], hs.table[untouched], "untouched rows")
    if decay == "id_tag":
        assert_exact(host(tag), sp["new_tag"], "tag")


@pytest.mark.parametrize("plan", [None, gba.SORT_HOT])
@pytest.mark.parametrize("D", [8, 32])
def test_sparse_fractional_token_weights(D, plan):
    """Weights other than 0 and 1 (other decay strategies than Eq. 1's) scale
    the rows they weigh; a zero weight still excludes."""
    K = 5
    sizes = np.array([700, 300, 0, 900, 450])
    ids, rows, off, tokens, tag = _case(K, sizes, 800, D, seed=41, kind=counter.KIND_DYADIC)
    w = np.array([1.0, 0.5, 0.0, 0.25, 0.0], np.float32)
    res = _run_sparse(ids, rows, off, w, tokens, 1000, 2, 800, plan=plan)
    _check_sparse(res, ids, rows, off, w, tokens, 1000, 2, expect_exact=True)


# ------------------------------------------ fused sparse aggregate + row apply
def _sparse_step(d_ids, d_rows, d_off, d_w, d_tok, step, iota, R, tag, decay, opt, fused, keep_agg, table0,
                 slots0, norm="per_id_count"):
    """One sparse step on device inputs, fused or as the two separate calls,
    from copies of the given table and state."""
    N, D = d_rows.shape
    K = d_off.numel() - 1
    cap = max(N, 1)
    out = dict(unique_ids=torch.full((cap,), -5, dtype=torch.int64, device=DEV),
               seg_offsets=torch.full((cap + 1,), -5, dtype=torch.int64, device=DEV),
               contrib_count=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
               active_count=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
               agg=torch.full((cap, D), float("nan"), dtype=torch.float32, device=DEV),
               num_unique=torch.full((1,), -5, dtype=torch.int64, device=DEV))
    table = table0.clone()
    slots = [s.clone() for s in slots0]
    tag_d = dev(tag) if decay == "id_tag" else None
    dec = gba.DECAY_ID_TAG if decay == "id_tag" else gba.DECAY_TOKEN
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    lr, eps, b1, b2, t = (0.01, 1e-8, 0.9, 0.999, 1) if opt == "adagrad" else (1e-3, 1e-8, 0.9, 0.999, 1001)
    nrm = gba.NORM_BY_K if norm == "by_k" else gba.NORM_PER_ID_COUNT
    common = (d_ids, d_rows, d_off, R, d_w, d_tok, step, iota, tag_d, dec, nrm,
              out["unique_ids"], out["seg_offsets"], out["contrib_count"], out["active_count"])
    if fused:
        ws = torch.empty(gba.gba_aggregate_apply_sparse_workspace_size(N, K, D, R, opt), dtype=torch.uint8,
                         device=DEV)
        agg = out["agg"] if keep_agg else None
        if opt == "adagrad":
            gba.gba_aggregate_apply_sparse_adagrad(*common, agg, out["num_unique"], table, slots[0], lr, eps, ws, err)
        else:
            gba.gba_aggregate_apply_sparse_adam(*common, agg, out["num_unique"], table, slots[0], slots[1], lr, b1,
                                                b2, eps, t, ws, err)
    else:
        ws = torch.empty(gba.gba_aggregate_sparse_workspace_size(N, K, D, R), dtype=torch.uint8, device=DEV)
        gba.gba_aggregate_sparse(*common, out["agg"], out["num_unique"], ws, err)
        rows_kw = dict(rows=out["unique_ids"], active=out["active_count"], num_rows=out["num_unique"], R=R, err=err)
        if opt == "adagrad":
            gba.gba_apply_adagrad(table, slots[0], out["agg"], lr, eps, **rows_kw)
        else:
            gba.gba_apply_adam(table, slots[0], slots[1], out["agg"], lr, b1, b2, eps, t, **rows_kw)
    torch.cuda.synchronize()
    res = {k: host(v) for k, v in out.items()}
    res.update(table=table, slots=slots, err=int(host(err)[0]), tag=host(tag_d) if tag_d is not None else None)
    return res


def _table_and_state(R, D, opt, seed):
    table = sdev.fill(torch.empty((R, D), dtype=torch.float32, device=DEV), seed, counter.STREAM_TABLE,
                      counter.KIND_PARAM)
    kinds = [counter.KIND_ACCUM] if opt == "adagrad" else [counter.KIND_ADAM_M, counter.KIND_ADAM_V]
    return table, [sdev.fill(torch.empty((R, D), dtype=torch.float32, device=DEV), seed, 90 + i, k)
                   for i, k in enumerate(kinds)]


@pytest.mark.parametrize("keep_agg", [False, True])
@pytest.mark.parametrize("D", [8, 20, 32, 64])
@pytest.mark.parametrize("decay", ["token", "id_tag"])
@pytest.mark.parametrize("opt", ["adagrad", "adam"])
def test_fused_sparse_matches_separate_calls(opt, decay, D, keep_agg):
    """gba_aggregate_apply_sparse_* gives bitwise the table, state and outputs
    of gba_aggregate_sparse followed by the row apply: with Adagrad, D = 20 and
    32 update the rows in the row pass, 8 and 64 aggregate and then apply (as
    Adam does at every width)."""
    K = 12
    sizes = np.random.default_rng(D).integers(0, 12_000, K)
    R = 40_000
    ids, rows, off, tokens, tag = _case(K, sizes, R, D, seed=D + 100)
    step, iota = 1000, 3
    w, _, _ = oracle.token_weights(tokens, step, iota)
    table0, slots0 = _table_and_state(R, D, opt, 5)
    d_in = (dev(ids), dev(rows), dev(off), dev(w), dev(tokens))
    sep = _sparse_step(*d_in, step, iota, R, tag, decay, opt, False, True, table0, slots0)
    fus = _sparse_step(*d_in, step, iota, R, tag, decay, opt, True, keep_agg, table0, slots0)
    assert sep["err"] == 0 and fus["err"] == 0
    U = int(sep["num_unique"][0])
    assert int(fus["num_unique"][0]) == U and U > 1000
    for k in ("unique_ids", "contrib_count", "active_count"):
        assert_exact(fus[k][:U], sep[k][:U], k)
    assert_exact(fus["seg_offsets"][:U + 1], sep["seg_offsets"][:U + 1], "seg_offsets")
    if keep_agg:
        assert_exact(fus["agg"][:U], sep["agg"][:U], "agg")
    assert torch.equal(fus["table"], sep["table"]), "table"
    for i in range(len(slots0)):
        assert torch.equal(fus["slots"][i], sep["slots"][i]), f"state {i}"
    assert not torch.equal(fus["table"], table0)
    if decay == "id_tag":
        assert_exact(fus["tag"], sep["tag"], "tag")


@pytest.mark.parametrize("R", [1, 3])
@pytest.mark.parametrize("D", [20, 32])
def test_fused_sparse_tiny_table(D, R):
    """A table of one or three rows: few, long segments, and at D = 20 lanes past
    the row width, which must read and write nothing outside the table."""
    K = 3
    rng = np.random.default_rng(R * 100 + D)
    sizes = np.array([3000, 11, 5000])
    N = int(sizes.sum())
    ids = rng.integers(0, R, N).astype(np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    rows = counter.values_range(8, counter.STREAM_ROWS, 0, N * D, counter.KIND_DYADIC).reshape(N, D)
    step, iota = 1000, 3
    tokens = np.array([1000, 996, 999])
    w, _, _ = oracle.token_weights(tokens, step, iota)
    table0, slots0 = _table_and_state(R, D, "adagrad", 9)
    d_in = (dev(ids), dev(rows), dev(off), dev(w), dev(tokens))
    sep = _sparse_step(*d_in, step, iota, R, None, "token", "adagrad", False, True, table0, slots0)
    fus = _sparse_step(*d_in, step, iota, R, None, "token", "adagrad", True, True, table0, slots0)
    assert sep["err"] == 0 and fus["err"] == 0
    U = int(sep["num_unique"][0])
    assert int(fus["num_unique"][0]) == U
    assert_exact(fus["agg"][:U], sep["agg"][:U], "agg")
    assert torch.equal(fus["table"], sep["table"]) and torch.equal(fus["slots"][0], sep["slots"][0])


@pytest.mark.parametrize("opt,decay", [("adagrad", "token"), ("adam", "token"), ("adagrad", "id_tag")])
def test_fused_sparse_large_hot_plan(opt, decay):
    """Above the size where the automatic sort plan takes frequent IDs apart:
    the hot IDs' rows are applied where their partial sums are joined."""
    K, n_m, R, D = 8, 600_000, 3_000_000, 32
    N = K * n_m
    rng = np.random.default_rng(77)
    r = rng.zipf(1.1, N).astype(np.int64) % R
    ids = (r * 2654435761 + 12345) % R                      # skewed, scrambled over the table
    off = np.arange(K + 1, dtype=np.int64) * n_m
    step, iota = 1000, 3
    tokens = step - rng.integers(0, 6, K)
    w, _, _ = oracle.token_weights(tokens, step, iota)
    d_rows = sdev.fill(torch.empty((N, D), dtype=torch.float32, device=DEV), 77, counter.STREAM_ROWS,
                       counter.KIND_GRAD, float(counter.grad_scale(1e-2)))
    table0, slots0 = _table_and_state(R, D, opt, 6)
    plain = gba.gba_aggregate_sparse_plan_workspace_size(N, K, D, R, gba.SORT_HOT)
    fused = gba.gba_aggregate_apply_sparse_workspace_size(N, K, D, R, opt)
    assert fused == (plain if opt == "adagrad" else plain + N * D * 4)   # Adam's means go through memory
    tag = workload.tag_values(77, np.arange(R), step) if decay == "id_tag" else None
    d_in = (dev(ids), d_rows, dev(off), dev(w), dev(tokens))
    sep = _sparse_step(*d_in, step, iota, R, tag, decay, opt, False, True, table0, slots0)
    fus = _sparse_step(*d_in, step, iota, R, tag, decay, opt, True, False, table0, slots0)
    assert sep["err"] == 0 and fus["err"] == 0
    U = int(sep["num_unique"][0])
    assert_exact(fus["unique_ids"][:U], sep["unique_ids"][:U], "unique_ids")
    assert_exact(fus["active_count"][:U], sep["active_count"][:U], "active_count")
    assert torch.equal(fus["table"], sep["table"]), "table"
    for i in range(len(slots0)):
        assert torch.equal(fus["slots"][i], sep["slots"][i]), f"state {i}"
    if decay == "id_tag":
        assert_exact(fus["tag"], sep["tag"], "tag")


# ------------------------------------------------ fused dense sum + optimiser
@pytest.mark.parametrize("opt", ["adagrad", "adam"])
@pytest.mark.parametrize("K,P,offset,keep_out", [(1, 1, 0, True), (3, 5, 0, False), (37, 100_003, 0, True),
                                                 (9, 4096 * 16 * 3 + 7, 0, False), (64, 70_001, 1, True),
                                                 (200, 8193, 3, False), (5, 262_144, 0, False)])
def test_fused_dense_matches_separate_calls(opt, K, P, offset, keep_out):
    """The fused call gives bitwise the parameters, state and (if asked) sum of
    gba_aggregate_dense followed by the dense optimiser, aligned or not."""
    rng = np.random.default_rng(K * 7 + P)
    grads = [dev_at(counter.values_range(5, 300 + m, 0, P, counter.KIND_GRAD, counter.grad_scale(1e-2)), offset)
             for m in range(K)]
    tokens = 80 - rng.integers(0, 7, K)
    w, _, _ = oracle.token_weights(tokens, 80, 4)
    table, w_d = gba.pointer_table(grads), dev(w)
    p0 = counter.values_range(6, 1, 0, P, counter.KIND_PARAM)
    kinds = workload.state_kinds(opt)
    s0 = [counter.values_range(6, 2 + k, 0, P, kind) for k, (_, _, kind) in enumerate(kinds)]
    # separate
    pa, sa = dev_at(p0, offset), [dev(x) for x in s0]
    g_bar = torch.empty(P, device=DEV)
    gba.gba_aggregate_dense(table, w_d, P, g_bar)
    if opt == "adagrad":
        gba.gba_apply_adagrad(pa, sa[0], g_bar, 0.01, 1e-8)
    else:
        gba.gba_apply_adam(pa, sa[0], sa[1], g_bar, 1e-3, 0.9, 0.999, 1e-8, 1001)
    # fused
    pb, sb = dev_at(p0, offset), [dev(x) for x in s0]
    out = torch.full((P,), float("nan"), device=DEV) if keep_out else None
    if opt == "adagrad":
        gba.gba_aggregate_apply_dense_adagrad(table, w_d, P, pb, sb[0], 0.01, 1e-8, out=out)
    else:
        gba.gba_aggregate_apply_dense_adam(table, w_d, P, pb, sb[0], sb[1], 1e-3, 0.9, 0.999, 1e-8, 1001, out=out)
    assert_exact(host(pb), host(pa), "param")
    for k in range(len(sa)):
        assert_exact(host(sb[k]), host(sa[k]), f"state {k}")
    if keep_out:
        assert_exact(host(out), host(g_bar), "sum")
    # and the sum itself against the oracle
    g_host = [host(g) for g in grads]
    assert_exact(host(g_bar), oracle.aggregate_dense(g_host, w), "g_bar vs oracle")


def test_fused_dense_host_checks():
    P = 16
    g = [torch.ones(P, device=DEV)]
    table, w = gba.pointer_table(g), torch.ones(1, device=DEV)
    p, a = torch.zeros(P, device=DEV), torch.ones(P, device=DEV)
    L = gba.lib()
    st = torch.cuda.current_stream().cuda_stream
    assert L.gba_aggregate_apply_dense_adagrad(table.data_ptr(), w.data_ptr(), 1, P, None, None, a.data_ptr(),
                                               0.1, 0.0, st) == 1
    assert L.gba_aggregate_apply_dense_adagrad(table.data_ptr(), w.data_ptr(), 0, P, None, p.data_ptr(),
                                               a.data_ptr(), 0.1, 0.0, st) == 2
    assert L.gba_aggregate_apply_dense_adam(table.data_ptr(), w.data_ptr(), 1, P, None, p.data_ptr(), a.data_ptr(),
                                            a.data_ptr(), 1e-3, 0.9, 0.999, 1e-8, 0, st) == 2
    assert L.gba_aggregate_apply_dense_adam(table.data_ptr(), w.data_ptr(), 1, P, None, p.data_ptr(), a.data_ptr(),
                                            None, 1e-3, 0.9, 0.999, 1e-8, 1, st) == 1
    torch.cuda.synchronize()
    assert np.all(host(p) == 0) and np.all(host(a) == 1)


# ------------------------------------------------ early weighted sum (App. B)
@pytest.mark.parametrize("opt", [None, "adagrad", "adam"])
@pytest.mark.parametrize("K,P,groups,offset", [(1, 5, [1], 0), (37, 100_003, [5, 1, 31], 0),
                                               (9, 4096 * 16 * 3 + 7, [3, 3, 3], 0), (64, 70_001, [64], 1),
                                               (200, 8193, [100, 99, 1], 0)])
def test_early_sum_matches_one_shot(opt, K, P, groups, offset):
    """Folding the contributions in as they arrive, in any grouping into calls,
    gives bitwise the one-shot sum (and parameters and state when the
    optimiser is applied at the end), and the oracle's running sum."""
    assert sum(groups) == K
    rng = np.random.default_rng(K + P)
    host_g = [counter.values_range(12, 900 + m, 0, P, counter.KIND_GRAD, counter.grad_scale(1e-2)) for m in range(K)]
    tokens = 70 - rng.integers(0, 7, K)
    w, _, _ = oracle.token_weights(tokens, 70, 4)
    grads = [dev_at(g if w[m] != 0 else np.full(P, np.nan, np.float32), offset) for m, g in enumerate(host_g)]
    run = torch.zeros(P, dtype=torch.float64, device=DEV)
    lo = 0
    for n in groups:
        gba.gba_accumulate_dense(gba.pointer_table(grads[lo:lo + n]), dev(w[lo:lo + n]), P, run)
        lo += n
    ref_run = oracle.accumulate_dense(np.zeros(P, np.float64), host_g, w)
    assert_exact(host(run), ref_run, "running sum vs oracle")
    table, w_d = gba.pointer_table(grads), dev(w)
    if opt is None:
        out, one_shot = torch.empty(P, device=DEV), torch.empty(P, device=DEV)
        gba.gba_finalize_dense(run, K, P, out, reset=True)
        gba.gba_aggregate_dense(table, w_d, P, one_shot)
        assert_exact(host(out), host(one_shot), "g_bar vs one-shot")
        assert_exact(host(out), oracle.finalize_dense(ref_run, K), "g_bar vs oracle")
        assert not host(run).any(), "reset leaves the running sum at zero"
        return
    p0 = counter.values_range(13, 1, 0, P, counter.KIND_PARAM)
    kinds = workload.state_kinds(opt)
    s0 = [counter.values_range(13, 2 + k, 0, P, kind) for k, (_, _, kind) in enumerate(kinds)]
    pa, sa, pb, sb = dev(p0), [dev(x) for x in s0], dev(p0), [dev(x) for x in s0]
    out = torch.full((P,), float("nan"), device=DEV)
    if opt == "adagrad":
        gba.gba_finalize_apply_dense_adagrad(run, K, P, pa, sa[0], 0.01, 1e-8, out=out, reset=False)
        gba.gba_aggregate_apply_dense_adagrad(table, w_d, P, pb, sb[0], 0.01, 1e-8)
    else:
        gba.gba_finalize_apply_dense_adam(run, K, P, pa, sa[0], sa[1], 1e-3, 0.9, 0.999, 1e-8, 1001, out=out,
                                          reset=False)
        gba.gba_aggregate_apply_dense_adam(table, w_d, P, pb, sb[0], sb[1], 1e-3, 0.9, 0.999, 1e-8, 1001)
    assert_exact(host(pa), host(pb), "param")
    for k in range(len(sa)):
        assert_exact(host(sa[k]), host(sb[k]), f"state {k}")
    assert_exact(host(out), oracle.finalize_dense(ref_run, K), "g_bar vs oracle")
    assert_exact(host(run), ref_run, "reset=False keeps the running sum")


def test_early_sum_host_checks():
    P = 8
    g = [torch.ones(P, device=DEV)]
    table, w = gba.pointer_table(g), torch.ones(1, device=DEV)
    run = torch.zeros(P, dtype=torch.float64, device=DEV)
    L = gba.lib()
    st = torch.cuda.current_stream().cuda_stream
    assert L.gba_accumulate_dense(table.data_ptr(), w.data_ptr(), 0, P, run.data_ptr(), st) == 2
    assert L.gba_accumulate_dense(table.data_ptr(), w.data_ptr(), 1, P, None, st) == 1
    assert L.gba_finalize_dense(run.data_ptr(), 0, P, run.data_ptr(), 1, st) == 2
    assert L.gba_finalize_apply_dense_adam(run.data_ptr(), 4, P, None, run.data_ptr(), run.data_ptr(), None, 1e-3,
                                           0.9, 0.999, 1e-8, 1, 1, st) == 1
    torch.cuda.synchronize()
    assert not host(run).any()


# ------------------------------------------------ pull side (Alg. 2 pull responder)
def _pull(ids, table_d, R):
    n = ids.size
    D = table_d.shape[1]
    cap = max(n, 1)
    out = dict(u=torch.full((cap,), -5, dtype=torch.int64, device=DEV),
               inv=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
               rows=torch.full((cap, D), float("nan"), device=DEV),
               nu=torch.full((1,), -5, dtype=torch.int64, device=DEV))
    ws = torch.empty(gba.gba_pull_workspace_size(n, R), dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ids_d = dev(ids) if n else torch.empty(0, dtype=torch.int64, device=DEV)
    gba.gba_pull_rows(ids_d, table_d, out["u"], out["inv"], out["rows"], out["nu"], ws, err)
    return {k: host(v) for k, v in out.items()}, int(host(err)[0])


@pytest.mark.parametrize("n,R,D,kind", [(0, 10, 4, "zipf"), (1, 10, 4, "zipf"), (1023, 3000, 16, "zipf"),
                                        (1025, 3000, 32, "zipf"), (256_000, 500_000_000 // 1000, 32, "zipf"),
                                        (70_001, 100_000, 64, "distinct"), (50_000, 50, 256, "zipf"),
                                        (40_000, 1 << 20, 8, "one")])
def test_pull_rows(n, R, D, kind):
    rng = np.random.default_rng(n + D)
    if kind == "zipf":
        from synth.zipf import ZipfRejectionInversion, rank_to_row
        ids = rank_to_row(ZipfRejectionInversion(R, 1.1).ranks(n + 1, np.arange(n)) - 1, R).astype(np.int64) \
            if n else np.zeros(0, np.int64)
    elif kind == "distinct":
        ids = rng.permutation(R)[:n].astype(np.int64)
    else:
        ids = np.full(n, R - 1, np.int64)
    table = counter.values_range(n + 1, counter.STREAM_TABLE, 0, R * D, counter.KIND_PARAM).reshape(R, D)
    got, err = _pull(ids, dev(table), R)
    assert err == 0
    u, inv, rows = oracle.pull_rows(ids, table)
    U = int(got["nu"][0])
    assert U == u.size
    assert_exact(got["u"][:U], u, "unique_ids")
    assert_exact(got["inv"][:n], inv, "inverse")
    assert_exact(got["rows"][:U], rows, "rows")


@pytest.mark.parametrize("n,R,D,s", [(100_000, 1000, 32, 1.1), (1_000_000, 70_000, 16, 0.7),
                                     (1_000_000, 1 << 22, 32, 2.0), (4_500_000, 1 << 22, 4, 1.1),
                                     (4_500_000, 20_000_000, 4, 0.7)])
def test_pull_rows_medium(n, R, D, s):
    """Requests of 0.1 M to 4.5 M IDs (the largest take the hot-key sort plan)
    over tables up to 20 M rows: unique IDs, inverse map and rows equal the
    oracle's."""
    print(f"pull case n={n} R={R} D={D} s={s}", flush=True)
    from synth.zipf import ZipfRejectionInversion, rank_to_row
    ids = rank_to_row(ZipfRejectionInversion(R, s).ranks(n + 3, np.arange(n)) - 1, R).astype(np.int64)
    seed = n + R
    table_d = sdev.fill(torch.empty((R, D), dtype=torch.float32, device=DEV), seed, counter.STREAM_TABLE,
                        counter.KIND_PARAM)
    table = host(table_d)
    for r in np.random.default_rng(seed).integers(0, R, 64):   # the device generator's rows are the host's
        assert_exact(table[r], counter.values_range(seed, counter.STREAM_TABLE, int(r) * D, D, counter.KIND_PARAM),
                     "generated table row")
    got, err = _pull(ids, table_d, R)
    assert err == 0
    u, inv, rows = oracle.pull_rows(ids, table)
    U = int(got["nu"][0])
    assert U == u.size
    assert_exact(got["u"][:U], u, "unique_ids")
    assert_exact(got["inv"][:n], inv, "inverse")
    assert_exact(got["rows"][:U], rows, "rows")


def test_pull_rows_reports_out_of_range_ids():
    R, D = 100, 4
    ids = np.array([3, 100, 7, -1, 3], np.int64)
    _, err = _pull(ids, torch.zeros((R, D), device=DEV), R)
    assert err & gba.DERR_ID_RANGE


def test_pull_rows_host_checks():
    L = gba.lib()
    t = torch.zeros((10, 6), device=DEV)          # D = 6 is not a multiple of 4
    ids = torch.zeros(4, dtype=torch.int64, device=DEV)
    nu = torch.zeros(1, dtype=torch.int64, device=DEV)
    ws = torch.empty(gba.gba_pull_workspace_size(4, 10), dtype=torch.uint8, device=DEV)
    st = torch.cuda.current_stream().cuda_stream
    assert L.gba_pull_rows(ids.data_ptr(), 4, 10, t.data_ptr(), 6, t.data_ptr(), t.data_ptr(), t.data_ptr(),
                           nu.data_ptr(), ws.data_ptr(), ws.numel(), None, st) == 3
    assert L.gba_pull_rows(ids.data_ptr(), 4, 10, t.data_ptr(), 4, None, t.data_ptr(), t.data_ptr(),
                           nu.data_ptr(), ws.data_ptr(), ws.numel(), None, st) == 1
    assert L.gba_pull_rows(ids.data_ptr(), 4, 10, t.data_ptr(), 4, t.data_ptr(), t.data_ptr(), t.data_ptr(),
                           nu.data_ptr(), ws.data_ptr(), 16, None, st) == 4


# ------------------------------------------------ storage keyed by 64-bit IDs
class _HashStore:
    def __init__(self, capacity, max_rows, n_max):
        self.slot_ids = torch.empty(capacity, dtype=torch.int64, device=DEV)
        self.slot_rows = torch.empty(capacity, dtype=torch.int32, device=DEV)
        gba.gba_hash_clear(self.slot_ids, self.slot_rows)
        self.max_rows = max_rows
        self.num_rows = torch.zeros(1, dtype=torch.int64, device=DEV)
        self.row_ids = torch.full((max_rows,), -7, dtype=torch.int64, device=DEV)
        self.ws = torch.empty(gba.gba_hash_workspace_size(n_max), dtype=torch.uint8, device=DEV)
        self.err = torch.zeros(1, dtype=torch.int32, device=DEV)

    def rows_of(self, ids):
        out = torch.full((max(ids.size, 1),), -9, dtype=torch.int64, device=DEV)
        nn = torch.full((1,), -9, dtype=torch.int64, device=DEV)
        gba.gba_hash_find_or_insert(self.slot_ids, self.slot_rows, dev(ids) if ids.size else out[:0], out,
                                    self.num_rows, self.max_rows, self.ws, row_ids=self.row_ids, num_new=nn,
                                    err=self.err)
        return host(out)[:ids.size], int(host(nn)[0])


def _ids64(rng, n, distinct):
    pool = rng.integers(-(2 ** 62), 2 ** 62, distinct, dtype=np.int64) * 2 + 1   # spread over all 64 bits
    pool[pool == gba.EMPTY_ID] = 5                                               # the reserved value
    pool = np.unique(pool)
    hot = rng.random(n) < 0.3
    ids = np.where(hot, pool[0], pool[rng.integers(0, pool.size, n)])
    return ids.astype(np.int64)


@pytest.mark.parametrize("capacity,n,distinct", [(1 << 10, 700, 300), (1 << 16, 50_000, 20_000),
                                                 (1 << 21, 400_000, 700_000)])
def test_hash_find_or_insert(capacity, n, distinct):
    rng = np.random.default_rng(capacity + n)
    ids = _ids64(rng, n, distinct)
    st = _HashStore(capacity, max_rows=n + 10, n_max=2 * n)
    rows, nn = st.rows_of(ids)
    assert int(host(st.err)[0]) == 0
    U = np.unique(ids).size
    assert nn == U and int(host(st.num_rows)[0]) == U
    # one row per distinct ID, rows 0..U-1, and the reverse map agrees
    pairs = np.unique(np.stack([ids, rows]), axis=1)
    assert pairs.shape[1] == U and np.unique(pairs[1]).size == U
    assert rows.min() == 0 and rows.max() == U - 1
    assert_exact(host(st.row_ids)[rows], ids, "row -> ID")
    sid, srow = host(st.slot_ids), host(st.slot_rows)
    assert int((sid != gba.EMPTY_ID).sum()) == U and np.all(srow[sid != gba.EMPTY_ID] >= 0)
    # a second call with old and new IDs: old IDs keep their rows, new ones get the next rows
    more = np.concatenate([ids[: n // 2], rng.integers(2 ** 40, 2 ** 41, n // 3).astype(np.int64)])
    rows2, nn2 = st.rows_of(more)
    assert int(host(st.err)[0]) == 0
    assert_exact(rows2[: n // 2], rows[: n // 2], "rows of known IDs")
    new_ids = np.setdiff1d(more, ids)
    assert nn2 == new_ids.size
    fresh = rows2[np.isin(more, new_ids)]
    assert fresh.min() == U and fresh.max() == U + new_ids.size - 1


def test_hash_full_index_full_pool_and_reserved_id():
    st = _HashStore(16, max_rows=100, n_max=64)
    st.rows_of(np.arange(20, dtype=np.int64) * 7 + 3)
    assert int(host(st.err)[0]) & gba.DERR_TABLE_FULL
    st = _HashStore(64, max_rows=30, n_max=64)
    st.max_rows = 10
    ids = np.repeat(np.arange(20, dtype=np.int64) + 100, 2)
    rows, _ = st.rows_of(ids)
    assert int(host(st.err)[0]) & gba.DERR_TABLE_FULL
    assert int(host(st.num_rows)[0]) == 10 and (rows == -1).sum() == 20
    # the pool grows: the IDs left without a row get the next rows, the others keep theirs
    st.max_rows = 30
    st.err.zero_()
    rows2, nn = st.rows_of(ids)
    assert int(host(st.err)[0]) == 0 and nn == 10
    kept = rows >= 0
    assert_exact(rows2[kept], rows[kept], "rows kept")
    assert_exact(np.unique(rows2[~kept]), np.arange(10, 20), "rows handed out later")
    assert_exact(rows2[0::2], rows2[1::2], "one row per ID")
    assert int(host(st.num_rows)[0]) == 20
    assert_exact(host(st.row_ids)[rows2], ids, "row -> ID")
    rows3, nn3 = st.rows_of(ids[::-1].copy())
    assert int(host(st.err)[0]) == 0 and nn3 == 0
    assert_exact(rows3[::-1], rows2, "rows of a third call")
    st = _HashStore(64, max_rows=10, n_max=64)
    st.rows_of(np.array([4, gba.EMPTY_ID, 4], np.int64))
    assert int(host(st.err)[0]) & gba.DERR_ID_RANGE


def test_hash_rehash_keeps_every_row():
    rng = np.random.default_rng(5)
    ids = _ids64(rng, 3000, 1500)
    st = _HashStore(1 << 12, max_rows=4000, n_max=3000)
    rows, _ = st.rows_of(ids)
    big_ids = torch.empty(1 << 14, dtype=torch.int64, device=DEV)
    big_rows = torch.empty(1 << 14, dtype=torch.int32, device=DEV)
    gba.gba_hash_rehash(st.slot_ids, st.slot_rows, big_ids, big_rows, err=st.err)
    st.slot_ids, st.slot_rows = big_ids, big_rows
    rows2, nn = st.rows_of(ids[::-1].copy())
    assert int(host(st.err)[0]) == 0 and nn == 0
    assert_exact(rows2[::-1], rows, "rows after rehash")


@pytest.mark.parametrize("opt", ["adagrad", "adam"])
def test_hash_backed_push_step(opt):
    """A push step on storage keyed by 64-bit IDs: IDs -> rows, the sparse call
    and the row apply on the pool give, per ID, the oracle's row-indexed step."""
    c = BY_NAME["c0"].scaled(optimizer=opt, lr=0.01 if opt == "adagrad" else 1e-3)
    hs = workload.host_step(c)
    scramble = lambda r: (r.astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15) + np.uint64(12345)).view(np.int64)  # noqa: E731
    ids64 = scramble(hs.ids)
    st = _HashStore(1 << 16, max_rows=c.R, n_max=c.N)
    rows, U = st.rows_of(ids64)
    assert int(host(st.err)[0]) == 0
    uniq = np.unique(hs.ids)
    # the caller initialises the new rows: the values the row-indexed table holds for those IDs
    orig_of_row = np.empty(U, np.int64)
    orig_of_row[rows] = hs.ids
    pool = dev(hs.table[orig_of_row])
    pslots = [dev(s_[orig_of_row]) for s_ in hs.table_slots]
    w, _, _ = oracle.token_weights(hs.tokens, hs.step, c.iota)
    K, N, D = c.K, c.N, c.D
    out_u = torch.empty(N, dtype=torch.int64, device=DEV)
    so = torch.empty(N + 1, dtype=torch.int64, device=DEV)
    cc = torch.empty(N, dtype=torch.int32, device=DEV)
    ww = torch.empty(N, dtype=torch.int32, device=DEV)
    agg = torch.empty((N, D), device=DEV)
    nu = torch.zeros(1, dtype=torch.int64, device=DEV)
    ws = torch.empty(gba.gba_aggregate_sparse_workspace_size(N, K, D, U), dtype=torch.uint8, device=DEV)
    gba.gba_aggregate_sparse(dev(rows), dev(hs.rows), dev(hs.offsets), U, dev(w), dev(hs.tokens), hs.step, c.iota,
                             None, gba.DECAY_TOKEN, gba.NORM_PER_ID_COUNT, out_u, so, cc, ww, agg, nu, ws, st.err)
    if opt == "adagrad":
        gba.gba_apply_adagrad(pool, pslots[0], agg, c.lr, c.eps, rows=out_u, active=ww, num_rows=nu, R=U, err=st.err)
    else:
        gba.gba_apply_adam(pool, pslots[0], pslots[1], agg, c.lr, c.beta1, c.beta2, c.eps, c.adam_t, rows=out_u,
                           active=ww, num_rows=nu, R=U, err=st.err)
    assert int(host(st.err)[0]) == 0
    Ud = int(host(nu)[0])
    assert Ud == uniq.size
    # the distinct rows name exactly the request's distinct IDs
    assert_exact(np.sort(host(st.row_ids)[host(out_u)[:Ud]]), np.sort(scramble(uniq)), "distinct IDs")
    hp = dict(lr=c.lr, eps=c.eps, beta1=c.beta1, beta2=c.beta2)
    ref = oracle.gba_step(hs.tokens, hs.step, c.iota, hs.grads, hs.ids, hs.rows, hs.offsets, hs.param,
                          hs.dense_slots, lambda r: hs.table[r], lambda k, r: hs.table_slots[k][r], opt, hp,
                          t=c.adam_t, magnitudes=True)
    row_of_orig = dict(zip(orig_of_row.tolist(), range(U)))
    act_rows = np.array([row_of_orig[r] for r in ref["active_ids"]])
    assert_rule_t(host(pool)[act_rows], ref["table_rows"], ref["table_rows_mu"], "rows")
    for k, (s_, mu) in enumerate(zip(ref["table_slot_rows"], ref["table_slot_rows_mu"])):
        assert_rule_t(host(pslots[k])[act_rows], s_, mu, f"slot {k}")


# ------------------------------------------------ capture in a HIP graph
@pytest.mark.parametrize("decay", ["token", "id_tag"])
def test_graph_replays_of_a_step_match_eager_steps(decay):
    """Every call of the step is capturable (no allocation, memset or sync
    inside): three replays of a captured step, with eager steps on a twin
    state and synchronisations between them, give bitwise the eager results."""
    c = BY_NAME["c0"].scaled(optimizer="adam", lr=1e-3)
    hs = workload.host_step(c)
    dec = gba.DECAY_ID_TAG if decay == "id_tag" else gba.DECAY_TOKEN

    def state():
        return dict(param=dev(hs.param), dense_slots=[dev(x) for x in hs.dense_slots], table=dev(hs.table),
                    table_slots=[dev(x) for x in hs.table_slots], tag=dev(hs.tags))
    inputs = dict(tokens=dev(hs.tokens), step=hs.step, iota=c.iota, grads=[dev(g) for g in hs.grads],
                  ids=dev(hs.ids), rows=dev(hs.rows), offsets=dev(hs.offsets), optimizer="adam", lr=c.lr,
                  eps=c.eps, t=c.adam_t, decay=dec)
    A, B = state(), state()
    sa, sb = GBAStep(c.K, c.N, c.D, c.R, c.P), GBAStep(c.K, c.N, c.D, c.R, c.P)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        sb.run(**inputs, **B, stream=side)             # first use: pointer table and buffers outside the capture
    sa.run(**inputs, **A)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        sb.run(**inputs, **B, stream=side)
    torch.cuda.synchronize()
    for i in range(3):
        sa.run(**inputs, **A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        U = int(host(sa.num_unique)[0])
        assert int(host(sb.num_unique)[0]) == U
        for name in ("param", "table", "tag"):
            assert torch.equal(A[name], B[name]), (i, name)
        for k in range(2):
            assert torch.equal(A["dense_slots"][k], B["dense_slots"][k]), (i, k)
            assert torch.equal(A["table_slots"][k], B["table_slots"][k]), (i, k)
        assert torch.equal(sa.g_bar, sb.g_bar) and torch.equal(sa.agg[:U], sb.agg[:U]), i
        assert int(host(sa.err)[0]) == 0 and int(host(sb.err)[0]) == 0


def test_graph_replays_of_a_pull_match_eager_pulls():
    R, D, n = 50_000, 32, 30_000
    rng = np.random.default_rng(2)
    ids = dev(rng.integers(0, R, n).astype(np.int64))
    table = dev(counter.values_range(3, counter.STREAM_TABLE, 0, R * D, counter.KIND_PARAM).reshape(R, D))
    ws = torch.empty(gba.gba_pull_workspace_size(n, R), dtype=torch.uint8, device=DEV)
    outs = [dict(u=torch.empty(n, dtype=torch.int64, device=DEV), inv=torch.empty(n, dtype=torch.int32, device=DEV),
                 rows=torch.empty((n, D), device=DEV), nu=torch.zeros(1, dtype=torch.int64, device=DEV))
            for _ in range(2)]
    err = torch.zeros(1, dtype=torch.int32, device=DEV)

    def pull(o, stream=None):
        gba.gba_pull_rows(ids, table, o["u"], o["inv"], o["rows"], o["nu"], ws, err, stream=stream)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        pull(outs[1], stream=side)
    torch.cuda.synchronize()
    for i in range(3):
        for v in outs[1].values():
            v.fill_(-3)
        pull(outs[0])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        U = int(host(outs[0]["nu"])[0])
        assert int(host(outs[1]["nu"])[0]) == U
        assert torch.equal(outs[0]["u"][:U], outs[1]["u"][:U]) and torch.equal(outs[0]["inv"], outs[1]["inv"])
        assert torch.equal(outs[0]["rows"][:U], outs[1]["rows"][:U]), i
    assert int(host(err)[0]) == 0


def test_hash_find_or_insert_empty_request():
    st = _HashStore(64, max_rows=10, n_max=1)
    st.rows_of(np.array([3, 9], np.int64))
    rows, nn = st.rows_of(np.zeros(0, np.int64))
    assert rows.size == 0 and nn == 0
    assert int(host(st.num_rows)[0]) == 2 and int(host(st.err)[0]) == 0


# ------------------------------------------------ randomised shapes (hypothesis)
from hypothesis import HealthCheck, given, settings, strategies as hst   # noqa: E402

# GBA_HYPOTHESIS_SCALE=n runs n times the examples below, drawn at random
# instead of from the fixed derandomised sequence (a longer search for rare
# shapes; the default run stays short and repeatable).
_HYP_SCALE = max(1, int(os.environ.get("GBA_HYPOTHESIS_SCALE", "1")))


def _hyp(n, **kw):
    return settings(max_examples=n * _HYP_SCALE, deadline=None, derandomize=_HYP_SCALE == 1, database=None, **kw)


@_hyp(60, suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(K=hst.integers(1, 12), n_max=hst.integers(0, 3000), R=hst.sampled_from([1, 2, 17, 1000, 70_000, 1 << 20]),
       D=hst.sampled_from([4, 8, 12, 32, 64, 256]), decay=hst.sampled_from(["token", "id_tag"]),
       norm=hst.sampled_from(["per_id_count", "by_k"]), seed=hst.integers(0, 2 ** 31 - 1),
       dyadic=hst.booleans(), zipf_s=hst.sampled_from([0.6, 1.1, 2.0]),
       plan=hst.sampled_from([None, gba.SORT_HOT]))
def test_sparse_random_shapes(K, n_max, R, D, decay, norm, seed, dyadic, zipf_s, plan):
    """Random shapes, empty contributions, tiny and large tables, hot and
    spread IDs: the GPU equals the oracle (exactly on dyadic values)."""
    rng = np.random.default_rng(seed)
    sizes = rng.integers(0, n_max + 1, K)
    sizes[rng.random(K) < 0.2] = 0
    kind = counter.KIND_DYADIC if dyadic else counter.KIND_GRAD
    ids, rows, off, tokens, tag = _case(K, sizes, R, D, seed % 100_000, zipf_s=zipf_s, kind=kind, stale_hi=4)
    w, _, _ = oracle.token_weights(tokens, 1000, 2)
    res = _run_sparse(ids, rows, off, w, tokens, 1000, 2, R, tag if decay == "id_tag" else None, decay, norm,
                      plan=plan)
    _check_sparse(res, ids, rows, off, w, tokens, 1000, 2, tag if decay == "id_tag" else None, decay, norm,
                  expect_exact=dyadic)


@_hyp(8, suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(K=hst.integers(1, 300), n_target=hst.sampled_from([200_000, 700_000, 2_000_000, 4_500_000, 6_000_000]),
       R=hst.sampled_from([1000, 70_000, 1 << 22, 20_000_000, 500_000_000]),
       D=hst.sampled_from([4, 16, 32, 64, 256]), decay=hst.sampled_from(["token", "id_tag"]),
       norm=hst.sampled_from(["per_id_count", "by_k"]), seed=hst.integers(0, 2 ** 31 - 1),
       dyadic=hst.booleans(), zipf_s=hst.sampled_from([0.7, 1.05, 1.2, 2.0]),
       plan=hst.sampled_from([None, gba.SORT_HOT]))
def test_sparse_random_medium_shapes(K, n_target, R, D, decay, norm, seed, dyadic, zipf_s, plan):
    """Random inputs of 0.2 M to 6 M occurrences (many sort tiles, row-pass
    tiles and hot chunks, segments running across tiles, the automatic plan
    turning to hot keys from 2^22 occurrences), uneven and empty
    contributions: the GPU equals the oracle (exactly on dyadic values)."""
    rng = np.random.default_rng(seed)
    n_target = min(n_target, 64_000_000 // D)          # at most 256 MB of rows
    sizes = rng.integers(0, 2 * n_target // K + 2, K)
    sizes[rng.random(K) < 0.2] = 0
    if R > 50_000_000:
        decay = "token"                                 # tags are drawn for tables up to 50 M rows
    kind = counter.KIND_DYADIC if dyadic else counter.KIND_GRAD
    print(f"medium sparse case K={K} N={int(sizes.sum())} R={R} D={D} decay={decay} norm={norm} "
          f"s={zipf_s} plan={plan} seed={seed}", flush=True)
    ids, rows, off, tokens, tag = _case(K, sizes, R, D, seed % 100_000, zipf_s=zipf_s, kind=kind, stale_hi=6)
    iota = 3
    w, _, _ = oracle.token_weights(tokens, 1000, iota)
    res = _run_sparse(ids, rows, off, w, tokens, 1000, iota, R, tag if decay == "id_tag" else None, decay, norm,
                      plan=plan)
    _check_sparse(res, ids, rows, off, w, tokens, 1000, iota, tag if decay == "id_tag" else None, decay, norm,
                  expect_exact=dyadic)


def _fused_vs_separate(K, sizes, R, D, decay, norm, seed, opt, keep_agg):
    """The fused sparse call against the aggregation and the row apply as two
    calls, from the same table and state: outputs, table and state bitwise."""
    ids, rows, off, tokens, tag = _case(K, sizes, R, D, seed % 100_000, stale_hi=4)
    step, iota = 1000, 2
    w, _, _ = oracle.token_weights(tokens, step, iota)
    table0, slots0 = _table_and_state(R, D, opt, seed % 1000)
    d_in = (dev(ids), dev(rows.reshape(-1, D)), dev(off), dev(w), dev(tokens))
    args = (step, iota, R, tag if decay == "id_tag" else None, decay, opt)
    sep = _sparse_step(*d_in, *args, False, True, table0, slots0, norm=norm)
    fus = _sparse_step(*d_in, *args, True, keep_agg, table0, slots0, norm=norm)
    assert sep["err"] == 0 and fus["err"] == 0
    U = int(sep["num_unique"][0])
    assert int(fus["num_unique"][0]) == U
    for k in ("unique_ids", "contrib_count", "active_count"):
        assert_exact(fus[k][:U], sep[k][:U], k)
    assert_exact(fus["seg_offsets"][:U + 1], sep["seg_offsets"][:U + 1], "seg_offsets")
    if keep_agg:
        assert_exact(fus["agg"][:U], sep["agg"][:U], "agg")
    assert torch.equal(fus["table"], sep["table"]), "table"
    for i in range(len(slots0)):
        assert torch.equal(fus["slots"][i], sep["slots"][i]), f"state {i}"
    if decay == "id_tag":
        assert_exact(fus["tag"], sep["tag"], "tag")


@_hyp(40, suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(K=hst.integers(1, 12), n_max=hst.integers(0, 3000), R=hst.sampled_from([1, 2, 17, 1000, 70_000]),
       D=hst.sampled_from([4, 16, 20, 24, 28, 32, 64]), decay=hst.sampled_from(["token", "id_tag"]),
       norm=hst.sampled_from(["per_id_count", "by_k"]), seed=hst.integers(0, 2 ** 31 - 1),
       opt=hst.sampled_from(["adagrad", "adam"]), keep_agg=hst.booleans())
def test_fused_sparse_random_shapes(K, n_max, R, D, decay, norm, seed, opt, keep_agg):
    """Random shapes, empty contributions and tiny tables: the fused sparse call
    gives bitwise the outputs, table and state of the two separate calls."""
    rng = np.random.default_rng(seed)
    sizes = rng.integers(0, n_max + 1, K)
    sizes[rng.random(K) < 0.2] = 0
    _fused_vs_separate(K, sizes, R, D, decay, norm, seed, opt, keep_agg)


@_hyp(6, suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(K=hst.integers(1, 300), n_target=hst.sampled_from([200_000, 700_000, 2_000_000, 4_500_000]),
       R=hst.sampled_from([70_000, 1 << 22, 20_000_000]), D=hst.sampled_from([16, 20, 24, 28, 32, 64]),
       decay=hst.sampled_from(["token", "id_tag"]), norm=hst.sampled_from(["per_id_count", "by_k"]),
       seed=hst.integers(0, 2 ** 31 - 1), opt=hst.sampled_from(["adagrad", "adam"]), keep_agg=hst.booleans())
def test_fused_sparse_random_medium_shapes(K, n_target, R, D, decay, norm, seed, opt, keep_agg):
    """0.2 M to 4.5 M occurrences (the row pass over many tiles, with the rows
    updated as their segments close where Adagrad meets rows of 20 to 32
    floats): the fused call gives bitwise the outputs, table and state of the
    two separate calls."""
    rng = np.random.default_rng(seed)
    n_target = min(n_target, 64_000_000 // D)
    sizes = rng.integers(0, 2 * n_target // K + 2, K)
    sizes[rng.random(K) < 0.2] = 0
    print(f"medium fused case K={K} N={int(sizes.sum())} R={R} D={D} decay={decay} norm={norm} opt={opt} "
          f"keep_agg={keep_agg} seed={seed}", flush=True)
    _fused_vs_separate(K, sizes, R, D, decay, norm, seed, opt, keep_agg)


@_hyp(40, suppress_health_check=[HealthCheck.too_slow])
@given(K=hst.integers(1, 70), P=hst.integers(1, 150_000), offset=hst.sampled_from([0, 0, 1, 3]),
       frac=hst.booleans(), seed=hst.integers(0, 2 ** 31 - 1), J=hst.integers(1, 9),
       opt=hst.sampled_from(["adagrad", "adam"]))
def test_dense_random_shapes(K, P, offset, frac, seed, J, opt):
    """Random K, P, alignment and weights (0/1 or fractional): the one-shot sum
    equals the oracle bitwise; the fused call and the early sum folded J at a
    time give bitwise the same parameters and state as the two separate calls."""
    rng = np.random.default_rng(seed)
    host_g = [counter.values_range(seed % 1000, 400 + m, 0, P, counter.KIND_GRAD, counter.grad_scale(1e-2))
              for m in range(K)]
    w = (rng.random(K) < 0.8).astype(np.float32)
    if frac:
        w *= rng.choice(np.array([0.25, 0.5, 1.0, 2.0], np.float32), K)
    grads = [dev_at(g if w[m] != 0 else np.full(P, np.nan, np.float32), offset) for m, g in enumerate(host_g)]
    table, w_d = gba.pointer_table(grads), dev(w)
    g_bar = torch.empty(P, device=DEV)
    gba.gba_aggregate_dense(table, w_d, P, g_bar)
    assert_exact(host(g_bar), oracle.aggregate_dense(host_g, w), "g_bar")
    p0 = counter.values_range(seed % 1000, 1, 0, P, counter.KIND_PARAM)
    kinds = workload.state_kinds(opt)
    s0 = [counter.values_range(seed % 1000, 2 + k, 0, P, kind) for k, (_, _, kind) in enumerate(kinds)]
    runs = []
    for mode in ("separate", "fused", "early"):
        p, s_ = dev_at(p0, offset), [dev(x) for x in s0]
        if mode == "separate":
            if opt == "adagrad":
                gba.gba_apply_adagrad(p, s_[0], g_bar, 0.01, 1e-8)
            else:
                gba.gba_apply_adam(p, s_[0], s_[1], g_bar, 1e-3, 0.9, 0.999, 1e-8, 7)
        elif mode == "fused":
            if opt == "adagrad":
                gba.gba_aggregate_apply_dense_adagrad(table, w_d, P, p, s_[0], 0.01, 1e-8)
            else:
                gba.gba_aggregate_apply_dense_adam(table, w_d, P, p, s_[0], s_[1], 1e-3, 0.9, 0.999, 1e-8, 7)
        else:
            run = torch.zeros(P, dtype=torch.float64, device=DEV)
            for lo in range(0, K, J):
                gba.gba_accumulate_dense(gba.pointer_table(grads[lo:lo + J]), w_d[lo:lo + J], P, run)
            if opt == "adagrad":
                gba.gba_finalize_apply_dense_adagrad(run, K, P, p, s_[0], 0.01, 1e-8)
            else:
                gba.gba_finalize_apply_dense_adam(run, K, P, p, s_[0], s_[1], 1e-3, 0.9, 0.999, 1e-8, 7)
        runs.append([host(p)] + [host(x) for x in s_])
    for other in runs[1:]:
        for a, b in zip(runs[0], other):
            assert_exact(b, a, "fused / early vs separate")


@_hyp(40, suppress_health_check=[HealthCheck.too_slow])
@given(calls=hst.integers(1, 4), n_max=hst.integers(0, 4000), pool=hst.integers(1, 3000),
       spare=hst.integers(0, 2), clustered=hst.booleans(), seed=hst.integers(0, 2 ** 31 - 1))
def test_hash_random_sequences(calls, n_max, pool, spare, clustered, seed):
    """A sequence of find-or-insert calls against a dictionary model: a known ID
    keeps its row, each call's distinct new IDs take the next rows (one each,
    the same for every occurrence), the count of new IDs and of rows in use
    follow the model, and the reverse map names each row's ID.  The index is
    at most half full; clustered IDs are consecutive values (neighbours in the
    key space, scattered only by the hash)."""
    rng = np.random.default_rng(seed)
    if clustered:
        ids_pool = rng.integers(-(2 ** 62), 2 ** 62) + np.arange(pool, dtype=np.int64)
    else:
        ids_pool = rng.integers(-(2 ** 63), 2 ** 63 - 1, pool, dtype=np.int64)
    ids_pool = np.unique(ids_pool[ids_pool != gba.EMPTY_ID])
    capacity = 1 << (int(2 * ids_pool.size - 1).bit_length() + spare)
    st = _HashStore(capacity, max_rows=ids_pool.size, n_max=max(n_max, 1))
    model = {}
    for _ in range(calls):
        n = int(rng.integers(0, n_max + 1))
        pick = np.where(rng.random(n) < 0.3, 0, rng.integers(0, ids_pool.size, n))   # a frequent ID among the rest
        ids = ids_pool[pick]
        rows, nn = st.rows_of(ids)
        assert int(host(st.err)[0]) == 0
        before = len(model)
        new_ids = [int(x) for x in np.unique(ids) if int(x) not in model]
        assert nn == len(new_ids)
        got = {}
        for x, r in zip(ids.tolist(), rows.tolist()):
            if x in model:
                assert r == model[x], "a known ID kept its row"
            else:
                assert got.setdefault(x, r) == r, "every occurrence of a new ID has one row"
        assert sorted(got.values()) == list(range(before, before + len(new_ids)))
        model.update(got)
        assert int(host(st.num_rows)[0]) == len(model)
    row_ids = host(st.row_ids)
    for x, r in model.items():
        assert int(row_ids[r]) == x
