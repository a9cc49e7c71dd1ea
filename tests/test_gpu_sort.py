"""The ID grouping step on its own (gba_sort_ids): the sorted IDs and the
occurrence index of every sorted entry must equal a stable sort, element for
element, with the plain plan and with the hot-key plan (frequent IDs placed by
the first pass), on skewed, uniform and degenerate inputs, including key
widths that give the hot plan its different digit layouts."""
import numpy as np
import pytest
import torch

import paper_2205_11048_amd as gba

pytestmark = pytest.mark.gpu
DEV = "cuda"


def zipf_ids(rng, n, R, s):
    """Skewed IDs spread over [0, R): a Zipf rank, folded and scrambled."""
    r = rng.zipf(s, n).astype(np.uint64) % np.uint64(R)
    a = np.uint64(2654435761 % R or 1)
    while np.gcd(int(a), R) != 1:
        a += np.uint64(1)
    return ((r * a + np.uint64(12345)) % np.uint64(R)).astype(np.int64)


def run_sort(ids, R, plan):
    n = ids.size
    d_ids = torch.from_numpy(ids).to(DEV)
    keys = torch.empty(max(n, 1), dtype=torch.int32, device=DEV)
    idx = torch.empty(max(n, 1), dtype=torch.int32, device=DEV)
    ws = torch.empty(gba.gba_sort_ids_workspace_size(n, R, plan), dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    gba.gba_sort_ids(d_ids, R, keys, idx, ws, plan=plan, err=err)
    torch.cuda.synchronize()
    return (keys.cpu().numpy()[:n].view(np.uint32), idx.cpu().numpy()[:n].view(np.uint32),
            int(err.cpu().numpy()[0]))


def check(ids, R, plan):
    print(f"sort n={ids.size} R={R} plan={plan}", flush=True)
    keys, idx, err = run_sort(ids, R, plan)
    mapped = np.where((ids >= 0) & (ids < R), ids, 0).astype(np.uint32)
    order = np.argsort(mapped, kind="stable")
    assert np.array_equal(keys, mapped[order]), "sorted keys"
    assert np.array_equal(idx, order.astype(np.uint32)), "occurrence indices (stable order)"
    bad = bool(((ids < 0) | (ids >= R)).any())
    assert bool(err & gba.DERR_ID_RANGE) == bad


@pytest.mark.parametrize("plan", [gba.SORT_PLAIN, gba.SORT_HOT])
@pytest.mark.parametrize("R", [1000, 100_003, 1 << 24, 500_000_000, (1 << 31) - 5])
@pytest.mark.parametrize("n", [1, 7, 2049, 100_003, 1_000_000])
def test_sort_zipf(n, R, plan):
    rng = np.random.default_rng(n * 7 + R % 1000)
    check(zipf_ids(rng, n, R, 1.1), R, plan)


@pytest.mark.parametrize("n", [511 * 4096, 512 * 4096, 512 * 4096 + 1])
def test_sort_tile_order_around_one_round_of_xcd_chunks(n):
    """Passes of 511, 512 and 513 tiles of 4096 keys (and 1022, 1024, 1025 of
    2048 on the first pass): below one round of 8 chunks of 64 tiles the tiles
    are split in eighths over the XCDs, from one round on in chunks, with the
    tiles past the last whole round in order."""
    rng = np.random.default_rng(n)
    check(zipf_ids(rng, n, 1 << 24, 1.1), 1 << 24, gba.SORT_PLAIN)


@pytest.mark.parametrize("plan", [gba.SORT_PLAIN, gba.SORT_HOT, gba.SORT_AUTO])
def test_sort_large_skewed_auto_picks_the_hot_plan(plan):
    # above the size where the automatic plan takes the hot keys apart
    rng = np.random.default_rng(5)
    check(zipf_ids(rng, 4_500_001, 500_000_000, 1.05), 500_000_000, plan)


@pytest.mark.parametrize("kind", ["uniform", "one", "three", "two_hot_rest_cold", "descending"])
@pytest.mark.parametrize("R", [4097, 20_000_000])
def test_sort_hot_plan_degenerate(kind, R):
    rng = np.random.default_rng(11)
    n = 300_001
    if kind == "uniform":          # nothing frequent enough: no hot IDs
        ids = rng.integers(0, R, n)
    elif kind == "one":            # a single ID: every key hot, no cold keys for the later passes
        ids = np.full(n, R // 3, np.int64)
    elif kind == "three":          # the smallest, the largest and a middle ID
        ids = rng.choice(np.array([0, R - 1, R // 2], np.int64), n)
    elif kind == "two_hot_rest_cold":
        ids = rng.integers(0, R, n)
        hot = rng.random(n) < 0.6
        ids[hot] = rng.choice(np.array([7, R - 8], np.int64), int(hot.sum()))
    else:                          # hot IDs below and above every cold one, reversed input order
        ids = np.sort(zipf_ids(rng, n, R, 1.3))[::-1].copy()
    for plan in (gba.SORT_PLAIN, gba.SORT_HOT):
        check(ids.astype(np.int64), R, plan)


def test_sort_hot_plan_with_ids_out_of_range():
    rng = np.random.default_rng(3)
    R = 1 << 20
    ids = zipf_ids(rng, 200_000, R, 1.2)
    ids[::997] = R + 5
    ids[5::1009] = -3
    check(ids, R, gba.SORT_HOT)


def test_sort_plan_is_plain_where_the_key_width_leaves_no_room():
    # 8-bit and 32-bit keys: the hot plan falls back to the plain sort
    rng = np.random.default_rng(2)
    for R in (200, 1 << 32):
        ids = zipf_ids(rng, 50_000, R, 1.1)
        assert gba.gba_sort_ids_workspace_size(50_000, R, gba.SORT_HOT) == \
            gba.gba_sort_ids_workspace_size(50_000, R, gba.SORT_PLAIN)
        check(ids, R, gba.SORT_HOT)


def test_sort_empty():
    keys, idx, err = run_sort(np.zeros(0, np.int64), 100, gba.SORT_HOT)
    assert keys.size == 0 and idx.size == 0 and err == 0


@pytest.mark.parametrize("R", [1 << 24, 500_000_000])
def test_sort_hot_ids_crowded_in_one_bucket(R):
    """Hot IDs close together in value (rows numbered in order of first
    appearance): they share one lookup bucket, searched by halving."""
    rng = np.random.default_rng(8)
    n = 400_000
    ids = rng.integers(0, R, n)
    hot = rng.random(n) < 0.7
    ids[hot] = rng.integers(0, 240, int(hot.sum()))        # 240 hot IDs, all in the first bucket
    check(ids.astype(np.int64), R, gba.SORT_HOT)
