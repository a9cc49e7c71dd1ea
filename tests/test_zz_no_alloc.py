"""The sparse call that allocates nothing (gba_aggregate_sparse_noalloc, for
callers that cannot allocate device memory): its outputs equal those of
gba_aggregate_sparse with a caller-provided workspace bit for bit, on two
calls in a row (the second smaller, so it runs on what the first left in
the library's fixed scratch array), and both agree with the oracle; sizes
beyond the array are refused before any device work."""
import numpy as np
import pytest
import torch

import oracle
import paper_2205_11048_amd as gba
from compare import assert_exact, assert_rule_t
from synth import counter, workload
from synth.zipf import ZipfRejectionInversion, rank_to_row

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _inputs(K, N, R, D, seed, step=1000, stale_hi=4):
    rng = np.random.default_rng(seed)
    cuts = np.sort(rng.integers(0, N + 1, K - 1))
    off = np.concatenate([[0], cuts, [N]]).astype(np.int64)
    ids = rank_to_row(ZipfRejectionInversion(R, 1.1).ranks(seed, np.arange(N)) - 1, R).astype(np.int64)
    rows = counter.values_range(seed, counter.STREAM_ROWS, 0, N * D, counter.KIND_GRAD,
                                counter.grad_scale(1e-2)).reshape(N, D)
    tokens = step - rng.integers(0, stale_hi + 1, K)
    tag = workload.tag_values(seed, np.arange(R), step)
    return ids, rows, off, tokens, tag


def _outputs(N, D):
    cap = max(N, 1)
    return dict(unique_ids=torch.full((cap,), -5, dtype=torch.int64, device=DEV),
                seg_offsets=torch.full((cap + 1,), -5, dtype=torch.int64, device=DEV),
                contrib_count=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
                active_count=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
                agg=torch.full((cap, D), float("nan"), dtype=torch.float32, device=DEV),
                num_unique=torch.full((1,), -5, dtype=torch.int64, device=DEV))


def _call(noalloc, ids, rows, off, w, tokens, step, iota, R, tag, decay):
    N, D = rows.shape
    K = len(off) - 1
    out = _outputs(N, D)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    tag_d = _dev(tag) if decay == gba.DECAY_ID_TAG else None
    args = (_dev(ids), _dev(rows), _dev(off), R, _dev(w), _dev(tokens), step, iota, tag_d, decay,
            gba.NORM_PER_ID_COUNT, out["unique_ids"], out["seg_offsets"], out["contrib_count"],
            out["active_count"], out["agg"], out["num_unique"])
    if noalloc:
        gba.gba_aggregate_sparse_noalloc(*args, err)
    else:
        ws = torch.empty(gba.gba_aggregate_sparse_workspace_size(N, K, D, R), dtype=torch.uint8, device=DEV)
        gba.gba_aggregate_sparse(*args, ws, err)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res["err"] = int(err.item())
    res["tag"] = tag_d.cpu().numpy() if tag_d is not None else None
    return res


# (K, N, R, D, decay): the first call fills most of the array, the second is
# smaller and runs on what the first left behind
CALLS = [(64, 1_500_000, 10_000_000, 32, gba.DECAY_TOKEN),
         (9, 20_011, 70_000, 16, gba.DECAY_ID_TAG)]


def test_noalloc_matches_the_workspace_call_on_two_calls_in_a_row():
    step, iota = 1000, 2
    for i, (K, N, R, D, decay) in enumerate(CALLS):
        print(f"noalloc call {i}: K={K} N={N} R={R} D={D} decay={decay}", flush=True)
        assert gba.gba_aggregate_sparse_workspace_size(N, K, D, R) <= gba.NOALLOC_SCRATCH_BYTES
        ids, rows, off, tokens, tag = _inputs(K, N, R, D, seed=17 + i)
        w, _, _ = oracle.token_weights(tokens, step, iota)
        got = _call(True, ids, rows, off, w, tokens, step, iota, R, tag, decay)
        want = _call(False, ids, rows, off, w, tokens, step, iota, R, tag, decay)
        assert got["err"] == 0 and want["err"] == 0
        U = int(want["num_unique"][0])
        assert int(got["num_unique"][0]) == U
        for k in ("unique_ids", "seg_offsets", "contrib_count", "active_count"):
            n = U + 1 if k == "seg_offsets" else U
            assert_exact(got[k][:n], want[k][:n], k)
        assert np.array_equal(got["agg"][:U].view(np.uint32), want["agg"][:U].view(np.uint32)), "agg bits"
        if decay == gba.DECAY_ID_TAG:
            assert_exact(got["tag"], want["tag"], "tag")
        # and both against the oracle
        mode = "id_tag" if decay == gba.DECAY_ID_TAG else "token"
        ref = oracle.aggregate_sparse(ids, rows, off, w, tokens, step, iota, tag if decay else None, mode,
                                      "per_id_count")
        assert U == ref["num_unique"]
        assert_exact(got["unique_ids"][:U], ref["unique_ids"], "unique_ids vs oracle")
        assert_exact(got["seg_offsets"][:U + 1], ref["seg_offsets"], "seg_offsets vs oracle")
        assert_exact(got["contrib_count"][:U], ref["contrib_count"], "c_r vs oracle")
        assert_exact(got["active_count"][:U], ref["active_count"], "W_r vs oracle")
        assert_rule_t(got["agg"][:U], ref["agg"], ref["agg_mu"], "agg vs oracle")
        if decay == gba.DECAY_ID_TAG:
            assert_exact(got["tag"], ref["new_tag"], "tag vs oracle")


def test_noalloc_refuses_sizes_beyond_its_array():
    # D = 256 at just over 2^20 occurrences needs more than the array holds
    K, N, R, D = 4, 1_100_000, 1000, 256
    assert gba.gba_aggregate_sparse_workspace_size(N, K, D, R) > gba.NOALLOC_SCRATCH_BYTES
    ids = torch.zeros(N, dtype=torch.int64, device=DEV)
    rows = torch.zeros((N, D), dtype=torch.float32, device=DEV)
    off = _dev(np.array([0, N, N, N, N], np.int64))
    w = torch.ones(K, dtype=torch.float32, device=DEV)
    tokens = torch.full((K,), 1000, dtype=torch.int64, device=DEV)
    out = _outputs(N, D)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    with pytest.raises(gba.GBAError, match="status 6"):
        gba.gba_aggregate_sparse_noalloc(ids, rows, off, R, w, tokens, 1000, 2, None, gba.DECAY_TOKEN,
                                         gba.NORM_PER_ID_COUNT, out["unique_ids"], out["seg_offsets"],
                                         out["contrib_count"], out["active_count"], out["agg"], out["num_unique"],
                                         err)
    torch.cuda.synchronize()
    assert int(out["num_unique"].item()) == -5, "nothing was enqueued"
    assert int(err.item()) == 0
