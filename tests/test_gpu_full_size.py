"""Parity at the five workloads' full sizes, through the same calls and launch
configuration the benchmark times (one GBAStep.run).

Outputs the oracle can produce whole at these sizes are compared whole: the
token weights, the distinct IDs, segment offsets, c_r and W_r.  Float outputs
are compared on samples the oracle computes one by one from regenerated
inputs: dense columns, the hottest IDs (whose segments span thousands of
tiles) plus random IDs, their updated table rows, and rows that must stay
untouched."""
import numpy as np
import pytest
import torch

import oracle
import paper_2205_11048_amd as gba
from compare import assert_exact, assert_rule_t
from paper_2205_11048_amd.step import GBAStep
from synth import counter, device as sdev, workload
from synth.configs import BY_NAME, STEP

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _table_rows(seed, stream, kind, D, r):
    idx = (np.asarray(r, np.int64)[:, None] * D + np.arange(D)[None, :]).reshape(-1)
    return counter.values(seed, stream, idx, kind).reshape(-1, D)


@pytest.mark.parametrize("name,decay", [("c0", "token"), ("c1", "token"), ("c1", "id_tag"), ("c2", "token"),
                                        ("c3", "token"), ("c4", "token")])
def test_full_size(name, decay):
    w = BY_NAME[name]
    ds = sdev.make_device_step(w, with_tags=(decay == "id_tag"))
    seed, D, K = ds.seed, w.D, w.K
    scale = counter.grad_scale(w.grad_sigma)
    st = GBAStep(K, w.N, D, w.R, w.P)
    st.run(tokens=ds.tokens, step=ds.step, iota=w.iota, grads=ds.grads, ids=ds.ids, rows=ds.rows,
           offsets=ds.offsets, param=ds.param, dense_slots=ds.dense_slots, table=ds.table,
           table_slots=ds.table_slots, optimizer=w.optimizer, lr=w.lr, eps=w.eps, beta1=w.beta1,
           beta2=w.beta2, t=w.adam_t, tag=ds.tags,
           decay=gba.DECAY_ID_TAG if decay == "id_tag" else gba.DECAY_TOKEN, keep_agg=True)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0

    # Eq. 1, whole
    rw, rs, rn = oracle.token_weights(ds.tokens_host, STEP, w.iota)
    assert_exact(st.w.cpu().numpy(), rw, "w")
    assert int(st.num_excluded.item()) == rn

    # dedup and counts, whole
    ids = ds.ids_host
    m_of_j = oracle.contribution_of_occurrence(ds.offsets_host)
    U = int(st.num_unique.item())
    uq, so, cc = oracle.dedup_occurrences(ids, m_of_j, K)
    assert U == uq.size
    assert_exact(st.unique_ids[:U].cpu().numpy(), uq, "unique_ids")
    assert_exact(st.seg_offsets[:U + 1].cpu().numpy(), so, "seg_offsets")
    assert_exact(st.contrib_count[:U].cpu().numpy(), cc, "contrib_count")
    tags0 = workload.tag_values(seed, uq, STEP) if decay == "id_tag" else None
    tag_of = tags0[np.searchsorted(uq, ids)].astype(np.int64) if decay == "id_tag" else None
    if decay == "token":
        wj = rw[m_of_j] != 0
    else:
        sj = np.maximum(0, tag_of - ds.tokens_host[m_of_j] + 1)
        wj = sj <= w.iota
    act_pairs = np.unique(ids[wj] * np.int64(K) + m_of_j[wj]) // np.int64(K)
    act = np.bincount(np.searchsorted(uq, act_pairs), minlength=U).astype(np.int32)
    assert_exact(st.active_count[:U].cpu().numpy(), act, "active_count")

    # dense columns, sampled
    rng = np.random.default_rng(7)
    cols = np.unique(np.concatenate([np.arange(min(64, w.P)), np.arange(max(0, w.P - 64), w.P),
                                     rng.integers(0, w.P, 4096)]))
    g_cols = [counter.values(seed, counter.STREAM_DENSE_GRAD_BASE + m, cols, ds.value_kind, scale)
              for m in range(K)]
    g_ref = oracle.aggregate_dense(g_cols, rw)
    assert_exact(st.g_bar.cpu().numpy()[cols], g_ref, "g_bar columns")
    p0 = counter.values(seed, counter.STREAM_DENSE_PARAM, cols, counter.KIND_PARAM)
    kinds = workload.state_kinds(w.optimizer)
    s0 = [counter.values(seed, d_, cols, kind) for d_, _, kind in kinds]
    p_dev = ds.param.cpu().numpy()[cols]
    if w.optimizer == "adagrad":
        rp, ra = oracle.adagrad(p0, s0[0], g_ref, w.lr, w.eps)
        assert_rule_t(p_dev, rp, None, "param")
        assert_rule_t(ds.dense_slots[0].cpu().numpy()[cols], ra, None, "accum")
    else:
        rp, rm, rv = oracle.adam(p0, s0[0], s0[1], g_ref, w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        assert_rule_t(p_dev, rp, None, "param")
        assert_rule_t(ds.dense_slots[0].cpu().numpy()[cols], rm, None, "m")
        assert_rule_t(ds.dense_slots[1].cpu().numpy()[cols], rv, None, "v")

    # embedding rows: the hottest ID, two more of the top 20, and random ones
    counts = np.diff(so)
    order = np.argsort(-counts, kind="stable")
    pick = np.unique(np.concatenate([order[:1], order[1:20][rng.permutation(19)[:2]],
                                     rng.integers(0, U, 300)]))
    sample_ids = uq[pick]
    occ = np.nonzero(np.isin(ids, sample_ids))[0]
    rows_sub = counter.values(seed, counter.STREAM_ROWS,
                              (occ[:, None] * D + np.arange(D)[None, :]).reshape(-1),
                              ds.value_kind, scale).reshape(-1, D)
    tag_arr = None
    if decay == "id_tag":
        tag_arr = np.full(int(sample_ids.max()) + 1, -1, np.int64)
        tag_arr[sample_ids] = workload.tag_values(seed, sample_ids, STEP)
    ref = oracle.aggregate_sparse_occurrences(ids[occ], m_of_j[occ], rows_sub, K, rw, ds.tokens_host, STEP,
                                              w.iota, tag_arr, decay)
    assert_exact(ref["unique_ids"], sample_ids, "sampled ids")
    agg_dev = st.agg[torch.from_numpy(pick).to(st.agg.device)].cpu().numpy()
    assert_rule_t(agg_dev, ref["agg"], ref["agg_mu"], "agg (sampled)")
    assert_exact(st.active_count.cpu().numpy()[pick], ref["active_count"], "W sampled")

    # their table rows after the apply (inactive rows keep their values)
    active = ref["active_count"] > 0
    r_act = sample_ids[active]
    g_act = ref["agg"][active]
    E0 = _table_rows(seed, counter.STREAM_TABLE, counter.KIND_PARAM, D, r_act)
    S0 = [_table_rows(seed, ts, kind, D, r_act) for _, ts, kind in kinds]
    r_t = torch.from_numpy(r_act).to(ds.table.device)
    E_dev = ds.table[r_t].cpu().numpy()
    if w.optimizer == "adagrad":
        re, ra = oracle.adagrad(E0, S0[0], g_act, w.lr, w.eps)
        assert_rule_t(E_dev, re, None, "table rows")
        assert_rule_t(ds.table_slots[0][r_t].cpu().numpy(), ra, None, "table accum")
    else:
        re, rm, rv = oracle.adam(E0, S0[0], S0[1], g_act, w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        assert_rule_t(E_dev, re, None, "table rows")
        assert_rule_t(ds.table_slots[0][r_t].cpu().numpy(), rm, None, "table m")
        assert_rule_t(ds.table_slots[1][r_t].cpu().numpy(), rv, None, "table v")
    inactive = sample_ids[~active]
    if inactive.size:
        assert_exact(ds.table[torch.from_numpy(inactive).to(ds.table.device)].cpu().numpy(),
                     _table_rows(seed, counter.STREAM_TABLE, counter.KIND_PARAM, D, inactive), "inactive rows")
    untouched = rng.integers(0, w.R, 2000)
    untouched = untouched[~np.isin(untouched, uq)]
    assert_exact(ds.table[torch.from_numpy(untouched).to(ds.table.device)].cpu().numpy(),
                 _table_rows(seed, counter.STREAM_TABLE, counter.KIND_PARAM, D, untouched), "untouched rows")
    if decay == "id_tag":
        t_after = ds.tags[torch.from_numpy(sample_ids).to(ds.tags.device)].cpu().numpy()
        exp = np.where(ref["active_count"] > 0, STEP, workload.tag_values(seed, sample_ids, STEP))
        assert_exact(t_after, exp, "tags")
    print(f"{name}/{decay}: K={K} N={w.N} U={U} hottest segment {int(counts[order[0]])} occurrences")
    del ds, st
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_full_size_early_sum(name):
    """The dense sum taken early (J = 16 arriving contributions per call, as the
    benchmark times it) gives bitwise the one-shot fused result at full size;
    the one-shot result is checked against the oracle in test_full_size."""
    w = BY_NAME[name]
    ds = sdev.make_device_step(w)
    st = GBAStep(w.K, w.N, w.D, w.R, w.P)
    gba.gba_token_weights(ds.tokens, ds.step, w.iota, st.w, err=st.err)
    p1, s1 = ds.param.clone(), [x.clone() for x in ds.dense_slots]
    out1, out2 = torch.empty(w.P, device=ds.param.device), torch.empty(w.P, device=ds.param.device)
    run = torch.zeros(w.P, dtype=torch.float64, device=ds.param.device)
    for lo in range(0, w.K, 16):
        gba.gba_accumulate_dense(gba.pointer_table(ds.grads[lo:lo + 16]), st.w[lo:lo + 16], w.P, run)
    if w.optimizer == "adagrad":
        gba.gba_aggregate_apply_dense_adagrad(st.grad_table(ds.grads), st.w, w.P, p1, s1[0], w.lr, w.eps, out=out1)
        gba.gba_finalize_apply_dense_adagrad(run, w.K, w.P, ds.param, ds.dense_slots[0], w.lr, w.eps, out=out2)
    else:
        gba.gba_aggregate_apply_dense_adam(st.grad_table(ds.grads), st.w, w.P, p1, s1[0], s1[1], w.lr, w.beta1,
                                           w.beta2, w.eps, w.adam_t, out=out1)
        gba.gba_finalize_apply_dense_adam(run, w.K, w.P, ds.param, ds.dense_slots[0], ds.dense_slots[1], w.lr,
                                          w.beta1, w.beta2, w.eps, w.adam_t, out=out2)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    assert torch.equal(out1, out2), "g_bar"
    assert torch.equal(p1, ds.param), "param"
    for a, b in zip(s1, ds.dense_slots):
        assert torch.equal(a, b), "state"
    assert int(torch.count_nonzero(run).item()) == 0, "reset"
    del ds, st
    torch.cuda.empty_cache()


def test_full_size_hash_storage():
    """c4 on storage keyed by 64-bit IDs, launched as the benchmark's hash leg
    (index of 2^25 slots, pool of 2^24 rows): per ID, the updated row and
    accumulator equal the row-indexed step's (checked against the oracle in
    test_full_size) to float rounding."""
    w = BY_NAME["c4"]
    ds = sdev.make_device_step(w)
    dev_ = ds.table.device
    st = GBAStep(w.K, w.N, w.D, w.R, w.P)
    gba.gba_token_weights(ds.tokens, ds.step, w.iota, st.w, err=st.err)
    ids64 = ds.ids * (1 << 32) + 7                      # injective for IDs < 2^31, never the reserved value
    cap, pool_rows = 1 << 25, 1 << 24
    slot_ids = torch.empty(cap, dtype=torch.int64, device=dev_)
    slot_rows = torch.empty(cap, dtype=torch.int32, device=dev_)
    gba.gba_hash_clear(slot_ids, slot_rows)
    num_rows = torch.zeros(1, dtype=torch.int64, device=dev_)
    row_ids = torch.full((pool_rows,), -1, dtype=torch.int64, device=dev_)
    rows_of = torch.empty(w.N, dtype=torch.int64, device=dev_)
    hws = torch.empty(gba.gba_hash_workspace_size(w.N), dtype=torch.uint8, device=dev_)
    gba.gba_hash_find_or_insert(slot_ids, slot_rows, ids64, rows_of, num_rows, pool_rows, hws, row_ids=row_ids,
                                err=st.err)
    torch.cuda.synchronize()
    U = int(num_rows.item())
    orig = (row_ids[:U] - 7) >> 32
    pool = torch.zeros((pool_rows, w.D), device=dev_)
    pacc = torch.zeros((pool_rows, w.D), device=dev_)
    pool[:U] = ds.table[orig]                           # the caller initialises the new rows
    pacc[:U] = ds.table_slots[0][orig]
    sws = torch.empty(gba.gba_aggregate_sparse_workspace_size(w.N, w.K, w.D, pool_rows), dtype=torch.uint8,
                      device=dev_)
    gba.gba_aggregate_sparse(rows_of, ds.rows, ds.offsets, pool_rows, st.w, ds.tokens, ds.step, w.iota, None,
                             gba.DECAY_TOKEN, gba.NORM_PER_ID_COUNT, st.unique_ids, st.seg_offsets, st.contrib_count,
                             st.active_count, st.agg, st.num_unique, sws, st.err)
    gba.gba_apply_adagrad(pool, pacc, st.agg, w.lr, w.eps, rows=st.unique_ids, active=st.active_count,
                          num_rows=st.num_unique, R=pool_rows, err=st.err)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    assert int(st.num_unique.item()) == U
    # the row-indexed step on the same inputs
    gba.gba_aggregate_sparse(ds.ids, ds.rows, ds.offsets, w.R, st.w, ds.tokens, ds.step, w.iota, None,
                             gba.DECAY_TOKEN, gba.NORM_PER_ID_COUNT, st.unique_ids, st.seg_offsets, st.contrib_count,
                             st.active_count, st.agg, st.num_unique, st.workspace, st.err)
    gba.gba_apply_adagrad(ds.table, ds.table_slots[0], st.agg, w.lr, w.eps, rows=st.unique_ids,
                          active=st.active_count, num_rows=st.num_unique, R=w.R, err=st.err)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    assert int(st.num_unique.item()) == U
    a, b = pool[:U], ds.table[orig]
    rel = ((a - b).abs() / b.abs().clamp_min(1e-30)).max().item()
    assert rel <= 1e-5, rel
    assert torch.allclose(pacc[:U], ds.table_slots[0][orig], rtol=1e-5, atol=0)
    same = torch.eq(a, b).float().mean().item()
    print(f"hash storage: U={U}, rows bitwise equal: {same:.4%}, max relative difference {rel:.2e}")
    del ds, st, pool, pacc, slot_ids, slot_rows
    torch.cuda.empty_cache()
