"""Parity at the five workloads' full sizes, through the same calls and launch
configuration the benchmark times (one GBAStep.run; at c4 also the
benchmark's leg on storage keyed by 64-bit IDs).

Integer outputs are compared whole: the token weights, the distinct IDs,
segment offsets, c_r, W_r and the per-ID tags.  Every touched row is compared
with the oracle: the per-ID mean of every distinct ID and, for every active
row, the updated table row and its optimiser state (the 1e-5 rule with the
oracle's magnitude companions); inactive rows must be bit-unchanged.  The
oracle takes the distinct IDs a range at a time (every occurrence of an ID
falls in its range), so the host holds one range's rows at once.  Dense
outputs are compared on a sample of columns regenerated on the host, and a
sample of untouched table rows must be bit-unchanged.

The oracle's inputs are the generator's: the contribution rows and the state
of the touched rows are read back from the device buffers the generator
filled, before the step runs, after a sample of them is checked bit for bit
against the generator's host definition."""
import gc

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

FULL = [("c0", "token"), ("c1", "token"), ("c1", "id_tag"), ("c2", "token"), ("c3", "token"),
        ("c4", "token"), ("c4", "id_tag")]
ROW_PARTS = {"c2": 2, "c4": 4}       # ID ranges the oracle takes one at a time
DENSE_SAMPLE = 65536                 # random dense columns (plus both ends)
HASH_LEG = ("c4", "token")           # the workload of the benchmark's hash-storage leg

_HOST = {}    # host-side dedup of one workload's IDs (shared by its decay modes)
_RUN = {}     # one (workload, decay) run at a time: outputs copied to the host


def _table_rows(seed, stream, kind, D, r):
    idx = (np.asarray(r, np.int64)[:, None] * D + np.arange(D)[None, :]).reshape(-1)
    return counter.values(seed, stream, idx, kind).reshape(-1, D)


def _host_ids(name, ds):
    """The oracle's dedup of the whole ID array, and the stable order of the
    occurrences by ID (each range of it is one ID range's occurrences, in
    occurrence order within each ID)."""
    if _HOST.get("name") != name:
        _HOST.clear()
        ids = ds.ids_host
        m_of_j = oracle.contribution_of_occurrence(ds.offsets_host)
        uq, so, cc = oracle.dedup_occurrences(ids, m_of_j, ds.w.K)
        _HOST.update(name=name, ids=ids, m_of_j=m_of_j, uq=uq, so=so, cc=cc,
                     order=np.argsort(ids, kind="stable"))
    return _HOST


def _inverse_odd(a):
    """Inverse of an odd number modulo 2^64 (Newton's iteration)."""
    a %= 1 << 64
    x = a
    for _ in range(6):
        x = (x * (2 - a * x)) % (1 << 64)
    assert (a * x) % (1 << 64) == 1
    return x


def _hash_leg(w, ds, st, h, E0, S0):
    """The benchmark's hash-storage leg on the same inputs: IDs scrambled over
    the 64-bit range, mapped to rows of a pool by find-or-insert, then the
    fused sparse call on the row numbers.  The caller initialises the pool's
    new rows; here each gets the state its ID had before the step.  Returns,
    per distinct ID (ascending), its pool row after the step, the state after
    and W_r."""
    dev_ = ds.table.device
    mult, add = -0x61C8864680B583EB, 12345
    ids64 = ds.ids * mult + add                         # a bijection of the 64-bit range (wraps)
    cap = 1 << max(20, (2 * w.N - 1).bit_length() - 2)
    pool_rows = min(cap // 2, w.R)
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
    assert int(st.err.item()) == 0
    Uh = int(num_rows.item())
    uq = h["uq"]
    assert Uh == uq.size
    # row -> original ID, by undoing the bijection
    rid = row_ids[:Uh].cpu().numpy().astype(np.uint64)
    inv = np.uint64(_inverse_odd(mult))
    with np.errstate(over="ignore"):
        orig = ((rid - np.uint64(add)) * inv).astype(np.int64)
    k_of_row = np.searchsorted(uq, orig)
    assert_exact(uq[np.minimum(k_of_row, uq.size - 1)], orig, "hash rows name the distinct IDs")
    row_of_k = np.empty(uq.size, np.int64)
    row_of_k[k_of_row] = np.arange(Uh)
    # every position's row holds its own ID (a sample)
    js = np.random.default_rng(3).integers(0, w.N, 100_000)
    assert_exact(rows_of[torch.from_numpy(js).to(dev_)].cpu().numpy(), row_of_k[np.searchsorted(uq, h["ids"][js])],
                 "row of each position")
    pool = torch.zeros((pool_rows, w.D), device=dev_)
    pacc = torch.zeros((pool_rows, w.D), device=dev_)
    pool[:Uh] = torch.from_numpy(E0[k_of_row]).to(dev_)
    pacc[:Uh] = torch.from_numpy(S0[0][k_of_row]).to(dev_)
    fused_ws = gba.gba_aggregate_apply_sparse_workspace_size(w.N, w.K, w.D, pool_rows, w.optimizer)
    plain_ws = gba.gba_aggregate_sparse_workspace_size(w.N, w.K, w.D, pool_rows)
    agg = None if fused_ws == plain_ws else st.agg
    sws = torch.empty(fused_ws, dtype=torch.uint8, device=dev_)
    gba.gba_aggregate_apply_sparse_adagrad(rows_of, ds.rows, ds.offsets, pool_rows, st.w, ds.tokens, ds.step, w.iota,
                                           None, gba.DECAY_TOKEN, gba.NORM_PER_ID_COUNT, st.unique_ids,
                                           st.seg_offsets, st.contrib_count, st.active_count, agg, st.num_unique,
                                           pool, pacc, w.lr, w.eps, sws, st.err)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    assert int(st.num_unique.item()) == Uh
    assert_exact(st.unique_ids[:Uh].cpu().numpy(), np.arange(Uh), "hash leg: distinct rows")
    W_of_row = st.active_count[:Uh].cpu().numpy()
    rk = torch.from_numpy(row_of_k).to(dev_)
    out = dict(E1=pool[rk].cpu().numpy(), S1=[pacc[rk].cpu().numpy()], W=W_of_row[row_of_k])
    del slot_ids, slot_rows, rows_of, hws, pool, pacc, sws, row_ids
    return out


def _run(name, decay):
    """Runs the step once on the device and keeps what the parts compare."""
    if _RUN.get("key") == (name, decay):
        return _RUN
    _RUN.clear()
    gc.collect()
    torch.cuda.empty_cache()
    w = BY_NAME[name]
    idt = decay == "id_tag"
    ds = sdev.make_device_step(w, with_tags=idt)
    seed, K, D = ds.seed, w.K, w.D
    h = _host_ids(name, ds)
    uq = h["uq"]
    dev_ = ds.table.device
    uq_t = torch.from_numpy(uq).to(dev_)
    rng = np.random.default_rng(7)
    # state of the touched rows before the step, and every contribution row
    E0 = ds.table[uq_t].cpu().numpy()
    S0 = [s_[uq_t].cpu().numpy() for s_ in ds.table_slots]
    rows_h = ds.rows.cpu().numpy()
    pick = rng.integers(0, uq.size, 4096)
    assert_exact(E0[pick], _table_rows(seed, counter.STREAM_TABLE, counter.KIND_PARAM, D, uq[pick]), "table rows")
    for k, (_, ts, kind) in enumerate(workload.state_kinds(w.optimizer)):
        assert_exact(S0[k][pick], _table_rows(seed, ts, kind, D, uq[pick]), "state rows")
    jp = rng.integers(0, w.N, 4096)
    assert_exact(rows_h[jp], counter.values(seed, counter.STREAM_ROWS, (jp[:, None] * D + np.arange(D)).reshape(-1),
                                            ds.value_kind, counter.grad_scale(w.grad_sigma)).reshape(-1, D), "rows")
    tags0 = workload.tag_values(seed, uq, STEP) if idt else None
    if idt:
        assert_exact(ds.tags[uq_t[pick]].cpu().numpy(), tags0[pick], "tags")
    untouched = rng.integers(0, w.R, 4000)
    untouched = untouched[~np.isin(untouched, uq)][:2000]

    st = GBAStep(K, w.N, D, w.R, w.P)
    st.run(tokens=ds.tokens, step=ds.step, iota=w.iota, grads=ds.grads, ids=ds.ids, rows=ds.rows,
           offsets=ds.offsets, param=ds.param, dense_slots=ds.dense_slots, table=ds.table,
           table_slots=ds.table_slots, optimizer=w.optimizer, lr=w.lr, eps=w.eps, beta1=w.beta1,
           beta2=w.beta2, t=w.adam_t, tag=ds.tags,
           decay=gba.DECAY_ID_TAG if idt else gba.DECAY_TOKEN, keep_agg=True)
    torch.cuda.synchronize()
    Ud = int(st.num_unique.item())
    cols = np.unique(np.concatenate([np.arange(min(64, w.P)), np.arange(max(0, w.P - 64), w.P),
                                     rng.integers(0, w.P, DENSE_SAMPLE)]))
    ct = torch.from_numpy(cols).to(dev_)
    _RUN.update(
        key=(name, decay), w=w, ds_seed=seed, value_kind=ds.value_kind, tokens=ds.tokens_host, idt=idt,
        err=int(st.err.item()), w_dev=st.w.cpu().numpy(), num_excluded=int(st.num_excluded.item()), U=Ud,
        unique_ids=st.unique_ids[:Ud].cpu().numpy(), seg_offsets=st.seg_offsets[:Ud + 1].cpu().numpy(),
        contrib_count=st.contrib_count[:Ud].cpu().numpy(), active_count=st.active_count[:Ud].cpu().numpy(),
        agg=st.agg[:Ud].cpu().numpy(), E0=E0, S0=S0, rows=rows_h, tags0=tags0,
        E1=ds.table[uq_t].cpu().numpy(), S1=[s_[uq_t].cpu().numpy() for s_ in ds.table_slots],
        tags1=ds.tags[uq_t].cpu().numpy() if idt else None,
        cols=cols, g_bar=st.g_bar[ct].cpu().numpy(), param=ds.param[ct].cpu().numpy(),
        dense_slots=[s_[ct].cpu().numpy() for s_ in ds.dense_slots],
        untouched=untouched,
        untouched_after=ds.table[torch.from_numpy(untouched).to(dev_)].cpu().numpy())
    if (name, decay) == HASH_LEG:
        _RUN["hash"] = _hash_leg(w, ds, st, h, E0, S0)
    del ds, st, uq_t
    gc.collect()
    torch.cuda.empty_cache()
    return _RUN


def _cases():
    out = []
    for name, decay in FULL:
        out.append((name, decay, "ids"))
        out += [(name, decay, f"rows{p}") for p in range(ROW_PARTS.get(name, 1))]
        out.append((name, decay, "dense"))
    return out


def _check_ids(r, h):
    w = r["w"]
    assert r["err"] == 0
    rw, _, rn = oracle.token_weights(r["tokens"], STEP, w.iota)
    assert_exact(r["w_dev"], rw, "w")
    assert r["num_excluded"] == rn
    assert r["U"] == h["uq"].size
    assert_exact(r["unique_ids"], h["uq"], "unique_ids")
    assert_exact(r["seg_offsets"], h["so"], "seg_offsets")
    assert_exact(r["contrib_count"], h["cc"], "contrib_count")


def _check_rows(r, h, part, nparts):
    """Every distinct ID of one ID range: W_r, the mean, and for active rows
    the updated row and state (row-indexed table, and the hash leg)."""
    w = r["w"]
    K, D = w.K, w.D
    so, uq, order = h["so"], h["uq"], h["order"]
    U = uq.size
    # ID ranges with about the same number of occurrences
    cut = np.searchsorted(so, np.linspace(0, so[-1], nparts + 1).round().astype(np.int64))
    cut[0], cut[-1] = 0, U
    s_lo, s_hi = int(cut[part]), int(cut[part + 1])
    if s_hi <= s_lo:
        return
    occ = order[so[s_lo]:so[s_hi]]
    rw, _, _ = oracle.token_weights(r["tokens"], STEP, w.iota)
    ids_p = h["ids"][occ]
    tag = None
    if r["idt"]:
        # IDs renumbered by rank (order-preserving), so the tags fit an array of U entries
        ids_p = np.searchsorted(uq, ids_p)
        tag = r["tags0"]
    ref = oracle.aggregate_sparse_occurrences(ids_p, h["m_of_j"][occ], r["rows"][occ], K, rw, r["tokens"], STEP,
                                              w.iota, tag, "id_tag" if r["idt"] else "token")
    sl = slice(s_lo, s_hi)
    assert_exact(ref["unique_ids"], np.arange(s_lo, s_hi) if r["idt"] else uq[sl], "oracle IDs of the range")
    assert_exact(ref["contrib_count"], h["cc"][sl], "c_r")
    assert_exact(r["active_count"][sl], ref["active_count"], "W_r")
    assert_rule_t(r["agg"][sl], ref["agg"], ref["agg_mu"], "per-ID means")
    act = ref["active_count"] > 0
    g, gmu = ref["agg"][act], ref["agg_mu"][act]
    E0, S0 = r["E0"][sl][act], [s_[sl][act] for s_ in r["S0"]]
    if w.optimizer == "adagrad":
        re, ra = oracle.adagrad(E0, S0[0], g, w.lr, w.eps)
        mu = oracle.adagrad_magnitude(E0, S0[0], g, gmu, w.lr, w.eps)
        want = [(re, mu[0], "table rows"), (ra, mu[1], "accumulator rows")]
    else:
        re, rm, rv = oracle.adam(E0, S0[0], S0[1], g, w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        mu = oracle.adam_magnitude(E0, S0[0], S0[1], g, gmu, w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        want = [(re, mu[0], "table rows"), (rm, mu[1], "m rows"), (rv, mu[2], "v rows")]
    legs = [("", r["E1"], r["S1"], None)]
    if "hash" in r:
        legs.append(("hash leg: ", r["hash"]["E1"], r["hash"]["S1"], r["hash"]["W"]))
    for tag_, E1, S1, W in legs:
        if W is not None:
            assert_exact(W[sl], ref["active_count"], tag_ + "W_r")
        got = [E1[sl][act]] + [s_[sl][act] for s_ in S1]
        for x, (ref_x, mu_x, what) in zip(got, want):
            assert_rule_t(x, ref_x, mu_x, tag_ + what)
        # rows with W_r = 0 are not touched
        assert_exact(E1[sl][~act], r["E0"][sl][~act], tag_ + "inactive rows")
        for k, s_ in enumerate(S1):
            assert_exact(s_[sl][~act], r["S0"][k][sl][~act], tag_ + "inactive state")
    if r["idt"]:
        assert_exact(r["tags1"][sl], np.where(act, STEP, r["tags0"][sl]).astype(np.int32), "tags")


def _check_dense(r):
    w = r["w"]
    seed, cols = r["ds_seed"], r["cols"]
    rw, _, _ = oracle.token_weights(r["tokens"], STEP, w.iota)
    scale = counter.grad_scale(w.grad_sigma)
    g_cols = [counter.values(seed, counter.STREAM_DENSE_GRAD_BASE + m, cols, r["value_kind"], scale)
              for m in range(w.K)]
    g_ref = oracle.aggregate_dense(g_cols, rw)
    g_mu = oracle.aggregate_dense_magnitude(g_cols, rw)
    assert_exact(r["g_bar"], g_ref, "g_bar columns")
    p0 = counter.values(seed, counter.STREAM_DENSE_PARAM, cols, counter.KIND_PARAM)
    s0 = [counter.values(seed, d_, cols, kind) for d_, _, kind in workload.state_kinds(w.optimizer)]
    if w.optimizer == "adagrad":
        rp, ra = oracle.adagrad(p0, s0[0], g_ref, w.lr, w.eps)
        mp, ma = oracle.adagrad_magnitude(p0, s0[0], g_ref, g_mu, w.lr, w.eps)
        assert_rule_t(r["param"], rp, mp, "param")
        assert_rule_t(r["dense_slots"][0], ra, ma, "accum")
    else:
        rp, rm, rv = oracle.adam(p0, s0[0], s0[1], g_ref, w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        mp, mm, mv = oracle.adam_magnitude(p0, s0[0], s0[1], g_ref, g_mu, w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        assert_rule_t(r["param"], rp, mp, "param")
        assert_rule_t(r["dense_slots"][0], rm, mm, "m")
        assert_rule_t(r["dense_slots"][1], rv, mv, "v")
    assert_exact(r["untouched_after"], _table_rows(seed, counter.STREAM_TABLE, counter.KIND_PARAM, w.D, r["untouched"]),
                 "untouched rows")


@pytest.mark.parametrize("name,decay,part", _cases())
def test_full_size(name, decay, part):
    r = _run(name, decay)
    h = _HOST
    if part == "ids":
        _check_ids(r, h)
        counts = np.diff(h["so"])
        print(f"{name}/{decay}: K={r['w'].K} N={r['w'].N} U={r['U']} "
              f"hottest segment {int(counts.max())} occurrences")
    elif part.startswith("rows"):
        _check_rows(r, h, int(part[4:]), ROW_PARTS.get(name, 1))
    else:
        _check_dense(r)
    if part == "dense" and (name, decay) == FULL[-1]:
        _RUN.clear()
        _HOST.clear()
        gc.collect()


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


