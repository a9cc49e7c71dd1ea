"""Throughput of the GBA push-step on one MI355X.

A step is one pass of the whole path over one global batch of K buffered
contributions: token weights (Eq. 1), dense weighted sum / K, embedding
dedup + decayed weighted sum / c_r (Alg. 2, push responder), and the
optimiser apply on the dense vector and the touched rows.  Inputs are
seeded synthetic recommendation-shaped workloads resident in HBM before the
timed region starts.

Prints ONE JSON line.  `value` is global batches (steps) per second on the
headline workload (c4: K=256 contributions of 256 x 1000 Zipf IDs over a
500M x 32 table, 16M dense parameters, Adagrad); embedding-grad rows/s and
the achieved algorithmic HBM bandwidth against the 8 TB/s peak are reported
beside it, and the same figures for the dense-heavy workload c3 under
`other_workloads`.  The dense sum and the dense optimiser run as one fused
call (`--separate-dense` for two).  Beside the step, each workload also
reports the step with the dense sum taken early as contributions arrive
(`early_weighted_sum`), one worker's pull request looked up once per distinct
ID (`pull`), and the step on storage keyed by 64-bit IDs (`hash_storage`).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--also", default="c3", help="comma list of extra workloads ('' for none)")
    ap.add_argument("--decay", default="token", choices=["token", "id_tag"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (torch), the known-size reference for "
                         "calibrating HBM byte counters")
    ap.add_argument("--overlap", action="store_true",
                    help="run the dense path on a second stream, concurrently with the sparse path")
    ap.add_argument("--separate-dense", action="store_true",
                    help="dense sum and dense optimiser as two calls instead of the fused one")
    ap.add_argument("--separate-sparse", action="store_true",
                    help="sparse aggregation and row apply as two calls instead of the fused one")
    ap.add_argument("--early-sum", default="16",
                    help="comma list of J: also time the step with the dense sum taken early, J arriving "
                         "contributions folded per call ('' for none)")
    ap.add_argument("--no-hash-storage", dest="hash_storage", action="store_false",
                    help="skip the leg that runs the step on storage keyed by 64-bit IDs")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="skip the leg that replays the step from a captured HIP graph")
    ap.add_argument("--step-only", action="store_true",
                    help="time the step only: no early-sum, pull or hash-storage legs (for kernel profiles)")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="time the oracle on 1/S of the workload, scaled by S (default 0: over the whole workload, "
                         "about a minute of host time at c4)")
    ap.add_argument("--no-ceilings", dest="ceilings", action="store_false",
                    help="skip the measurement kernels (read stream, copy stream, random row gathers)")
    return ap.parse_args()


def algorithmic_bytes(w, K_eff, N_act, U, U_act, id_tag):
    """Bytes the step must move at least once (inputs read, state read and
    written, outputs written); sort passes and intermediate round trips are
    overhead and are not counted."""
    S = 1 if w.optimizer == "adagrad" else 2
    dense = K_eff * w.P * 4 + (2 + 2 * S) * w.P * 4
    sparse = (w.N * 8 + N_act * w.D * 4 + U_act * (2 + 2 * S) * w.D * 4 + U * 24)
    if id_tag:
        sparse += U * 4 + U_act * 4
    return dense, sparse


def kernel_source_sha(path):
    with open(os.path.join(ROOT, path), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(kernel, workload_name):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    were taken on the current source of the kernel; else None."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        data = json.load(f)
    e = data.get(f"{kernel}@{workload_name}")
    if not e or e.get("source_sha256_16") != kernel_source_sha(e["source"]):
        return None
    return e["bytes_per_launch"]


def run_workload(name, args, torch, gba_step_mod, sdev, gba):
    from synth.configs import BY_NAME
    w = BY_NAME[name]
    t0 = time.time()
    ds = sdev.make_device_step(w, with_tags=(args.decay == "id_tag"))
    torch.cuda.synchronize()
    setup_s = time.time() - t0
    print(f"[bench] {name}: inputs resident in HBM after {setup_s:.1f} s", file=sys.stderr, flush=True)
    st = gba_step_mod.GBAStep(w.K, w.N, w.D, w.R, w.P)
    decay = gba.DECAY_ID_TAG if args.decay == "id_tag" else gba.DECAY_TOKEN
    stream = torch.cuda.current_stream()
    # the dense path (token weights -> dense sum -> dense apply) runs on its own
    # stream, concurrently with the sparse path; both wait only for the weights
    dstream = torch.cuda.Stream() if args.overlap else stream

    run = None       # float64 running sum of the early weighted sum, allocated on first use
    early_tables = {}

    def dense_early(J, dkw):
        """The dense path with the weighted sum taken early (App. B): K/J calls
        that fold J arriving contributions each, then one finishing call."""
        nonlocal run
        if run is None:
            run = torch.zeros(w.P, dtype=torch.float64, device="cuda")
        if J not in early_tables:
            early_tables[J] = [(lo, gba.pointer_table(ds.grads[lo:lo + J])) for lo in range(0, w.K, J)]
        for lo, tab in early_tables[J]:
            gba.gba_accumulate_dense(tab, st.w[lo:lo + tab.numel()], w.P, run, **dkw)
        if w.optimizer == "adagrad":
            gba.gba_finalize_apply_dense_adagrad(run, w.K, w.P, ds.param, ds.dense_slots[0], w.lr, w.eps, **dkw)
        else:
            gba.gba_finalize_apply_dense_adam(run, w.K, w.P, ds.param, ds.dense_slots[0], ds.dense_slots[1], w.lr,
                                              w.beta1, w.beta2, w.eps, w.adam_t, **dkw)

    def one_step(ev=None, early_J=0, on=None):
        kw = dict(stream=on or stream)
        dkw = dict(stream=on or dstream)
        if ev is not None:
            ev["t0"].record(stream)
        gba.gba_token_weights(ds.tokens, ds.step, w.iota, st.w, st.staleness, st.num_excluded, st.err, **kw)
        if ev is not None:
            ev["t1"].record(stream)
        if args.overlap:
            w_ready = torch.cuda.Event()
            w_ready.record(stream)
            dstream.wait_event(w_ready)
        if ev is not None:
            ev["d0"].record(dstream)
        if early_J:
            dense_early(early_J, dkw)
            if ev is not None:
                ev["d1"].record(dstream)
        elif args.separate_dense:
            gba.gba_aggregate_dense(st.grad_table(ds.grads), st.w, w.P, st.g_bar, **dkw)
            if ev is not None:
                ev["d1"].record(dstream)
            if w.optimizer == "adagrad":
                gba.gba_apply_adagrad(ds.param, ds.dense_slots[0], st.g_bar, w.lr, w.eps, **dkw)
            else:
                gba.gba_apply_adam(ds.param, ds.dense_slots[0], ds.dense_slots[1], st.g_bar, w.lr, w.beta1,
                                   w.beta2, w.eps, w.adam_t, **dkw)
        else:
            # the weighted sum and the dense optimiser in one pass; g_bar is not stored
            if w.optimizer == "adagrad":
                gba.gba_aggregate_apply_dense_adagrad(st.grad_table(ds.grads), st.w, w.P, ds.param,
                                                      ds.dense_slots[0], w.lr, w.eps, **dkw)
            else:
                gba.gba_aggregate_apply_dense_adam(st.grad_table(ds.grads), st.w, w.P, ds.param, ds.dense_slots[0],
                                                   ds.dense_slots[1], w.lr, w.beta1, w.beta2, w.eps, w.adam_t,
                                                   **dkw)
            if ev is not None:
                ev["d1"].record(dstream)
        if ev is not None:
            ev["d2"].record(dstream)
        if ev is not None:
            ev["s0"].record(stream)
        if not args.separate_sparse:
            # one call: the rows are applied as the aggregation finishes them
            # (agg kept only where the row width takes the separate apply)
            agg = None if st.fuses_rows[w.optimizer] else st.agg
            sparse = (ds.ids, ds.rows, ds.offsets, w.R, st.w, ds.tokens, ds.step, w.iota, ds.tags, decay,
                      gba.NORM_PER_ID_COUNT, st.unique_ids, st.seg_offsets, st.contrib_count, st.active_count, agg,
                      st.num_unique)
            if w.optimizer == "adagrad":
                gba.gba_aggregate_apply_sparse_adagrad(*sparse, ds.table, ds.table_slots[0], w.lr, w.eps,
                                                       st.workspace, st.err, **kw)
            else:
                gba.gba_aggregate_apply_sparse_adam(*sparse, ds.table, ds.table_slots[0], ds.table_slots[1], w.lr,
                                                    w.beta1, w.beta2, w.eps, w.adam_t, st.workspace, st.err, **kw)
            if ev is not None:
                ev["s1"].record(stream)
                ev["s2"].record(stream)
            if args.overlap:
                d_done = torch.cuda.Event()
                d_done.record(dstream)
                stream.wait_event(d_done)
            return
        gba.gba_aggregate_sparse(ds.ids, ds.rows, ds.offsets, w.R, st.w, ds.tokens, ds.step, w.iota,
                                 ds.tags, decay, gba.NORM_PER_ID_COUNT, st.unique_ids, st.seg_offsets,
                                 st.contrib_count, st.active_count, st.agg, st.num_unique, st.workspace,
                                 st.err, **kw)
        if ev is not None:
            ev["s1"].record(stream)
        if w.optimizer == "adagrad":
            gba.gba_apply_adagrad(ds.table, ds.table_slots[0], st.agg, w.lr, w.eps, rows=st.unique_ids,
                                  active=st.active_count, num_rows=st.num_unique, R=w.R, err=st.err, **kw)
        else:
            gba.gba_apply_adam(ds.table, ds.table_slots[0], ds.table_slots[1], st.agg, w.lr, w.beta1,
                               w.beta2, w.eps, w.adam_t, rows=st.unique_ids, active=st.active_count,
                               num_rows=st.num_unique, R=w.R, err=st.err, **kw)
        if ev is not None:
            ev["s2"].record(stream)
        if args.overlap:
            d_done = torch.cuda.Event()
            d_done.record(dstream)
            stream.wait_event(d_done)

    full_cpu = args.cpu_sample <= 0 and not args.no_cpu_baseline and name == args.workload
    pre = capture_state(w, ds, torch) if full_cpu else None
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    if int(st.err.item()) != 0:
        raise RuntimeError(f"device error bits {int(st.err.item())}")

    # timed region: K whole steps, no host synchronisation and no events inside
    # (a timing event between two calls makes the queue drain before it)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        one_step()
    end.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    print(f"[bench] {name}: {args.steps} steps timed", file=sys.stderr, flush=True)
    total_ms = start.elapsed_time(end)
    ms = total_ms / args.steps
    # the per-call breakdown: K more steps with an event around every call
    evs = [{k: torch.cuda.Event(enable_timing=True) for k in ("t0", "t1", "d0", "d1", "d2", "s0", "s1", "s2")}
           for _ in range(args.steps)]
    for i in range(args.steps):
        one_step(evs[i])
    torch.cuda.synchronize()
    if args.separate_sparse:
        spans = {"token_weights": ("t0", "t1"), "aggregate_sparse": ("s0", "s1"), "apply_rows": ("s1", "s2")}
    else:
        spans = {"token_weights": ("t0", "t1"), "aggregate_apply_sparse": ("s0", "s1")}
    if args.separate_dense:
        spans.update(aggregate_dense=("d0", "d1"), apply_dense=("d1", "d2"))
    else:
        spans.update(aggregate_apply_dense=("d0", "d1"))
    breakdown = {n: float(np.mean([e[a].elapsed_time(e[b]) for e in evs])) for n, (a, b) in spans.items()}

    # realised sizes (the same every step: the batch is re-applied)
    w_h = st.w.cpu().numpy()
    K_eff = int((w_h != 0).sum())
    m_of_j = np.repeat(np.arange(w.K), np.diff(ds.offsets_host))
    N_act = int((w_h[m_of_j] != 0).sum()) if args.decay == "token" else None
    U = int(st.num_unique.item())
    act = st.active_count[:U]
    U_act = int((act > 0).sum().item())
    if N_act is None:
        N_act = w.N  # upper bound for the per-ID mode (weights differ per row)
    dense_b, sparse_b = algorithmic_bytes(w, K_eff, N_act, U, U_act, args.decay == "id_tag")
    step_gbs = (dense_b + sparse_b) / (ms * 1e-3) / 1e9

    # dominant kernel: the dense reduction, fused with the dense optimiser
    # unless --separate-dense.  A call is one launch, or one launch per round
    # of resident blocks at large P; the figures are per launch (the call's
    # bytes and time over its launches, which split the work evenly but for
    # the last).
    S = 1 if w.optimizer == "adagrad" else 2
    # vectors per thread of the dense kernel: 16 unless P is too small for
    # 16 to give every compute unit a block step (4, else 1)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    nvec = w.P // 4
    vecs = 16 if -(-nvec // (512 * 16)) >= cus else (4 if -(-nvec // (512 * 4)) >= cus else 1)
    if args.separate_dense:
        dense_call_bytes = K_eff * w.P * 4 + w.P * 4
        call_ms = breakdown["aggregate_dense"]
        kname = f"aggregate_dense_kernel<0, false, {vecs}>"
        launches = gba.gba_aggregate_dense_launches(w.P, w.K, gba.DENSE_SUM)
    else:
        dense_call_bytes = K_eff * w.P * 4 + (2 + 2 * S) * w.P * 4
        call_ms = breakdown["aggregate_apply_dense"]
        kname = f"aggregate_dense_kernel<{S}, false, {vecs}>"
        launches = gba.gba_aggregate_dense_launches(w.P, w.K, gba.DENSE_ADAGRAD if S == 1 else gba.DENSE_ADAM)
    dense_kernel_bytes = dense_call_bytes / launches
    dk_ms = call_ms / launches
    dk_gbs = dense_kernel_bytes / (dk_ms * 1e-3) / 1e9
    traffic = measured_traffic(kname, name)
    res = dict(
        workload=name, ms_per_step=ms, wall_ms_per_step=wall_ms / args.steps,
        global_batches_per_s=1000.0 / ms, embedding_grad_rows_per_s=w.N / (ms * 1e-3),
        samples_per_s=w.K * w.B / (ms * 1e-3),
        step_alg_bytes=dense_b + sparse_b, step_alg_gbs=step_gbs, step_frac_of_hbm_peak=step_gbs / HBM_PEAK_GBS,
        breakdown_ms=breakdown, overlap=args.overlap, fused_dense=not args.separate_dense, fused_sparse=not args.separate_sparse, K_eff=K_eff, N=w.N, N_act=N_act, U=U, U_act=U_act, setup_s=setup_s,
        roofline=dict(kernel=kname, bound="hbm", achieved=dk_gbs, peak=HBM_PEAK_GBS,
                      unit="GB/s", frac=dk_gbs / HBM_PEAK_GBS, traffic=traffic,
                      alg_bytes_per_launch=dense_kernel_bytes, avg_launch_ms=dk_ms, launches_per_call=launches),
    )
    # the same step with the dense sum taken early, for each J asked for
    res["early_sum"] = []
    for J in [int(x) for x in args.early_sum.split(",") if x.strip()]:
        for _ in range(2):
            one_step(early_J=J)
        torch.cuda.synchronize()
        n = max(3, args.steps // 2)
        evs = [{k: torch.cuda.Event(enable_timing=True) for k in ("t0", "t1", "d0", "d1", "d2", "s0", "s1", "s2")}
               for _ in range(n)]
        start.record(stream)
        for i in range(n):
            one_step(evs[i], early_J=J)
        end.record(stream)
        torch.cuda.synchronize()
        res["early_sum"].append(dict(
            J=J, calls_per_step=-(-w.K // J) + 1, ms_per_step=start.elapsed_time(end) / n,
            dense_ms=float(np.mean([e["d0"].elapsed_time(e["d1"]) for e in evs])),
            running_sum_bytes=w.P * 8, buffered_gradient_bytes_saved=w.K * w.P * 4 - w.P * 8))
    # the same step captured once in a HIP graph and replayed (no per-launch
    # host work); every library call is capturable: no allocation, memset or
    # synchronisation inside
    if args.graph and not args.overlap:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            one_step(on=side)               # warm the pointer tables outside the capture
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=side):
                one_step(on=side)
        torch.cuda.synchronize()
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        n = max(3, args.steps)
        start.record(stream)
        for _ in range(n):
            g.replay()
        end.record(stream)
        torch.cuda.synchronize()
        res["graph"] = dict(ms_per_step=start.elapsed_time(end) / n)
        del g

    # storage keyed by 64-bit IDs: the same step with the IDs scrambled over the
    # whole 64-bit range and mapped to rows of a pool by the hash index first
    if args.hash_storage:
        res["hash_storage"] = hash_leg(w, ds, st, gba, torch, stream, decay, start, end, max(3, args.steps // 2))

    # the bandwidth of the step's access patterns (measurement kernels)
    if args.ceilings and name == args.workload:
        res["ceilings"] = ceilings(w, ds.table, ds.rows, gba, torch, stream)
        print(f"[bench] {name}: ceilings measured", file=sys.stderr, flush=True)

    if full_cpu:
        res["cpu_baseline"] = cpu_baseline_full(w, ds, pre)
        del pre
        print(f"[bench] {name}: oracle timed over the whole workload", file=sys.stderr, flush=True)

    # pull side: one worker's request (the IDs of one contribution), rows looked
    # up once per distinct ID
    if args.step_only:
        if int(st.err.item()) != 0:
            raise RuntimeError(f"device error bits {int(st.err.item())}")
        del ds, st
        torch.cuda.empty_cache()
        return res
    n_req = int(ds.offsets_host[1] - ds.offsets_host[0])
    req = ds.ids[:n_req]
    pu = torch.empty(n_req, dtype=torch.int64, device="cuda")
    pinv = torch.empty(n_req, dtype=torch.int32, device="cuda")
    prows = torch.empty((n_req, w.D), dtype=torch.float32, device="cuda")
    pnu = torch.zeros(1, dtype=torch.int64, device="cuda")
    pws = torch.empty(gba.gba_pull_workspace_size(n_req, w.R), dtype=torch.uint8, device="cuda")
    for _ in range(3):
        gba.gba_pull_rows(req, ds.table, pu, pinv, prows, pnu, pws, st.err)
    torch.cuda.synchronize()
    n_pull = 20
    start.record(stream)
    for _ in range(n_pull):
        gba.gba_pull_rows(req, ds.table, pu, pinv, prows, pnu, pws, st.err)
    end.record(stream)
    torch.cuda.synchronize()
    pull_ms = start.elapsed_time(end) / n_pull
    # the same request replayed from a captured HIP graph: the 17 small launches
    # of one request then cost no host work
    pg = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(pg, stream=side):
        gba.gba_pull_rows(req, ds.table, pu, pinv, prows, pnu, pws, st.err, stream=side)
    torch.cuda.synchronize()
    for _ in range(3):
        pg.replay()
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(n_pull):
        pg.replay()
    end.record(stream)
    torch.cuda.synchronize()
    pull_graph_ms = start.elapsed_time(end) / n_pull
    del pg
    U_req = int(pnu.item())
    pull_bytes = n_req * 8 + U_req * w.D * 4 * 2 + U_req * 8 + n_req * 4
    res["pull"] = dict(ids_per_request=n_req, distinct=U_req, us_per_request=pull_ms * 1e3,
                       requests_per_s=1e3 / pull_ms, alg_gbs=pull_bytes / (pull_ms * 1e-3) / 1e9,
                       us_per_request_graph=pull_graph_ms * 1e3)
    del pu, pinv, prows, pws
    if int(st.err.item()) != 0:
        raise RuntimeError(f"device error bits {int(st.err.item())}")
    del ds, st
    torch.cuda.empty_cache()
    return res


def hash_leg(w, ds, st, gba, torch, stream, decay, start, end, n):
    """Time the step on storage keyed by 64-bit IDs; after the first step every
    ID is known, so the timed steps look IDs up without inserting."""
    ids64 = ds.ids * -0x61C8864680B583EB + 12345          # a bijection of the 64-bit range
    cap = 1 << max(20, (2 * w.N - 1).bit_length() - 2)   # index for N/2 distinct IDs at load <= 0.5
    slot_ids = torch.empty(cap, dtype=torch.int64, device="cuda")
    slot_rows = torch.empty(cap, dtype=torch.int32, device="cuda")
    gba.gba_hash_clear(slot_ids, slot_rows)
    pool_rows = min(cap // 2, w.R)     # rows of the pool (the table's first rows); index load <= 0.5
    num_rows = torch.zeros(1, dtype=torch.int64, device="cuda")
    rows_of = torch.empty(w.N, dtype=torch.int64, device="cuda")
    hws = torch.empty(gba.gba_hash_workspace_size(w.N), dtype=torch.uint8, device="cuda")
    # the fused sparse call, agg kept only where the means must go through memory
    fused_ws = gba.gba_aggregate_apply_sparse_workspace_size(w.N, w.K, w.D, pool_rows, w.optimizer)
    plain_ws = gba.gba_aggregate_sparse_workspace_size(w.N, w.K, w.D, pool_rows)
    agg = None if fused_ws == plain_ws else st.agg
    sws = torch.empty(plain_ws, dtype=torch.uint8, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]

    def step(e=None):
        gba.gba_token_weights(ds.tokens, ds.step, w.iota, st.w, st.staleness, st.num_excluded, st.err)
        if w.optimizer == "adagrad":
            gba.gba_aggregate_apply_dense_adagrad(st.grad_table(ds.grads), st.w, w.P, ds.param, ds.dense_slots[0],
                                                  w.lr, w.eps)
        else:
            gba.gba_aggregate_apply_dense_adam(st.grad_table(ds.grads), st.w, w.P, ds.param, ds.dense_slots[0],
                                               ds.dense_slots[1], w.lr, w.beta1, w.beta2, w.eps, w.adam_t)
        if e is not None:
            e[0].record(stream)
        gba.gba_hash_find_or_insert(slot_ids, slot_rows, ids64, rows_of, num_rows, pool_rows, hws, err=st.err)
        if e is not None:
            e[1].record(stream)
        sparse = (rows_of, ds.rows, ds.offsets, pool_rows, st.w, ds.tokens, ds.step, w.iota, ds.tags, decay,
                  gba.NORM_PER_ID_COUNT, st.unique_ids, st.seg_offsets, st.contrib_count, st.active_count, agg,
                  st.num_unique)
        if w.optimizer == "adagrad":
            gba.gba_aggregate_apply_sparse_adagrad(*sparse, ds.table, ds.table_slots[0], w.lr, w.eps, sws, st.err)
        else:
            gba.gba_aggregate_apply_sparse_adam(*sparse, ds.table, ds.table_slots[0], ds.table_slots[1], w.lr,
                                                w.beta1, w.beta2, w.eps, w.adam_t, sws, st.err)

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(n):
        step(ev[i])
    end.record(stream)
    torch.cuda.synchronize()
    if int(st.err.item()) != 0:
        raise RuntimeError(f"device error bits {int(st.err.item())} on the hash-storage leg")
    return dict(index_capacity=cap, pool_rows=pool_rows, rows_in_use=int(num_rows.item()),
                ms_per_step=start.elapsed_time(end) / n,
                find_or_insert_ms=float(np.mean([a.elapsed_time(b) for a, b in ev])))


def ceilings(w, table, contrib_rows, gba, torch, stream):
    """Bandwidth of the step's access patterns on this GPU, each from the
    plainest kernel that has it (include/gba_ceilings.h): a 4 GiB stream of
    16-byte non-temporal reads (the dense sum's pattern), a 2 GiB stream copy,
    N gathers of random whole rows of the workload's table, and N/2 gathers of
    random rows of the contribution rows [N][D] (the row passes' pattern, at
    about the hot-ID pass's count and footprint).  Each is timed over 5
    launches per grid size, after one warm-up, for a few grid sizes; the best
    grid is reported."""
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, reps=5):
        fn()
        start.record(stream)
        for _ in range(reps):
            fn()
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / reps

    out = {}
    grids = (1024, 2048, 4096, 8192)
    sink = torch.empty(gba.gba_ceiling_sink_words(max(grids)), dtype=torch.int32, device="cuda")
    src = torch.empty(1 << 30, dtype=torch.float32, device="cuda")        # 4 GiB
    best = min((timed(lambda: gba.gba_ceiling_read(src, sink, b)), b) for b in (512,) + grids)
    nbytes = src.numel() * 4
    out["read_stream"] = dict(bytes=nbytes, blocks=best[1], us=best[0] * 1e3, gbs=nbytes / (best[0] * 1e-3) / 1e9)
    del src
    a = torch.empty(1 << 29, dtype=torch.float32, device="cuda")           # 2 GiB each way
    b_ = torch.empty_like(a)
    best = min((timed(lambda: gba.gba_ceiling_copy(a, b_, b)), b) for b in grids)
    nbytes = a.numel() * 4
    out["copy_stream"] = dict(bytes_read=nbytes, bytes_written=nbytes, blocks=best[1], us=best[0] * 1e3,
                              gbs=2 * nbytes / (best[0] * 1e-3) / 1e9)
    del a, b_
    g = torch.Generator(device="cuda")
    g.manual_seed(2205110480)
    rows = torch.randint(0, w.R, (w.N,), device="cuda", generator=g, dtype=torch.int64)
    best = min((timed(lambda: gba.gba_ceiling_gather_rows(table, rows, sink, b)), b) for b in grids)
    nbytes = w.N * w.D * 4 + w.N * 8
    out["random_row_gather"] = dict(rows=w.N, row_bytes=w.D * 4, table_rows=w.R, bytes=nbytes, blocks=best[1],
                                    us=best[0] * 1e3, gbs=nbytes / (best[0] * 1e-3) / 1e9)
    del rows
    # the row passes' own pattern: half as many random rows as occurrences
    # (about the hot occurrences at c4) from the contribution rows [N][D]
    n_half = max(1, w.N // 2)
    rows = torch.randint(0, w.N, (n_half,), device="cuda", generator=g, dtype=torch.int64)
    gg = grids + (16384,)
    sink = torch.empty(gba.gba_ceiling_sink_words(max(gg)), dtype=torch.int32, device="cuda")
    best = min((timed(lambda: gba.gba_ceiling_gather_rows(contrib_rows, rows, sink, b)), b) for b in gg)
    nbytes = n_half * w.D * 4 + n_half * 8
    out["random_contribution_row_gather"] = dict(rows=n_half, row_bytes=w.D * 4, table_rows=w.N, bytes=nbytes,
                                                 blocks=best[1], us=best[0] * 1e3,
                                                 gbs=nbytes / (best[0] * 1e-3) / 1e9)
    del rows, sink
    torch.cuda.empty_cache()
    return out


def host_cpu():
    """CPU model of this host and the cores this process may run on."""
    model = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        avail = os.cpu_count()
    return dict(cpu_model=model, nproc=os.cpu_count(), cores_available=avail)


class _OracleClock:
    """Wall and process CPU time spent inside oracle calls only."""

    def __init__(self):
        self.wall = 0.0
        self.cpu = 0.0

    def __call__(self, fn, *a, **kw):
        w0, c0 = time.perf_counter(), time.process_time()
        out = fn(*a, **kw)
        self.wall += time.perf_counter() - w0
        self.cpu += time.process_time() - c0
        return out


def cpu_baseline(name, S):
    """The oracle, untuned, on 1/S of the workload (all K contributions, B/S
    samples each, P/S dense parameters), one host thread; the measured time is
    scaled by S to a whole step."""
    import oracle
    from synth import counter, workload
    from synth.configs import BY_NAME, seed_of
    w = BY_NAME[name]
    ws = w.scaled(B=max(1, w.B // S), P=max(1, w.P // S))
    seed = seed_of(name)
    ids = workload.embedding_ids(ws, seed)
    off = workload.contrib_offsets(ws)
    rows = workload.row_values(ws, seed, 0, ws.N)
    grads = np.stack([workload.dense_grad(ws, seed, m) for m in range(ws.K)])
    tok = workload.tokens_from_staleness(workload.staleness_draws(ws, seed))
    param = counter.values_range(seed, counter.STREAM_DENSE_PARAM, 0, ws.P, counter.KIND_PARAM)
    kinds = workload.state_kinds(ws.optimizer)
    dslots = [counter.values_range(seed, ds_, 0, ws.P, kind) for ds_, _, kind in kinds]
    uniq = np.unique(ids)
    trows = {}
    idx = (uniq[:, None] * ws.D + np.arange(ws.D)[None, :]).reshape(-1)
    trows["E"] = counter.values(seed, counter.STREAM_TABLE, idx, counter.KIND_PARAM).reshape(-1, ws.D)
    for k, (_, ts, kind) in enumerate(kinds):
        trows[k] = counter.values(seed, ts, idx, kind).reshape(-1, ws.D)

    def rows_of(r):
        return trows["E"][np.searchsorted(uniq, r)]

    def slot_rows_of(k, r):
        return trows[k][np.searchsorted(uniq, r)]

    hp = dict(lr=ws.lr, eps=ws.eps, beta1=ws.beta1, beta2=ws.beta2)
    clock = _OracleClock()
    clock(oracle.gba_step, tok, 1000, ws.iota, grads, ids, rows, off, param, dslots, rows_of, slot_rows_of,
          ws.optimizer, hp, t=ws.adam_t)
    dt = clock.wall
    full_s = dt * S
    return dict(value=1.0 / full_s, unit="global batches/s", cores=1, kind="oracle",
                sample=f"{name} at 1/{S}: K={ws.K} contributions of B={ws.B} samples x L={ws.L} IDs "
                       f"(N={ws.N}), P={ws.P} dense params, same Zipf law and R; oracle time {dt:.2f} s x {S}",
                seconds_measured=dt, cpu_seconds=clock.cpu, **host_cpu())


def capture_state(w, ds, torch):
    """Host copies of the step's state before any step runs: the dense
    parameters and optimiser slots, and for every distinct ID its table row
    and slot rows (what the oracle reads; the generator's values)."""
    uq = np.unique(ds.ids_host)
    uq_t = torch.from_numpy(uq).to(ds.table.device)
    st = dict(uq=uq, param=ds.param.cpu().numpy(), dslots=[x.cpu().numpy() for x in ds.dense_slots],
              E=ds.table[uq_t].cpu().numpy(), S=[x[uq_t].cpu().numpy() for x in ds.table_slots])
    del uq_t
    return st


def cpu_baseline_full(w, ds, pre, J=16):
    """The oracle, untuned, over the whole workload on one host thread.  Its
    inputs are the ones the device step reads, copied to the host and never
    timed: the contributions as the generator wrote them (gradients, IDs,
    rows) and the state captured before any step ran; only the oracle's calls
    are timed.  The dense gradients arrive J contributions at a time and are
    folded into the float64 running sum by the oracle's early weighted sum
    (App. B), which in buffer order is bit for bit its one-shot sum; the
    embedding part takes all N occurrences at once."""
    import oracle
    from synth.configs import STEP
    clock = _OracleClock()
    t0 = time.perf_counter()
    tok = ds.tokens_host
    wts, _, _ = clock(oracle.token_weights, tok, STEP, w.iota)
    run = np.zeros(w.P, dtype=np.float64)
    for lo in range(0, w.K, J):
        hi = min(w.K, lo + J)
        chunk = [ds.grads[m].cpu().numpy() if wts[m] != 0 else None for m in range(lo, hi)]
        clock(oracle.accumulate_dense, run, chunk, wts[lo:hi])
        del chunk
    g_bar = clock(oracle.finalize_dense, run, w.K)
    del run
    hp = dict(lr=w.lr, eps=w.eps, beta1=w.beta1, beta2=w.beta2)
    if w.optimizer == "adagrad":
        clock(oracle.adagrad, pre["param"], pre["dslots"][0], g_bar, hp["lr"], hp["eps"])
    else:
        clock(oracle.adam, pre["param"], pre["dslots"][0], pre["dslots"][1], g_bar, hp["lr"], hp["beta1"],
              hp["beta2"], hp["eps"], w.adam_t)
    rows = ds.rows.cpu().numpy()
    sp = clock(oracle.aggregate_sparse, ds.ids_host, rows, ds.offsets_host, wts, tok, STEP, w.iota)
    del rows
    assert np.array_equal(sp["unique_ids"], pre["uq"])
    act = sp["active_count"] > 0
    if w.optimizer == "adagrad":
        clock(oracle.adagrad, pre["E"][act], pre["S"][0][act], sp["agg"][act], hp["lr"], hp["eps"])
    else:
        clock(oracle.adam, pre["E"][act], pre["S"][0][act], pre["S"][1][act], sp["agg"][act], hp["lr"],
              hp["beta1"], hp["beta2"], hp["eps"], w.adam_t)
    total_s = time.perf_counter() - t0
    return dict(value=1.0 / clock.wall, unit="global batches/s", cores=1, kind="oracle",
                sample=f"{w.name} in full: K={w.K} contributions of B={w.B} samples x L={w.L} IDs (N={w.N}), "
                       f"P={w.P} dense params; dense gradients handed over {J} contributions at a time and "
                       f"folded by the oracle's early weighted sum; oracle time {clock.wall:.1f} s (copies to "
                       f"the host, not timed, {total_s - clock.wall:.1f} s)",
                seconds_measured=clock.wall, cpu_seconds=clock.cpu, U=int(sp["num_unique"]),
                U_act=int(act.sum()), **host_cpu())


# The paper's own figures, placed beside the result as context and not as a
# target: whole training jobs on a cluster of Tesla V100S GPUs and Skylake CPUs
# shared with other jobs (Sec. 4.1); global QPS from Table 2, AUC and local
# QPS of the private task from Table 3.  The paper times no parameter-server
# step of its own, so none of these is comparable with a step time.
PAPER_CONTEXT = {
    "hardware": "training cluster of Tesla V100S GPUs and Skylake CPUs, shared with other jobs (Sec. 4.1)",
    "global_qps_samples_per_s": {
        "criteo_deepfm": {"gba": 3240e3, "sync": 1436e3, "async": 3253e3},
        "alimama_dien": {"gba": 399e3, "sync": 182e3, "async": 403e3},
        "private_youtubednn": {"gba": 87e3, "sync": 43e3, "async": 90e3},
    },
    "private_task_auc": {"sync": 0.7864, "gba": [0.7864, 0.7866, 0.7865]},
    "source": "Table 2 (global QPS), Table 3 (AUC of the private task at three local batch sizes)",
    "comparable": False,
}


def main():
    args = parse()
    if args.step_only:
        args.early_sum, args.hash_storage, args.graph = "", False, False
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library runs one PS shard per GPU and has no multi-GPU "
              "path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2205_11048_amd as gba
    from paper_2205_11048_amd import step as gba_step_mod
    from synth import device as sdev

    torch.cuda.set_device(0)
    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    head = run_workload(args.workload, args, torch, gba_step_mod, sdev, gba)
    others = [run_workload(n, args, torch, gba_step_mod, sdev, gba) for n in args.also.split(",") if n and n != args.workload]
    from synth.configs import BY_NAME
    w = BY_NAME[args.workload]
    out = {
        "metric": "global batches/sec and embedding-grad rows/sec; achieved HBM GB/s vs peak",
        "value": head["global_batches_per_s"],
        "unit": "global batches/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (f64 accumulation)",
        "data": "synthetic (seeded; Zipf IDs, counter-based gradients; no dataset)",
        "config": {"workload": f"{args.workload}: K={w.K} contributions, local batch {w.B}, "
                               f"{w.L} IDs/sample Zipf s={w.zipf_s} over {w.R}x{w.D} fp32 table, "
                               f"{w.P} dense params, {w.optimizer}, decay={args.decay}",
                   "global_batch": w.K * w.B, "K": w.K, "N": w.N, "R": w.R, "D": w.D, "P": w.P,
                   "parallelism": "one PS shard on one GPU"},
        "embedding_grad_rows_per_s": head["embedding_grad_rows_per_s"],
        "step_alg_gbs": head["step_alg_gbs"],
        "step_frac_of_hbm_peak": head["step_frac_of_hbm_peak"],
        "breakdown_ms": head["breakdown_ms"],
        "realised": {k: head[k] for k in ("K_eff", "N", "N_act", "U", "U_act", "step_alg_bytes")},
        "roofline": head["roofline"],
        "ceilings": head.get("ceilings"),
        "early_weighted_sum": head["early_sum"],
        "pull": head.get("pull"),
        "hash_storage": head.get("hash_storage"),
        "graph": head.get("graph"),
        "other_workloads": others,
        "paper_context": PAPER_CONTEXT,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = head.get("cpu_baseline") or cpu_baseline(args.workload, max(1, args.cpu_sample))
    print(json.dumps(out))


if __name__ == "__main__":
    main()
