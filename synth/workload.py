"""Seeded synthetic inputs of one PS step (host side).

A step's inputs are: the K contributions of one global batch in buffer
(arrival) order, each with its token, its dense gradient (P floats) and its
sparse part (n_m embedding IDs with one gradient row of D floats each, in
contribution-major order); and the PS state (dense parameters and optimiser
slots, the embedding table and its slots, the per-ID step tags).

Nothing here is a step of the aggregation itself.  The same functions feed the
oracle and, through ``synth/gen.hip`` for arrays too large for the host, the
device path.  Every value is a function of (seed, stream, index), so any
element can be regenerated on its own to check a sampled output.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import counter
from .configs import STEP, Workload, seed_of
from .zipf import ZipfRejectionInversion, rank_to_row


def staleness_draws(w: Workload, seed: int) -> np.ndarray:
    """Per-contribution staleness s_m >= 0 (int64), from the workload's law."""
    u = counter.uniform01(seed, counter.STREAM_STALENESS, np.arange(w.K, dtype=np.uint64))
    law, par = w.staleness
    if law == "uniform":
        return np.floor(u * (int(par) + 1)).astype(np.int64)
    if law == "geometric":
        # P(s) = p (1 - p)^s for s >= 0, by inversion of the survival function
        return np.floor(np.log1p(-u) / np.log1p(-float(par))).astype(np.int64)
    if law == "zero":
        return np.zeros(w.K, dtype=np.int64)
    raise ValueError(law)


def tokens_from_staleness(s: np.ndarray, step: int = STEP) -> np.ndarray:
    return (np.int64(step) - np.asarray(s, dtype=np.int64)).astype(np.int64)


def contrib_offsets(w: Workload, sizes=None) -> np.ndarray:
    n = np.full(w.K, w.n_per_contribution, dtype=np.int64) if sizes is None else np.asarray(sizes, np.int64)
    return np.concatenate([[0], np.cumsum(n)]).astype(np.int64)


def embedding_ids(w: Workload, seed: int, start: int = 0, count: int | None = None) -> np.ndarray:
    """IDs of occurrences [start, start + count) in contribution-major order.

    Occurrence j belongs to sample j // L and slot j % L.  Multi-hot workloads
    draw every slot from one Zipf law over all R rows; one-hot workloads give
    slot f its own field of floor(R / L) rows.
    """
    if count is None:
        count = w.N - start
    chunk = 1 << 21
    if count > 2 * chunk:
        # independent chunks (every ID depends only on its index): run them on threads
        import os
        from concurrent.futures import ThreadPoolExecutor
        starts = list(range(start, start + count, chunk))
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            parts = list(ex.map(lambda s0: embedding_ids(w, seed, s0, min(chunk, start + count - s0)),
                                starts))
        return np.concatenate(parts)
    j = np.arange(start, start + count, dtype=np.int64)
    if w.one_hot_fields:
        field_rows = w.R // w.L
        z = ZipfRejectionInversion(field_rows, w.zipf_s)
        rank = z.ranks(seed, j)
        f = j % w.L
        return f * field_rows + rank_to_row(rank - 1, field_rows)
    z = ZipfRejectionInversion(w.R, w.zipf_s)
    return rank_to_row(z.ranks(seed, j) - 1, w.R)


def row_values(w: Workload, seed: int, j_start: int, j_count: int, kind=counter.KIND_GRAD,
               d_count: int | None = None) -> np.ndarray:
    """Embedding-gradient rows of occurrences [j_start, j_start + j_count) as [j_count, D]."""
    D = w.D
    flat = counter.values_range(seed, counter.STREAM_ROWS, j_start * D, j_count * D, kind,
                                counter.grad_scale(w.grad_sigma))
    return flat.reshape(j_count, D)


def dense_grad(w: Workload, seed: int, m: int, start: int = 0, count: int | None = None,
               kind=counter.KIND_GRAD) -> np.ndarray:
    if count is None:
        count = w.P - start
    return counter.values_range(seed, counter.STREAM_DENSE_GRAD_BASE + m, start, count, kind,
                                counter.grad_scale(w.grad_sigma))


def tag_values(seed: int, rows: np.ndarray, step: int = STEP) -> np.ndarray:
    """Step tag of each row: -1 (never updated) for half the rows, else
    step - 1 - G with G geometric(1/2), G = trailing zeros of the row's word."""
    wd = counter.words(seed, counter.STREAM_TAGS, np.asarray(rows, dtype=np.uint64))
    g = counter.ctz64(wd, cap=62)
    seen = (wd >> np.uint64(63)) == np.uint64(1)
    t = np.int64(step) - 1 - g
    return np.where(seen, np.maximum(t, -1), -1).astype(np.int32)


# Optimiser-state kinds of the dense vector and of the table, per slot.
def state_kinds(optimizer: str):
    if optimizer == "adagrad":
        return [(counter.STREAM_DENSE_SLOT1, counter.STREAM_TABLE_SLOT1, counter.KIND_ACCUM)]
    if optimizer == "adam":
        return [(counter.STREAM_DENSE_SLOT1, counter.STREAM_TABLE_SLOT1, counter.KIND_ADAM_M),
                (counter.STREAM_DENSE_SLOT2, counter.STREAM_TABLE_SLOT2, counter.KIND_ADAM_V)]
    raise ValueError(optimizer)


@dataclass
class HostStep:
    """All inputs of one step held on the host (small workloads only)."""
    w: Workload
    seed: int
    step: int
    tokens: np.ndarray          # int64 [K]
    staleness: np.ndarray       # int64 [K]
    offsets: np.ndarray         # int64 [K + 1]
    ids: np.ndarray             # int64 [N]
    rows: np.ndarray            # float32 [N, D]
    grads: np.ndarray           # float32 [K, P]
    param: np.ndarray           # float32 [P]
    dense_slots: list           # float32 [P] per slot
    table: np.ndarray           # float32 [R, D]
    table_slots: list           # float32 [R, D] per slot
    tags: np.ndarray            # int32 [R]


def host_step(w: Workload, seed: int | None = None, step: int = STEP,
              value_kind: int = counter.KIND_GRAD, staleness=None) -> HostStep:
    """Materialise every input of one step on the host (for R * D, K * P small)."""
    seed = seed_of(w.name) if seed is None else seed
    s = staleness_draws(w, seed) if staleness is None else np.asarray(staleness, np.int64)
    off = contrib_offsets(w)
    ids = embedding_ids(w, seed)
    rows = row_values(w, seed, 0, w.N, value_kind)
    grads = np.stack([dense_grad(w, seed, m, kind=value_kind) for m in range(w.K)]) if w.K else \
        np.zeros((0, w.P), np.float32)
    param = counter.values_range(seed, counter.STREAM_DENSE_PARAM, 0, w.P, counter.KIND_PARAM)
    table = counter.values_range(seed, counter.STREAM_TABLE, 0, w.R * w.D,
                                 counter.KIND_PARAM).reshape(w.R, w.D)
    dslots, tslots = [], []
    for ds, ts, kind in state_kinds(w.optimizer):
        dslots.append(counter.values_range(seed, ds, 0, w.P, kind))
        tslots.append(counter.values_range(seed, ts, 0, w.R * w.D, kind).reshape(w.R, w.D))
    tags = tag_values(seed, np.arange(w.R), step)
    return HostStep(w, seed, step, tokens_from_staleness(s, step), s, off, ids, rows, grads,
                    param, dslots, table, tslots, tags)
