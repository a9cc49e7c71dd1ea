"""Python binding of libgba.so, the GBA push-step for MI355X (gfx950).

Each function has the name of the C entry point it calls (include/gba.h)
and does argument marshalling only: it reads sizes off torch tensors that
already live on the GPU, passes their device pointers and the current HIP
stream, and raises ``GBAError`` on a non-zero status.  Every step of the
computation runs in the library's HIP kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "GBAError", "lib", "gba_token_weights", "gba_aggregate_dense", "gba_aggregate_sparse",
    "gba_aggregate_sparse_workspace_size", "gba_apply_adagrad", "gba_apply_adam",
    "gba_aggregate_apply_dense_adagrad", "gba_aggregate_apply_dense_adam", "gba_accumulate_dense",
    "gba_finalize_dense", "gba_finalize_apply_dense_adagrad", "gba_finalize_apply_dense_adam",
    "gba_token_of_batch", "gba_pull_workspace_size", "gba_pull_rows", "gba_hash_clear",
    "gba_hash_workspace_size", "gba_hash_find_or_insert", "gba_hash_rehash", "EMPTY_ID", "DERR_TABLE_FULL",
    "gba_sort_ids_workspace_size", "gba_sort_ids", "SORT_AUTO", "SORT_PLAIN", "SORT_HOT",
    "gba_aggregate_sparse_plan_workspace_size", "gba_aggregate_sparse_plan", "gba_aggregate_sparse_noalloc",
    "NOALLOC_SCRATCH_BYTES", "ERR_SCRATCH_LIMIT", "gba_ceiling_read", "gba_ceiling_copy",
    "gba_ceiling_gather_rows", "gba_ceiling_sink_words",
    "pointer_table", "DECAY_TOKEN", "DECAY_ID_TAG", "NORM_PER_ID_COUNT", "NORM_BY_K",
    "DERR_ID_RANGE", "DERR_FUTURE_TOKEN", "DERR_OFFSETS", "DERR_ROW_RANGE", "MAX_K", "MAX_D",
    "LIB_PATH",
]

# GBA_LIBRARY may name another build of the library (for example one made for
# a different launch configuration); by default the in-tree build is used.
LIB_PATH = os.environ.get("GBA_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                         "libgba.so")

DECAY_TOKEN, DECAY_ID_TAG = 0, 1
NORM_PER_ID_COUNT, NORM_BY_K = 0, 1
DERR_ID_RANGE, DERR_FUTURE_TOKEN, DERR_OFFSETS, DERR_ROW_RANGE, DERR_TABLE_FULL = 1, 2, 4, 8, 16
EMPTY_ID = -1
SORT_AUTO, SORT_PLAIN, SORT_HOT = -1, 0, 1
MAX_K, MAX_D = 4096, 256
NOALLOC_SCRATCH_BYTES = 64 << 20     # GBA_NOALLOC_SCRATCH_BYTES
ERR_SCRATCH_LIMIT = 6

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_F64 = ctypes.c_double

_SIGNATURES = {
    "gba_status_string": ([_I32], ctypes.c_char_p),
    "gba_token_weights": ([_P, _I32, _I64, _I64, _P, _P, _P, _P, _P], _I32),
    "gba_aggregate_dense": ([_P, _P, _I32, _I64, _P, _P], _I32),
    "gba_aggregate_sparse_workspace_size": ([_I64, _I32, _I32, _I64, ctypes.POINTER(ctypes.c_size_t)], _I32),
    "gba_aggregate_sparse": ([_P, _P, _P, _I32, _I64, _I32, _I64, _P, _P, _I64, _I64, _P, _I32, _I32,
                              _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P, _P], _I32),
    "gba_aggregate_sparse_plan_workspace_size": ([_I64, _I32, _I32, _I64, _I32, ctypes.POINTER(ctypes.c_size_t)],
                                                 _I32),
    "gba_aggregate_sparse_plan": ([_P, _P, _P, _I32, _I64, _I32, _I64, _P, _P, _I64, _I64, _P, _I32, _I32,
                                   _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _I32, _P, _P], _I32),
    "gba_ceiling_read": ([_P, _I64, _P, _I32, _P], _I32),
    "gba_ceiling_copy": ([_P, _P, _I64, _I32, _P], _I32),
    "gba_ceiling_gather_rows": ([_P, _I64, _I32, _P, _I64, _P, _I32, _P], _I32),
    "gba_ceiling_sink_words": ([_I32], _I64),
    "gba_aggregate_sparse_noalloc": ([_P, _P, _P, _I32, _I64, _I32, _I64, _P, _P, _I64, _I64, _P, _I32, _I32,
                                      _P, _P, _P, _P, _P, _P, _P, _P], _I32),
    "gba_aggregate_apply_dense_adagrad": ([_P, _P, _I32, _I64, _P, _P, _P, _F64, _F64, _P], _I32),
    "gba_aggregate_apply_dense_adam": ([_P, _P, _I32, _I64, _P, _P, _P, _P, _F64, _F64, _F64, _F64, _I64, _P],
                                       _I32),
    "gba_accumulate_dense": ([_P, _P, _I32, _I64, _P, _P], _I32),
    "gba_aggregate_dense_launches": ([_I64, _I32, _I32, ctypes.POINTER(_I64)], _I32),
    "gba_aggregate_apply_sparse_workspace_size": ([_I64, _I32, _I32, _I64, _I32, ctypes.POINTER(ctypes.c_size_t)],
                                                  _I32),
    "gba_aggregate_apply_sparse_adagrad": ([_P, _P, _P, _I32, _I64, _I32, _I64, _P, _P, _I64, _I64, _P, _I32, _I32,
                                            _P, _P, _P, _P, _P, _P, _P, _P, _F64, _F64, _P, ctypes.c_size_t, _P,
                                            _P], _I32),
    "gba_aggregate_apply_sparse_adam": ([_P, _P, _P, _I32, _I64, _I32, _I64, _P, _P, _I64, _I64, _P, _I32, _I32,
                                         _P, _P, _P, _P, _P, _P, _P, _P, _P, _F64, _F64, _F64, _F64, _I64, _P,
                                         ctypes.c_size_t, _P, _P], _I32),
    "gba_finalize_dense": ([_P, _I32, _I64, _P, _I32, _P], _I32),
    "gba_finalize_apply_dense_adagrad": ([_P, _I32, _I64, _P, _P, _P, _F64, _F64, _I32, _P], _I32),
    "gba_finalize_apply_dense_adam": ([_P, _I32, _I64, _P, _P, _P, _P, _F64, _F64, _F64, _F64, _I64, _I32, _P],
                                      _I32),
    "gba_token_of_batch": ([_I64, _I32], _I64),
    "gba_pull_workspace_size": ([_I64, _I64, ctypes.POINTER(ctypes.c_size_t)], _I32),
    "gba_pull_rows": ([_P, _I64, _I64, _P, _I32, _P, _P, _P, _P, _P, ctypes.c_size_t, _P, _P], _I32),
    "gba_sort_ids_workspace_size": ([_I64, _I64, _I32, ctypes.POINTER(ctypes.c_size_t)], _I32),
    "gba_sort_ids": ([_P, _I64, _I64, _I32, _P, _P, _P, ctypes.c_size_t, _P, _P], _I32),
    "gba_hash_clear": ([_P, _P, _I64, _P], _I32),
    "gba_hash_workspace_size": ([_I64, ctypes.POINTER(ctypes.c_size_t)], _I32),
    "gba_hash_find_or_insert": ([_P, _P, _I64, _P, _I64, _P, _P, _I64, _P, _P, _P, ctypes.c_size_t, _P, _P], _I32),
    "gba_hash_rehash": ([_P, _P, _I64, _P, _P, _I64, _P, _P], _I32),
    "gba_apply_adagrad": ([_P, _P, _P, _P, _P, _P, _I64, _I32, _I64, _F64, _F64, _P, _P], _I32),
    "gba_apply_adam": ([_P, _P, _P, _P, _P, _P, _P, _I64, _I32, _I64, _F64, _F64, _F64, _F64, _I64,
                        _P, _P], _I32),
}

_LIB = None


class GBAError(RuntimeError):
    pass


def lib() -> ctypes.CDLL:
    """Load libgba.so (built in-tree by ``python -m paper_2205_11048_amd.build``)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise GBAError(f"{LIB_PATH} is missing: build it with `python -m paper_2205_11048_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _LIB = L
    return _LIB


def _check(status: int):
    if status != 0:
        raise GBAError(f"status {status}: {lib().gba_status_string(status).decode()}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _need(t, dtype, name, numel=None):
    if t is None:
        return
    if not t.is_cuda or t.dtype != dtype or not t.is_contiguous():
        raise GBAError(f"{name}: expected a contiguous {dtype} tensor on the GPU")
    if numel is not None and t.numel() < numel:
        raise GBAError(f"{name}: expected at least {numel} elements, got {t.numel()}")


def pointer_table(tensors, device=None) -> torch.Tensor:
    """Device int64 array of the tensors' device pointers (the `grads` argument)."""
    for i, t in enumerate(tensors):
        _need(t, torch.float32, f"grads[{i}]")
    device = device or tensors[0].device
    return torch.tensor([t.data_ptr() for t in tensors], dtype=torch.int64, device=device)


def gba_token_weights(tokens, step, iota, w, staleness=None, num_excluded=None, err=None, stream=None):
    K = tokens.numel()
    _need(tokens, torch.int64, "tokens")
    _need(w, torch.float32, "w", K)
    _need(staleness, torch.int64, "staleness", K)
    _need(num_excluded, torch.int32, "num_excluded", 1)
    _need(err, torch.int32, "err", 1)
    _check(lib().gba_token_weights(_ptr(tokens), K, int(step), int(iota), _ptr(w), _ptr(staleness),
                                   _ptr(num_excluded), _ptr(err), _stream(stream)))


def gba_aggregate_dense(grads, w, P, out, stream=None):
    """``grads``: device int64 tensor of K gradient pointers (see pointer_table)."""
    K = grads.numel()
    _need(grads, torch.int64, "grads")
    _need(w, torch.float32, "w", K)
    _need(out, torch.float32, "out", P)
    _check(lib().gba_aggregate_dense(_ptr(grads), _ptr(w), K, int(P), _ptr(out), _stream(stream)))


DENSE_SUM, DENSE_ADAGRAD, DENSE_ADAM, DENSE_ACCUMULATE = 0, 1, 2, 3


def gba_aggregate_dense_launches(P, K, opt=DENSE_SUM):
    """Kernel launches one dense call makes on the current device (host query)."""
    n = _I64(0)
    _check(lib().gba_aggregate_dense_launches(int(P), int(K), int(opt), ctypes.byref(n)))
    return int(n.value)


def _dense_common(grads, w, P, out, **state):
    K = grads.numel()
    _need(grads, torch.int64, "grads")
    _need(w, torch.float32, "w", K)
    _need(out, torch.float32, "out", P)
    for name, x in state.items():
        if x is None:
            raise GBAError(f"{name} is required")
        _need(x, torch.float32, name, P)
    return K


def gba_aggregate_apply_dense_adagrad(grads, w, P, param, accum, lr, eps, out=None, stream=None):
    """gba_aggregate_dense + dense Adagrad in one pass; ``out`` (the sum) may be None."""
    K = _dense_common(grads, w, P, out, param=param, accum=accum)
    _check(lib().gba_aggregate_apply_dense_adagrad(_ptr(grads), _ptr(w), K, int(P), _ptr(out), _ptr(param),
                                                   _ptr(accum), float(lr), float(eps), _stream(stream)))


def gba_aggregate_apply_dense_adam(grads, w, P, param, m, v, lr, beta1, beta2, eps, t, out=None, stream=None):
    """gba_aggregate_dense + dense Adam in one pass; ``out`` (the sum) may be None."""
    K = _dense_common(grads, w, P, out, param=param, m=m, v=v)
    _check(lib().gba_aggregate_apply_dense_adam(_ptr(grads), _ptr(w), K, int(P), _ptr(out), _ptr(param), _ptr(m),
                                                _ptr(v), float(lr), float(beta1), float(beta2), float(eps), int(t),
                                                _stream(stream)))


def gba_accumulate_dense(grads, w, P, run, stream=None):
    """Early weighted sum: run += sum_j w_j g_j in float64, in order.
    ``grads``: device int64 tensor of J gradient pointers; ``run``: float64 [P]."""
    J = grads.numel()
    _need(grads, torch.int64, "grads")
    _need(w, torch.float32, "w", J)
    _need(run, torch.float64, "run", P)
    _check(lib().gba_accumulate_dense(_ptr(grads), _ptr(w), J, int(P), _ptr(run), _stream(stream)))


def gba_finalize_dense(run, K, P, out, reset=True, stream=None):
    _need(run, torch.float64, "run", P)
    _need(out, torch.float32, "out", P)
    _check(lib().gba_finalize_dense(_ptr(run), int(K), int(P), _ptr(out), int(bool(reset)), _stream(stream)))


def gba_finalize_apply_dense_adagrad(run, K, P, param, accum, lr, eps, out=None, reset=True, stream=None):
    _need(run, torch.float64, "run", P)
    _need(out, torch.float32, "out", P)
    for name, x in (("param", param), ("accum", accum)):
        _need(x, torch.float32, name, P)
    _check(lib().gba_finalize_apply_dense_adagrad(_ptr(run), int(K), int(P), _ptr(out), _ptr(param), _ptr(accum),
                                                  float(lr), float(eps), int(bool(reset)), _stream(stream)))


def gba_finalize_apply_dense_adam(run, K, P, param, m, v, lr, beta1, beta2, eps, t, out=None, reset=True,
                                  stream=None):
    _need(run, torch.float64, "run", P)
    _need(out, torch.float32, "out", P)
    for name, x in (("param", param), ("m", m), ("v", v)):
        _need(x, torch.float32, name, P)
    _check(lib().gba_finalize_apply_dense_adam(_ptr(run), int(K), int(P), _ptr(out), _ptr(param), _ptr(m), _ptr(v),
                                               float(lr), float(beta1), float(beta2), float(eps), int(t),
                                               int(bool(reset)), _stream(stream)))


def gba_token_of_batch(i, M) -> int:
    """Token of the i-th batch handed out: floor(i / M), each value M times."""
    return int(lib().gba_token_of_batch(int(i), int(M)))


def gba_pull_workspace_size(n, R) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gba_pull_workspace_size(int(n), int(R), ctypes.byref(b)))
    return int(b.value)


def gba_pull_rows(ids, table, unique_ids, inverse, rows, num_unique, workspace, err=None, stream=None):
    """Rows of a worker's request, once per distinct ID: table[unique_ids] and
    the inverse map (ids == unique_ids[inverse])."""
    n = ids.numel()
    R, D = table.shape
    _need(ids, torch.int64, "ids")
    _need(table, torch.float32, "table")
    _need(unique_ids, torch.int64, "unique_ids", n)
    _need(inverse, torch.int32, "inverse", n)
    _need(rows, torch.float32, "rows", n * D)
    _need(num_unique, torch.int64, "num_unique", 1)
    _need(workspace, torch.uint8, "workspace")
    _need(err, torch.int32, "err", 1)
    _check(lib().gba_pull_rows(_ptr(ids), n, int(R), _ptr(table), int(D), _ptr(unique_ids), _ptr(inverse), _ptr(rows),
                               _ptr(num_unique), _ptr(workspace), workspace.numel(), _ptr(err), _stream(stream)))


def gba_sort_ids_workspace_size(n, R, plan=SORT_AUTO) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gba_sort_ids_workspace_size(int(n), int(R), int(plan), ctypes.byref(b)))
    return int(b.value)


def gba_sort_ids(ids, R, keys_out, index_out, workspace, plan=SORT_AUTO, err=None, stream=None):
    """Stable sort of the IDs: keys_out = the IDs ascending (uint32 stored in
    int32), index_out = each sorted entry's occurrence index."""
    n = ids.numel()
    _need(ids, torch.int64, "ids")
    _need(keys_out, torch.int32, "keys_out", n)
    _need(index_out, torch.int32, "index_out", n)
    _need(workspace, torch.uint8, "workspace")
    _need(err, torch.int32, "err", 1)
    _check(lib().gba_sort_ids(_ptr(ids), n, int(R), int(plan), _ptr(keys_out), _ptr(index_out), _ptr(workspace),
                              workspace.numel(), _ptr(err), _stream(stream)))


def gba_hash_clear(slot_ids, slot_rows, stream=None):
    _need(slot_ids, torch.int64, "slot_ids")
    _need(slot_rows, torch.int32, "slot_rows", slot_ids.numel())
    _check(lib().gba_hash_clear(_ptr(slot_ids), _ptr(slot_rows), slot_ids.numel(), _stream(stream)))


def gba_hash_workspace_size(n) -> int:
    b = ctypes.c_size_t(0)
    _check(lib().gba_hash_workspace_size(int(n), ctypes.byref(b)))
    return int(b.value)


def gba_hash_find_or_insert(slot_ids, slot_rows, ids, rows_out, num_rows, max_rows, workspace, row_ids=None,
                            num_new=None, err=None, stream=None):
    """rows_out[i] = row of ids[i] in the pool; new IDs get the next rows."""
    n = ids.numel()
    _need(slot_ids, torch.int64, "slot_ids")
    _need(slot_rows, torch.int32, "slot_rows", slot_ids.numel())
    _need(ids, torch.int64, "ids")
    _need(rows_out, torch.int64, "rows_out", n)
    _need(num_rows, torch.int64, "num_rows", 1)
    _need(row_ids, torch.int64, "row_ids", max_rows if row_ids is not None else None)
    _need(num_new, torch.int64, "num_new", 1)
    _need(workspace, torch.uint8, "workspace")
    _need(err, torch.int32, "err", 1)
    _check(lib().gba_hash_find_or_insert(_ptr(slot_ids), _ptr(slot_rows), slot_ids.numel(), _ptr(ids), n,
                                         _ptr(rows_out), _ptr(num_rows), int(max_rows), _ptr(row_ids), _ptr(num_new),
                                         _ptr(workspace), workspace.numel(), _ptr(err), _stream(stream)))


def gba_hash_rehash(old_ids, old_rows, new_ids, new_rows, err=None, stream=None):
    for name, x, dt in (("old_ids", old_ids, torch.int64), ("old_rows", old_rows, torch.int32),
                        ("new_ids", new_ids, torch.int64), ("new_rows", new_rows, torch.int32)):
        _need(x, dt, name)
    _need(err, torch.int32, "err", 1)
    _check(lib().gba_hash_rehash(_ptr(old_ids), _ptr(old_rows), old_ids.numel(), _ptr(new_ids), _ptr(new_rows),
                                 new_ids.numel(), _ptr(err), _stream(stream)))


def gba_aggregate_sparse_workspace_size(N, K, D, R) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().gba_aggregate_sparse_workspace_size(int(N), int(K), int(D), int(R), ctypes.byref(n)))
    return int(n.value)


def gba_aggregate_sparse_plan_workspace_size(N, K, D, R, plan) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().gba_aggregate_sparse_plan_workspace_size(int(N), int(K), int(D), int(R), int(plan),
                                                          ctypes.byref(n)))
    return int(n.value)


def _sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets, contrib_count,
                 active_count, agg, num_unique, workspace, err):
    N = ids.numel()
    K = contrib_offsets.numel() - 1
    D = rows.shape[-1]
    _need(ids, torch.int64, "ids")
    _need(rows, torch.float32, "rows", N * D)
    _need(contrib_offsets, torch.int64, "contrib_offsets")
    _need(w, torch.float32, "w", K)
    _need(tokens, torch.int64, "tokens", K)
    _need(tag, torch.int32, "tag", R if tag is not None else None)
    _need(unique_ids, torch.int64, "unique_ids", N)
    _need(seg_offsets, torch.int64, "seg_offsets", N + 1)
    _need(contrib_count, torch.int32, "contrib_count", N)
    _need(active_count, torch.int32, "active_count", N)
    _need(agg, torch.float32, "agg", N * D)
    _need(num_unique, torch.int64, "num_unique", 1)
    _need(workspace, torch.uint8, "workspace")
    _need(err, torch.int32, "err", 1)
    return N, K, D


def gba_aggregate_sparse(ids, rows, contrib_offsets, R, w, tokens, step, iota, tag, decay, norm,
                         unique_ids, seg_offsets, contrib_count, active_count, agg, num_unique,
                         workspace, err=None, stream=None):
    N, K, D = _sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets, contrib_count,
                           active_count, agg, num_unique, workspace, err)
    _check(lib().gba_aggregate_sparse(
        _ptr(ids), _ptr(rows), _ptr(contrib_offsets), K, N, D, int(R), _ptr(w), _ptr(tokens), int(step),
        int(iota), _ptr(tag), int(decay), int(norm), _ptr(unique_ids), _ptr(seg_offsets),
        _ptr(contrib_count), _ptr(active_count), _ptr(agg), _ptr(num_unique), _ptr(workspace),
        workspace.numel(), _ptr(err), _stream(stream)))


def gba_aggregate_sparse_plan(ids, rows, contrib_offsets, R, w, tokens, step, iota, tag, decay, norm,
                              unique_ids, seg_offsets, contrib_count, active_count, agg, num_unique,
                              workspace, plan, err=None, stream=None):
    """gba_aggregate_sparse with the sort plan chosen by the caller (SORT_AUTO, SORT_PLAIN, SORT_HOT)."""
    N, K, D = _sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets, contrib_count,
                           active_count, agg, num_unique, workspace, err)
    _check(lib().gba_aggregate_sparse_plan(
        _ptr(ids), _ptr(rows), _ptr(contrib_offsets), K, N, D, int(R), _ptr(w), _ptr(tokens), int(step),
        int(iota), _ptr(tag), int(decay), int(norm), _ptr(unique_ids), _ptr(seg_offsets),
        _ptr(contrib_count), _ptr(active_count), _ptr(agg), _ptr(num_unique), _ptr(workspace),
        workspace.numel(), int(plan), _ptr(err), _stream(stream)))


def gba_aggregate_sparse_noalloc(ids, rows, contrib_offsets, R, w, tokens, step, iota, tag, decay, norm,
                                 unique_ids, seg_offsets, contrib_count, active_count, agg, num_unique,
                                 err=None, stream=None):
    """gba_aggregate_sparse with the library's fixed device scratch array
    instead of a workspace (the call allocates nothing); sizes whose workspace
    would exceed NOALLOC_SCRATCH_BYTES raise GBAError (status ERR_SCRATCH_LIMIT)."""
    N = ids.numel()
    K = contrib_offsets.numel() - 1
    D = rows.shape[-1]
    _need(ids, torch.int64, "ids")
    _need(rows, torch.float32, "rows", N * D)
    _need(contrib_offsets, torch.int64, "contrib_offsets")
    _need(w, torch.float32, "w", K)
    _need(tokens, torch.int64, "tokens", K)
    _need(tag, torch.int32, "tag", R if tag is not None else None)
    _need(unique_ids, torch.int64, "unique_ids", N)
    _need(seg_offsets, torch.int64, "seg_offsets", N + 1)
    _need(contrib_count, torch.int32, "contrib_count", N)
    _need(active_count, torch.int32, "active_count", N)
    _need(agg, torch.float32, "agg", N * D)
    _need(num_unique, torch.int64, "num_unique", 1)
    _need(err, torch.int32, "err", 1)
    _check(lib().gba_aggregate_sparse_noalloc(
        _ptr(ids), _ptr(rows), _ptr(contrib_offsets), K, N, D, int(R), _ptr(w), _ptr(tokens), int(step),
        int(iota), _ptr(tag), int(decay), int(norm), _ptr(unique_ids), _ptr(seg_offsets),
        _ptr(contrib_count), _ptr(active_count), _ptr(agg), _ptr(num_unique), _ptr(err), _stream(stream)))


OPTIMIZER_ADAGRAD, OPTIMIZER_ADAM = 1, 2


def gba_aggregate_apply_sparse_workspace_size(N, K, D, R, optimizer) -> int:
    """``optimizer``: "adagrad", "adam" or OPTIMIZER_ADAGRAD / OPTIMIZER_ADAM."""
    opt = {"adagrad": OPTIMIZER_ADAGRAD, "adam": OPTIMIZER_ADAM}.get(optimizer, optimizer)
    n = ctypes.c_size_t(0)
    _check(lib().gba_aggregate_apply_sparse_workspace_size(int(N), int(K), int(D), int(R), int(opt),
                                                           ctypes.byref(n)))
    return int(n.value)


def _apply_sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets, contrib_count,
                       active_count, agg, num_unique, workspace, err, table, state):
    N, K, D = _sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets, contrib_count,
                           active_count, None, num_unique, workspace, err)
    _need(agg, torch.float32, "agg", N * D)
    for name, t in [("table", table)] + state:
        _need(t, torch.float32, name, int(R) * D)
    return N, K, D


def gba_aggregate_apply_sparse_adagrad(ids, rows, contrib_offsets, R, w, tokens, step, iota, tag, decay, norm,
                                       unique_ids, seg_offsets, contrib_count, active_count, agg, num_unique,
                                       table, accum, lr, eps, workspace, err=None, stream=None):
    """gba_aggregate_sparse + the row form of gba_apply_adagrad in one call; ``agg`` may be None."""
    N, K, D = _apply_sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets,
                                 contrib_count, active_count, agg, num_unique, workspace, err, table,
                                 [("accum", accum)])
    _check(lib().gba_aggregate_apply_sparse_adagrad(
        _ptr(ids), _ptr(rows), _ptr(contrib_offsets), K, N, D, int(R), _ptr(w), _ptr(tokens), int(step),
        int(iota), _ptr(tag), int(decay), int(norm), _ptr(unique_ids), _ptr(seg_offsets),
        _ptr(contrib_count), _ptr(active_count), _ptr(agg), _ptr(num_unique), _ptr(table), _ptr(accum),
        float(lr), float(eps), _ptr(workspace), workspace.numel(), _ptr(err), _stream(stream)))


def gba_aggregate_apply_sparse_adam(ids, rows, contrib_offsets, R, w, tokens, step, iota, tag, decay, norm,
                                    unique_ids, seg_offsets, contrib_count, active_count, agg, num_unique,
                                    table, m, v, lr, beta1, beta2, eps, t, workspace, err=None, stream=None):
    """gba_aggregate_sparse + the row form of gba_apply_adam in one call; ``agg`` may be None."""
    N, K, D = _apply_sparse_args(ids, rows, contrib_offsets, R, w, tokens, tag, unique_ids, seg_offsets,
                                 contrib_count, active_count, agg, num_unique, workspace, err, table,
                                 [("m", m), ("v", v)])
    _check(lib().gba_aggregate_apply_sparse_adam(
        _ptr(ids), _ptr(rows), _ptr(contrib_offsets), K, N, D, int(R), _ptr(w), _ptr(tokens), int(step),
        int(iota), _ptr(tag), int(decay), int(norm), _ptr(unique_ids), _ptr(seg_offsets),
        _ptr(contrib_count), _ptr(active_count), _ptr(agg), _ptr(num_unique), _ptr(table), _ptr(m), _ptr(v),
        float(lr), float(beta1), float(beta2), float(eps), int(t), _ptr(workspace), workspace.numel(), _ptr(err),
        _stream(stream)))


def gba_apply_adagrad(param, accum, grad, lr, eps, rows=None, active=None, num_rows=None, R=0,
                      err=None, stream=None):
    """Dense form when ``rows`` is None, else the row form over [R, D] tables."""
    _need(param, torch.float32, "param")
    _need(accum, torch.float32, "accum")
    _need(grad, torch.float32, "grad")
    _need(rows, torch.int64, "rows")
    _need(active, torch.int32, "active")
    _need(num_rows, torch.int64, "num_rows", 1 if rows is not None else None)
    _need(err, torch.int32, "err", 1)
    if rows is None:
        n, D = grad.numel(), 0
        if param.numel() < n or accum.numel() < n:
            raise GBAError("param/accum shorter than grad")
    else:
        n, D = rows.numel(), param.shape[-1]
        if grad.numel() < n * D or param.numel() < R * D or accum.numel() < R * D:
            raise GBAError("row-form sizes do not match")
    _check(lib().gba_apply_adagrad(_ptr(param), _ptr(accum), _ptr(grad), _ptr(rows), _ptr(active),
                                   _ptr(num_rows), n, D, int(R), float(lr), float(eps), _ptr(err),
                                   _stream(stream)))


def gba_apply_adam(param, m, v, grad, lr, beta1, beta2, eps, t, rows=None, active=None, num_rows=None,
                   R=0, err=None, stream=None):
    for name, x in (("param", param), ("m", m), ("v", v), ("grad", grad)):
        _need(x, torch.float32, name)
    _need(rows, torch.int64, "rows")
    _need(active, torch.int32, "active")
    _need(num_rows, torch.int64, "num_rows", 1 if rows is not None else None)
    _need(err, torch.int32, "err", 1)
    if rows is None:
        n, D = grad.numel(), 0
        if min(param.numel(), m.numel(), v.numel()) < n:
            raise GBAError("param/m/v shorter than grad")
    else:
        n, D = rows.numel(), param.shape[-1]
        if grad.numel() < n * D or min(param.numel(), m.numel(), v.numel()) < R * D:
            raise GBAError("row-form sizes do not match")
    _check(lib().gba_apply_adam(_ptr(param), _ptr(m), _ptr(v), _ptr(grad), _ptr(rows), _ptr(active),
                                _ptr(num_rows), n, D, int(R), float(lr), float(beta1), float(beta2),
                                float(eps), int(t), _ptr(err), _stream(stream)))


# ------------------------------------------------- measurement kernels
# (include/gba_ceilings.h: the bandwidth of the step's access patterns)
def gba_ceiling_sink_words(blocks) -> int:
    return int(lib().gba_ceiling_sink_words(int(blocks)))


def _bytes16(t, name):
    if not t.is_cuda or not t.is_contiguous():
        raise GBAError(f"{name}: expected a contiguous tensor on the GPU")
    return t.numel() * t.element_size() // 16


def gba_ceiling_read(src, sink, blocks, stream=None):
    """Reads every whole 16-byte vector of ``src`` once (non-temporal loads)."""
    _need(sink, torch.int32, "sink", gba_ceiling_sink_words(blocks))
    _check(lib().gba_ceiling_read(_ptr(src), _bytes16(src, "src"), _ptr(sink), int(blocks), _stream(stream)))


def gba_ceiling_copy(src, dst, blocks, stream=None):
    """Copies the whole 16-byte vectors of ``src`` to ``dst``."""
    n16 = _bytes16(src, "src")
    if _bytes16(dst, "dst") < n16:
        raise GBAError("dst: smaller than src")
    _check(lib().gba_ceiling_copy(_ptr(src), _ptr(dst), n16, int(blocks), _stream(stream)))


def gba_ceiling_gather_rows(table, rows, sink, blocks, stream=None):
    """Gathers table[rows[i]] for every i (rows: int64 on the GPU)."""
    _need(table, torch.float32, "table")
    _need(rows, torch.int64, "rows")
    _need(sink, torch.int32, "sink", gba_ceiling_sink_words(blocks))
    R, D = table.shape
    _check(lib().gba_ceiling_gather_rows(_ptr(table), int(R), int(D), _ptr(rows), rows.numel(), _ptr(sink),
                                         int(blocks), _stream(stream)))
