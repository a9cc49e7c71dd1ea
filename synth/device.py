"""Seeded synthetic inputs made directly in GPU memory (libgba_synth.so).

The device generator computes the same counter-based values as
``synth.counter``; the host can re-derive any element to check a sampled
output.  Embedding IDs are drawn on the host (``synth.workload``) and
uploaded.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np
import torch

from . import counter, workload
from .configs import STEP, Workload, seed_of

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgba_synth.so")
_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} missing: build with `python -m paper_2205_11048_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.synth_fill_f32.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32,
                                     ctypes.c_uint64, ctypes.c_int, ctypes.c_float, ctypes.c_void_p]
        L.synth_fill_f32.restype = ctypes.c_int
        L.synth_fill_tags.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32,
                                      ctypes.c_int64, ctypes.c_void_p]
        L.synth_fill_tags.restype = ctypes.c_int
        _LIB = L
    return _LIB


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def fill(t: torch.Tensor, seed: int, stream: int, kind: int, scale: float = 0.0, start: int = 0):
    assert t.dtype == torch.float32 and t.is_cuda and t.is_contiguous()
    rc = lib().synth_fill_f32(ctypes.c_void_p(t.data_ptr()), t.numel(), seed & (2 ** 64 - 1), stream,
                              start, kind, float(scale), _stream())
    if rc != 0:
        raise RuntimeError(f"synth_fill_f32 failed ({rc})")
    return t


def fill_tags(t: torch.Tensor, seed: int, step: int = STEP):
    assert t.dtype == torch.int32 and t.is_cuda and t.is_contiguous()
    rc = lib().synth_fill_tags(ctypes.c_void_p(t.data_ptr()), t.numel(), seed & (2 ** 64 - 1),
                               counter.STREAM_TAGS, step, _stream())
    if rc != 0:
        raise RuntimeError(f"synth_fill_tags failed ({rc})")
    return t


@dataclass
class DeviceStep:
    """Every input of one step, resident in GPU memory."""
    w: Workload
    seed: int
    step: int
    tokens_host: np.ndarray
    offsets_host: np.ndarray
    ids_host: np.ndarray
    tokens: torch.Tensor
    offsets: torch.Tensor
    ids: torch.Tensor
    rows: torch.Tensor
    grads: list
    param: torch.Tensor
    dense_slots: list
    table: torch.Tensor
    table_slots: list
    tags: torch.Tensor | None
    value_kind: int


def make_device_step(w: Workload, seed: int | None = None, step: int = STEP, device="cuda",
                     value_kind: int = counter.KIND_GRAD, with_tags: bool = False, ids=None,
                     staleness=None) -> DeviceStep:
    seed = seed_of(w.name) if seed is None else seed
    scale = float(counter.grad_scale(w.grad_sigma))
    s = workload.staleness_draws(w, seed) if staleness is None else np.asarray(staleness, np.int64)
    tokens_h = workload.tokens_from_staleness(s, step)
    off_h = workload.contrib_offsets(w)
    ids_h = workload.embedding_ids(w, seed) if ids is None else np.asarray(ids, np.int64)
    dev = torch.device(device)
    rows = fill(torch.empty((w.N, w.D), dtype=torch.float32, device=dev), seed, counter.STREAM_ROWS,
                value_kind, scale)
    grads = [fill(torch.empty(w.P, dtype=torch.float32, device=dev), seed,
                  counter.STREAM_DENSE_GRAD_BASE + m, value_kind, scale) for m in range(w.K)]
    param = fill(torch.empty(w.P, dtype=torch.float32, device=dev), seed, counter.STREAM_DENSE_PARAM,
                 counter.KIND_PARAM)
    table = fill(torch.empty((w.R, w.D), dtype=torch.float32, device=dev), seed, counter.STREAM_TABLE,
                 counter.KIND_PARAM)
    dslots, tslots = [], []
    for ds, ts, kind in workload.state_kinds(w.optimizer):
        dslots.append(fill(torch.empty(w.P, dtype=torch.float32, device=dev), seed, ds, kind))
        tslots.append(fill(torch.empty((w.R, w.D), dtype=torch.float32, device=dev), seed, ts, kind))
    tags = fill_tags(torch.empty(w.R, dtype=torch.int32, device=dev), seed, step) if with_tags else None
    return DeviceStep(w, seed, step, tokens_h, off_h, ids_h,
                      torch.from_numpy(tokens_h).to(dev), torch.from_numpy(off_h).to(dev),
                      torch.from_numpy(ids_h).to(dev), rows, grads, param, dslots, table, tslots, tags,
                      value_kind)
