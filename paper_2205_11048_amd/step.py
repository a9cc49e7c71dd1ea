"""One GBA push-step on one PS shard, through the C ABI.

Alg. 2 (push responder) of the paper, once N_a = K gradients are buffered:
token weights (Eq. 1) -> dense weighted sum / K -> embedding dedup, per-ID
decay and weighted sum / c_r -> optimiser apply on the dense vector and on
the touched rows.  This class owns only the output and scratch buffers of the
step (allocated once, reused every step); inputs and PS state are the
caller's tensors.  All calls are enqueued on one stream with no host
synchronisation in between.  The dense sum and the dense optimiser run as one
fused call by default (``fused_dense=False`` makes them two), and so do the
sparse aggregation and the row apply (``fused_sparse=False`` makes them two).
"""
from __future__ import annotations

import torch

from . import (DECAY_ID_TAG, DECAY_TOKEN, NORM_PER_ID_COUNT, gba_aggregate_apply_dense_adagrad,
               gba_aggregate_apply_dense_adam, gba_aggregate_apply_sparse_adagrad, gba_aggregate_apply_sparse_adam,
               gba_aggregate_apply_sparse_workspace_size, gba_aggregate_dense, gba_aggregate_sparse,
               gba_aggregate_sparse_workspace_size, gba_apply_adagrad, gba_apply_adam, gba_token_weights,
               pointer_table)


class GBAStep:
    def __init__(self, K: int, N: int, D: int, R: int, P: int, device="cuda"):
        self.K, self.N, self.D, self.R, self.P = K, N, D, R, P
        dev = torch.device(device)
        self.device = dev
        self.w = torch.empty(K, dtype=torch.float32, device=dev)
        self.staleness = torch.empty(K, dtype=torch.int64, device=dev)
        self.num_excluded = torch.zeros(1, dtype=torch.int32, device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.g_bar = torch.empty(P, dtype=torch.float32, device=dev)
        cap = max(N, 1)
        self.unique_ids = torch.empty(cap, dtype=torch.int64, device=dev)
        self.seg_offsets = torch.empty(cap + 1, dtype=torch.int64, device=dev)
        self.contrib_count = torch.empty(cap, dtype=torch.int32, device=dev)
        self.active_count = torch.empty(cap, dtype=torch.int32, device=dev)
        self.agg = torch.empty((cap, D), dtype=torch.float32, device=dev)
        self.num_unique = torch.zeros(1, dtype=torch.int64, device=dev)
        ws = gba_aggregate_sparse_workspace_size(N, K, D, R)
        # the fused sparse call needs no more workspace where it applies the
        # rows as it goes; otherwise the means go through agg (ours)
        self.fuses_rows = {opt: gba_aggregate_apply_sparse_workspace_size(N, K, D, R, opt) == ws
                           for opt in ("adagrad", "adam")}
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=dev)
        self._grad_table = None
        self._grad_table_key = None

    def grad_table(self, grads):
        key = tuple(g.data_ptr() for g in grads)
        if key != self._grad_table_key:
            self._grad_table = pointer_table(grads, self.device)
            self._grad_table_key = key
        return self._grad_table

    def run(self, *, tokens, step, iota, grads, ids, rows, offsets, param, dense_slots, table,
            table_slots, optimizer, lr, eps, beta1=0.9, beta2=0.999, t=1, tag=None,
            decay=DECAY_TOKEN, norm=NORM_PER_ID_COUNT, stream=None, fused_dense=True, keep_g_bar=True,
            fused_sparse=True, keep_agg=False):
        """One push-step.  On the fused dense path, ``keep_g_bar`` also stores
        the dense sum in ``self.g_bar`` (the separate path always does); on the
        fused sparse path, ``keep_agg`` stores the per-ID means in ``self.agg``
        (the separate path always does)."""
        if optimizer not in ("adagrad", "adam"):
            raise ValueError(optimizer)
        gba_token_weights(tokens, step, iota, self.w, self.staleness, self.num_excluded, self.err,
                          stream=stream)
        table_grads = self.grad_table(grads)
        g_out = self.g_bar if keep_g_bar else None
        if fused_dense and optimizer == "adagrad":
            gba_aggregate_apply_dense_adagrad(table_grads, self.w, self.P, param, dense_slots[0], lr, eps,
                                              out=g_out, stream=stream)
        elif fused_dense:
            gba_aggregate_apply_dense_adam(table_grads, self.w, self.P, param, dense_slots[0], dense_slots[1], lr,
                                           beta1, beta2, eps, t, out=g_out, stream=stream)
        else:
            gba_aggregate_dense(table_grads, self.w, self.P, self.g_bar, stream=stream)
            if optimizer == "adagrad":
                gba_apply_adagrad(param, dense_slots[0], self.g_bar, lr, eps, stream=stream)
            else:
                gba_apply_adam(param, dense_slots[0], dense_slots[1], self.g_bar, lr, beta1, beta2, eps, t,
                               stream=stream)
        sparse_tag = tag if decay == DECAY_ID_TAG else None
        if fused_sparse:
            agg = self.agg if (keep_agg or not self.fuses_rows[optimizer]) else None
            if optimizer == "adagrad":
                gba_aggregate_apply_sparse_adagrad(ids, rows, offsets, self.R, self.w, tokens, step, iota, sparse_tag,
                                                   decay, norm, self.unique_ids, self.seg_offsets, self.contrib_count,
                                                   self.active_count, agg, self.num_unique, table, table_slots[0],
                                                   lr, eps, self.workspace, self.err, stream=stream)
            else:
                gba_aggregate_apply_sparse_adam(ids, rows, offsets, self.R, self.w, tokens, step, iota, sparse_tag,
                                                decay, norm, self.unique_ids, self.seg_offsets, self.contrib_count,
                                                self.active_count, agg, self.num_unique, table, table_slots[0],
                                                table_slots[1], lr, beta1, beta2, eps, t, self.workspace, self.err,
                                                stream=stream)
            return
        gba_aggregate_sparse(ids, rows, offsets, self.R, self.w, tokens, step, iota, sparse_tag, decay, norm,
                             self.unique_ids, self.seg_offsets, self.contrib_count, self.active_count, self.agg,
                             self.num_unique, self.workspace, self.err, stream=stream)
        if optimizer == "adagrad":
            gba_apply_adagrad(table, table_slots[0], self.agg, lr, eps, rows=self.unique_ids,
                              active=self.active_count, num_rows=self.num_unique, R=self.R,
                              err=self.err, stream=stream)
        else:
            gba_apply_adam(table, table_slots[0], table_slots[1], self.agg, lr, beta1, beta2, eps, t,
                           rows=self.unique_ids, active=self.active_count, num_rows=self.num_unique,
                           R=self.R, err=self.err, stream=stream)
