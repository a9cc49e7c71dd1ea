"""Plain CPU oracle of the GBA push-step (test infrastructure only).

This module is the independent reference that the device library is checked
against.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import it; the product path never calls it.  It shares no code with the
device library and holds no kernel-shaped blocking or fusion: every function
follows the paper's definition in the paper's order, in float64, with float32
only where a stored result is float32.

Paper: Wang et al., "Global Batch gradients Aggregation (GBA) for training
recommendation models" (arXiv 2205.11048).

* Eq. 1 (Sec. 3.1): the staleness-decay (tolerance) function f.
* Alg. 2 (PS workflow, push responder): when N_a gradients are buffered, pop
  them, update each ID's tag of last appearance, decay dense gradients by the
  token, decay embedding gradients by the ID tag and the token, sum the dense
  gradients with the weights and divide by N_a, sum the embedding gradients
  with the weights and divide by how many workers sent the ID.
* App. B (workflows of GBA): part of the weighted sum may be taken ahead of
  time, from the tokens (the early weighted sum).
* Table 1 (Sec. 4.1): GBA runs with Adam; the asynchronous baseline with
  Adagrad.  The update rules are the textbook ones (Duchi, Hazan and Singer,
  JMLR 2011; Kingma and Ba, ICLR 2015), since the paper names them only.

Readings taken where the paper is silent or ambiguous (each is listed in the
design notes of the repository, with its reason):

* R1  K is the paper's M = N_a, the number of gradients aggregated per step.
* R2  Eq. 1 keeps s <= iota and excludes s > iota.  An excluded gradient is
      never read: its values cannot reach the result, even if they are NaN.
* R3  The dense divisor is K itself (excluded contributions still count).
* R4  The embedding divisor c_r is the number of contributions in the buffer
      that contain ID r, whatever their weight; a contribution with several
      occurrences of r counts once and its rows for r are summed.  The
      alternative ``norm="by_k"`` divides by K, which makes the all-fresh case
      equal to the synchronous global-batch gradient.
* R5  Per-ID decay ("id_tag"): with tag[r] the last global step at which row
      r was updated (-1 if never), the staleness of contribution m for row r
      is max(0, tag[r] - tau_m + 1), read before the tag is rewritten; tag[r]
      then becomes k for every row that received a non-zero weight.  The
      default ("token") gives every row of contribution m the weight of m.
* R6  Only active rows (at least one non-excluded contribution, W_r > 0) are
      updated.  The dense update always runs, with a zero gradient when every
      contribution is excluded.
* R7  Optimiser state is read as float32, updated in float64 and rounded once
      per stored value; Adam's bias corrections use one step count t for the
      dense vector and for rows (rows are updated lazily).
* R8  A token newer than the step being applied (tau_m > k) cannot occur by
      construction; it is an error.
* R9  The early weighted sum folds each arriving dense gradient, with its
      token weight for the step it will be applied at, into a float64 running
      sum in arrival order; the buffer order is the arrival order, so the
      result equals the one-shot sum bit for bit.  Embedding rows are kept as
      they arrive (their buffer is already O(sum of n_m D)) and reduced at the
      step.
* R10 The token of the i-th batch is floor(i / M): the text gives M batches
      per token value, in ascending order, while the printed formula divides
      by K, the number of updates; the M batches per value are followed.
"""
from __future__ import annotations

import numpy as np

DECAY_TOKEN = "token"
DECAY_ID_TAG = "id_tag"
NORM_PER_ID_COUNT = "per_id_count"
NORM_BY_K = "by_k"


# --------------------------------------------------------------------------
# Eq. 1: staleness and the tolerance function
# --------------------------------------------------------------------------
def token_weights(tokens, step: int, iota: int):
    """Eq. 1.  s_m = k - tau_m; f = 1 when s_m <= iota, else 0 (excluded).

    Returns (w float32 [K], s int64 [K], number of excluded contributions)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    s = np.int64(step) - tokens
    if np.any(s < 0):
        raise ValueError("token newer than the step being applied (R8)")
    w = np.where(s <= iota, 1.0, 0.0).astype(np.float32)
    return w, s, int(np.sum(w == 0))


# --------------------------------------------------------------------------
# Alg. 2: decayed dense gradients, weighted sum divided by N_a
# --------------------------------------------------------------------------
def aggregate_dense(grads, w):
    """g_bar = (sum over m with w_m != 0 of w_m * g_m) / K, summed in float64
    in buffer order and rounded to float32 once (Alg. 2; R2, R3).

    ``grads`` is a sequence of K float32 vectors (or a [K, P] array)."""
    K = len(grads)
    if K == 0:
        raise ValueError("K must be positive")
    P = len(grads[0])
    acc = np.zeros(P, dtype=np.float64)
    for m in range(K):
        if w[m] != 0:                               # excluded: never read (R2)
            acc += np.float64(w[m]) * np.asarray(grads[m], dtype=np.float64)
    return (acc / K).astype(np.float32)


def aggregate_dense_magnitude(grads, w):
    """Companion mu = (sum of |w_m g_m|) / K used by the comparison rule."""
    K = len(grads)
    acc = np.zeros(len(grads[0]), dtype=np.float64)
    for m in range(K):
        if w[m] != 0:
            acc += abs(np.float64(w[m])) * np.abs(np.asarray(grads[m], dtype=np.float64))
    return acc / K


# --------------------------------------------------------------------------
# App. B: the early weighted sum (contributions folded in as they arrive)
# --------------------------------------------------------------------------
def accumulate_dense(run, grads, w):
    """Fold arriving contributions into the float64 running sum, in arrival
    order: run += w_j * g_j for every j with w_j != 0 (App. B allows part of
    the weighted sum to be taken ahead of time; a weight depends only on the
    token and the step it is applied at).
    ``run`` is updated in place and returned."""
    for j in range(len(grads)):
        if w[j] != 0:                               # excluded: never read (R2)
            run += np.float64(w[j]) * np.asarray(grads[j], dtype=np.float64)
    return run


def finalize_dense(run, K: int):
    """g_bar = run / K, rounded to float32 once (Alg. 2's divisor N_a = K)."""
    if K <= 0:
        raise ValueError("K must be positive")
    return (run / K).astype(np.float32)


# --------------------------------------------------------------------------
# Alg. 2: embedding gradients by ID
# --------------------------------------------------------------------------
def contribution_of_occurrence(offsets):
    """m(j) for every occurrence j, from the contribution offsets [K + 1]."""
    offsets = np.asarray(offsets, dtype=np.int64)
    sizes = np.diff(offsets)
    if np.any(sizes < 0) or offsets[0] != 0:
        raise ValueError("contribution offsets must start at 0 and not decrease")
    return np.repeat(np.arange(len(sizes), dtype=np.int64), sizes)


def dedup(ids, offsets):
    """Distinct IDs in ascending order, the exclusive prefix of their
    occurrence counts, and c_r = number of contributions that contain r."""
    ids = np.asarray(ids, dtype=np.int64)
    m_of_j = contribution_of_occurrence(offsets)
    if m_of_j.size != ids.size:
        raise ValueError("offsets[K] must equal the number of occurrences")
    return dedup_occurrences(ids, m_of_j, len(offsets) - 1)


def dedup_occurrences(ids, m_of_j, K: int):
    """``dedup`` for occurrences given with their contribution index."""
    ids = np.asarray(ids, dtype=np.int64)
    unique_ids, counts = np.unique(ids, return_counts=True)
    seg_offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    # one (ID, contribution) pair per contribution that contains the ID (R4)
    pair_ids = np.unique(ids * np.int64(K) + m_of_j) // np.int64(K)
    contrib_count = np.bincount(np.searchsorted(unique_ids, pair_ids),
                                minlength=unique_ids.size).astype(np.int32)
    return unique_ids, seg_offsets, contrib_count


def row_weights(w, tokens, m_of_j, ids, iota: int, decay: str, tag=None):
    """Weight of each occurrence's (row, contribution) pair (Alg. 2; R5).

    token:  w_{m,r} = w_m.
    id_tag: w_{m,r} = 1 when max(0, tag[r] - tau_m + 1) <= iota, else 0."""
    w = np.asarray(w, dtype=np.float64)
    if decay == DECAY_TOKEN:
        return w[m_of_j]
    if decay == DECAY_ID_TAG:
        tau = np.asarray(tokens, dtype=np.int64)[m_of_j]
        s = np.maximum(0, np.asarray(tag, dtype=np.int64)[ids] - tau + 1)
        return np.where(s <= iota, 1.0, 0.0)
    raise ValueError(decay)


def aggregate_sparse(ids, rows, offsets, w, tokens, step: int, iota: int,
                     tag=None, decay: str = DECAY_TOKEN, norm: str = NORM_PER_ID_COUNT):
    """Alg. 2, embedding part, for one PS shard.

    ids: int64 [N] contribution-major; rows: float32 [N, D]; offsets: int64 [K+1];
    w, tokens: per contribution; tag: int32 [R] (id_tag mode only).

    Returns a dict with unique_ids, seg_offsets, contrib_count (c_r),
    active_count (W_r = contributions of r with non-zero weight), agg
    (float32 [U, D], the weighted sum divided by c_r, or by K), the
    magnitude companion agg_mu, and new_tag (id_tag mode)."""
    ids = np.asarray(ids, dtype=np.int64)
    m_of_j = contribution_of_occurrence(offsets)
    if m_of_j.size != ids.size:
        raise ValueError("offsets[K] must equal the number of occurrences")
    return aggregate_sparse_occurrences(ids, m_of_j, rows, len(offsets) - 1, w, tokens, step,
                                        iota, tag, decay, norm)


def aggregate_sparse_occurrences(ids, m_of_j, rows, K: int, w, tokens, step: int, iota: int,
                                 tag=None, decay: str = DECAY_TOKEN,
                                 norm: str = NORM_PER_ID_COUNT):
    """``aggregate_sparse`` for occurrences given with their contribution index
    (any subset that holds every occurrence of the IDs it contains)."""
    ids = np.asarray(ids, dtype=np.int64)
    m_of_j = np.asarray(m_of_j, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.float32)
    if decay == DECAY_ID_TAG and tag is None:
        raise ValueError("id_tag decay needs the tag array")
    D = rows.shape[1]
    unique_ids, seg_offsets, contrib_count = dedup_occurrences(ids, m_of_j, K)
    U = unique_ids.size
    seg_of_j = np.searchsorted(unique_ids, ids)

    # weights from the tags as they were before this step (R5)
    weight_j = row_weights(w, tokens, m_of_j, ids, iota, decay, tag)
    keep = weight_j != 0

    # W_r: distinct contributions of r with non-zero weight
    act_pairs = np.unique(ids[keep] * np.int64(K) + m_of_j[keep]) // np.int64(K)
    active_count = np.bincount(np.searchsorted(unique_ids, act_pairs),
                               minlength=U).astype(np.int32)

    # weighted sum in float64, in occurrence order; excluded rows are never read (R2)
    G = np.zeros((U, D), dtype=np.float64)
    mu = np.zeros((U, D), dtype=np.float64)
    contrib = weight_j[keep, None] * rows[keep].astype(np.float64)
    np.add.at(G, seg_of_j[keep], contrib)
    np.add.at(mu, seg_of_j[keep], np.abs(contrib))

    if norm == NORM_PER_ID_COUNT:
        div = np.maximum(contrib_count, 1).astype(np.float64)[:, None]
    elif norm == NORM_BY_K:
        div = np.float64(K)
    else:
        raise ValueError(norm)
    out = dict(unique_ids=unique_ids, seg_offsets=seg_offsets, contrib_count=contrib_count,
               active_count=active_count, agg=(G / div).astype(np.float32), agg_mu=mu / div,
               num_unique=U)
    if decay == DECAY_ID_TAG:
        new_tag = np.array(tag, dtype=np.int32, copy=True)
        new_tag[unique_ids[active_count > 0]] = step
        out["new_tag"] = new_tag
    return out


# --------------------------------------------------------------------------
# Sec. 3.1 token list and Alg. 2 pull responder
# --------------------------------------------------------------------------
def token_of_batch(i: int, M: int) -> int:
    """Token attached to the i-th batch of the data list: batches 0 .. M-1
    get 0, the next M batches 1, and so on (Sec. 3.1; R10)."""
    if i < 0 or M < 1:
        raise ValueError("i >= 0 and M >= 1 required")
    return i // M


def pull_rows(ids, table):
    """Rows of a worker's request, looked up once per distinct ID (Alg. 2,
    pull responder): the distinct IDs ascending, for each request position
    the index of its ID among them, and the table rows of the distinct IDs."""
    ids = np.asarray(ids, dtype=np.int64)
    unique_ids, inverse = np.unique(ids, return_inverse=True)
    return unique_ids, inverse.astype(np.int32), np.asarray(table)[unique_ids]


# --------------------------------------------------------------------------
# Optimisers (Table 1 names them; textbook rules, R7)
# --------------------------------------------------------------------------
def adagrad(param, accum, grad, lr: float, eps: float):
    """Duchi et al. 2011: a' = a + g^2; p' = p - lr g / (sqrt(a') + eps)."""
    p = np.asarray(param, np.float32).astype(np.float64)
    a = np.asarray(accum, np.float32).astype(np.float64)
    g = np.asarray(grad, np.float32).astype(np.float64)
    a_new = a + g * g
    p_new = p - lr * g / (np.sqrt(a_new) + eps)
    return p_new.astype(np.float32), a_new.astype(np.float32)


def adagrad_magnitude(param, accum, grad, grad_mu, lr: float, eps: float):
    """Companions (mu_p, mu_a) of the comparison rule for one Adagrad update."""
    p = np.asarray(param, np.float32).astype(np.float64)
    a = np.asarray(accum, np.float32).astype(np.float64)
    g = np.asarray(grad, np.float32).astype(np.float64)
    gm = np.maximum(np.asarray(grad_mu, np.float64), np.abs(g))
    a_new = a + g * g
    mu_a = a_new + 2.0 * np.abs(g) * gm
    p_new = p - lr * g / (np.sqrt(a_new) + eps)
    mu_p = np.abs(p_new) + np.abs(p) + lr * gm / (np.sqrt(a_new) + eps)
    return mu_p, mu_a


def adam(param, m, v, grad, lr: float, beta1: float, beta2: float, eps: float, t: int):
    """Kingma and Ba 2015, Alg. 1: m' = b1 m + (1-b1) g; v' = b2 v + (1-b2) g^2;
    p' = p - lr (m'/(1-b1^t)) / (sqrt(v'/(1-b2^t)) + eps)."""
    p = np.asarray(param, np.float32).astype(np.float64)
    m0 = np.asarray(m, np.float32).astype(np.float64)
    v0 = np.asarray(v, np.float32).astype(np.float64)
    g = np.asarray(grad, np.float32).astype(np.float64)
    m_new = beta1 * m0 + (1.0 - beta1) * g
    v_new = beta2 * v0 + (1.0 - beta2) * g * g
    m_hat = m_new / (1.0 - beta1 ** t)
    v_hat = v_new / (1.0 - beta2 ** t)
    p_new = p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p_new.astype(np.float32), m_new.astype(np.float32), v_new.astype(np.float32)


def adam_magnitude(param, m, v, grad, grad_mu, lr, beta1, beta2, eps, t):
    """Companions (mu_p, mu_m, mu_v) of the comparison rule for one Adam update."""
    p = np.asarray(param, np.float32).astype(np.float64)
    m0 = np.asarray(m, np.float32).astype(np.float64)
    v0 = np.asarray(v, np.float32).astype(np.float64)
    g = np.asarray(grad, np.float32).astype(np.float64)
    gm = np.maximum(np.asarray(grad_mu, np.float64), np.abs(g))
    m_new = beta1 * m0 + (1.0 - beta1) * g
    v_new = beta2 * v0 + (1.0 - beta2) * g * g
    mu_m = np.abs(m_new) + np.abs(beta1 * m0) + (1.0 - beta1) * gm
    mu_v = v_new + 2.0 * (1.0 - beta2) * np.abs(g) * gm
    v_hat = v_new / (1.0 - beta2 ** t)
    p_new = p - lr * (m_new / (1.0 - beta1 ** t)) / (np.sqrt(v_hat) + eps)
    mu_p = np.abs(p_new) + np.abs(p) + lr * (mu_m / (1.0 - beta1 ** t)) / (np.sqrt(v_hat) + eps)
    return mu_p, mu_m, mu_v


# --------------------------------------------------------------------------
# The whole push-step (Alg. 2 with the optimiser apply)
# --------------------------------------------------------------------------
def gba_step(tokens, step, iota, grads, ids, rows, offsets, param, dense_slots,
             table_rows_of, table_slot_rows_of, optimizer: str, hp: dict,
             tag=None, decay=DECAY_TOKEN, norm=NORM_PER_ID_COUNT, t=None, magnitudes=False):
    """One global step on one shard.

    ``table_rows_of(r_array)`` and ``table_slot_rows_of(slot, r_array)`` return
    the current float32 rows of the table and its slots for the given IDs, so
    a caller can serve rows of a large table without materialising it.

    Returns a dict: w, s, num_excluded, g_bar, param', dense slots', the
    sparse aggregate (see ``aggregate_sparse``), and for the active rows the
    updated table rows and slot rows (keyed by ``active_ids``).  With
    ``magnitudes``, also each updated value's magnitude companion (``*_mu``)
    for the comparison rule."""
    w, s, n_ex = token_weights(tokens, step, iota)
    g_bar = aggregate_dense(grads, w)
    sp = aggregate_sparse(ids, rows, offsets, w, tokens, step, iota, tag, decay, norm)
    active = sp["unique_ids"][sp["active_count"] > 0]
    act_agg = sp["agg"][sp["active_count"] > 0]
    E = table_rows_of(active)
    act_mu = sp["agg_mu"][sp["active_count"] > 0]
    g_mu = aggregate_dense_magnitude(grads, w) if magnitudes else None
    if optimizer == "adagrad":
        p_new, a_new = adagrad(param, dense_slots[0], g_bar, hp["lr"], hp["eps"])
        S0 = table_slot_rows_of(0, active)
        e_new, ea_new = adagrad(E, S0, act_agg, hp["lr"], hp["eps"])
        dense_new, rows_new = [a_new], [ea_new]
        if magnitudes:
            mu_p, mu_a = adagrad_magnitude(param, dense_slots[0], g_bar, g_mu, hp["lr"], hp["eps"])
            mu_e, mu_ea = adagrad_magnitude(E, S0, act_agg, act_mu, hp["lr"], hp["eps"])
            dense_mu, rows_mu = [mu_a], [mu_ea]
    elif optimizer == "adam":
        p_new, m_new, v_new = adam(param, dense_slots[0], dense_slots[1], g_bar, hp["lr"],
                                   hp["beta1"], hp["beta2"], hp["eps"], t)
        S0, S1 = table_slot_rows_of(0, active), table_slot_rows_of(1, active)
        e_new, em_new, ev_new = adam(E, S0, S1, act_agg, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], t)
        dense_new, rows_new = [m_new, v_new], [em_new, ev_new]
        if magnitudes:
            mu_p, mu_m, mu_v = adam_magnitude(param, dense_slots[0], dense_slots[1], g_bar, g_mu, hp["lr"],
                                              hp["beta1"], hp["beta2"], hp["eps"], t)
            mu_e, mu_em, mu_ev = adam_magnitude(E, S0, S1, act_agg, act_mu, hp["lr"], hp["beta1"],
                                                hp["beta2"], hp["eps"], t)
            dense_mu, rows_mu = [mu_m, mu_v], [mu_em, mu_ev]
    else:
        raise ValueError(optimizer)
    out = dict(w=w, s=s, num_excluded=n_ex, g_bar=g_bar, param=p_new, dense_slots=dense_new,
               sparse=sp, active_ids=active, table_rows=e_new, table_slot_rows=rows_new)
    if magnitudes:
        out.update(param_mu=mu_p, dense_slots_mu=dense_mu, table_rows_mu=mu_e, table_slot_rows_mu=rows_mu)
    return out
