"""Plain fp64 CPU oracle of the beam step that feeds the paged rearrangement.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import, call or time this module.  It
shares no code with the HIP path.

What is computed (GRACE, arXiv 2608.00938):

* Beam score update (Sec. 3.1).  After the constraint filter removes invalid or
  ineligible next tokens, each surviving candidate (beam m, token v) scores the
  beam's accumulated log-probability plus the token's log-probability.
* Beam top-k (Sec. 3.1, Sec. 3.3).  Per request, the k best of the M_t * |V|
  candidates become the next step's beams; with dynamic per-step widths
  (M_1, ..., M_L) the selection at step t keeps k = M_{t+1}.
* Paged rearrangement with dynamic widths (Sec. 3.3, Sec. 5.3).  New row
  r = b*M_cur + j copies the block ids of its parent row b*M_prev + p_r and
  takes a fresh block for the current position.

Readings where the paper is silent (each also listed in the design notes):

* The token log-probability is the log-softmax of the row's logits over the
  whole vocabulary; the filter then drops candidates (score -inf).  There is no
  renormalisation over the surviving tokens.
* Candidates are totally ordered by score (descending), then by flat index
  ``m*|V| + v`` (ascending): the lowest index wins a tie.  -0.0 equals +0.0;
  NaN ranks below every number, -inf included.
* Top-k always returns k candidates in that order; when fewer than k are
  finite, the rest are filtered (-inf) candidates, i.e. dead beams whose
  descendants keep score -inf.
* Pools hold slab t with B*M_t rows at a fixed row stride R_s >= B*max_t M_t;
  the fresh block of (step t, row r) is ``t*R_s + r``.
"""
from __future__ import annotations

import numpy as np

__all__ = ["log_softmax", "candidate_scores", "order_keys", "topk_select", "beam_topk",
           "fresh_block_dyn", "kv_append_table_dyn", "unpack_mask"]


def log_softmax(x) -> np.ndarray:
    """log(softmax(x)) over the last axis in fp64, shifted by the row maximum."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.max(axis=-1, keepdims=True)
    return x - mu - np.log(np.exp(x - mu).sum(axis=-1, keepdims=True))


def unpack_mask(bits, V: int) -> np.ndarray:
    """Bool [R, V] from the packed filter: bit (v % 32) of word v // 32, 1 = allowed."""
    bits = np.asarray(bits, dtype=np.uint32)
    v = np.arange(V)
    return ((bits[:, v // 32] >> (v % 32).astype(np.uint32)) & 1).astype(bool)


def candidate_scores(logits, prev_scores, allowed=None) -> np.ndarray:
    """Score of every (beam row, token) candidate: prefix score + token log-prob (Sec. 3.1).

    logits [R, V]; prev_scores [R]; allowed: bool [R, V] or None (all allowed).
    Filtered candidates score -inf.
    """
    s = np.asarray(prev_scores, dtype=np.float64)[:, None] + log_softmax(logits)
    if allowed is not None:
        s = np.where(np.asarray(allowed, dtype=bool), s, -np.inf)
    return s


def order_keys(scores) -> tuple[np.ndarray, np.ndarray]:
    """(primary, nan) sort keys realising the reading's order for one request."""
    s = np.asarray(scores, dtype=np.float64)
    nan = np.isnan(s)
    return np.where(nan, -np.inf, s), nan


def topk_select(scores, k: int):
    """Indices and scores of the k best candidates of one request, in order.

    scores: [N] (any float dtype; compared exactly).  Order: NaN last, then
    score descending, then index ascending.  Brute force: one stable sort.
    """
    s = np.asarray(scores)
    prim, nan = order_keys(s)
    idx = np.arange(s.shape[0])
    order = np.lexsort((idx, -prim, nan))   # last key is the primary one
    sel = order[:k]
    return sel.astype(np.int64), s[sel]


def beam_topk(cand, B: int, M: int, V: int, k: int):
    """Per-request top-k over the M*V candidates of request b.

    cand: [B*M, V] candidate scores (row b*M + m).  Returns parents (request-local
    beam in [0, M)), tokens and scores, each [B, k], the k selected in order.
    """
    cand = np.asarray(cand)
    parents = np.empty((B, k), dtype=np.int64)
    tokens = np.empty((B, k), dtype=np.int64)
    scores = np.empty((B, k), dtype=cand.dtype)
    for b in range(B):
        idx, sc = topk_select(cand[b * M:(b + 1) * M].reshape(-1), k)
        parents[b], tokens[b], scores[b] = idx // V, idx % V, sc
    return parents, tokens, scores


def fresh_block_dyn(step: int, r, R_s: int):
    """Fresh block of (step, row r) with slab row stride R_s."""
    return step * R_s + np.asarray(r, dtype=np.int64)


def kv_append_table_dyn(table_prev, parents, B: int, M_prev: int, M_cur: int, step: int,
                        R_s: int) -> np.ndarray:
    """Block table after the rearrangement at ``step`` with widths M_prev -> M_cur.

    table_prev: [B*M_prev, >= step]; parents: [B*M_cur] request-local parents in
    [0, M_prev) (ignored at step 0).  Row r = b*M_cur + j copies row
    b*M_prev + parents[r] for positions < step (Sec. 3.3, Sec. 5.3).
    Returns int64 [B*M_cur, step + 1].
    """
    R = B * M_cur
    table = np.empty((R, step + 1), dtype=np.int64)
    if step > 0:
        prev = np.asarray(table_prev, dtype=np.int64)
        r = np.arange(R)
        parent_row = (r // M_cur) * M_prev + np.asarray(parents, dtype=np.int64)
        table[:, :step] = prev[parent_row, :step]
    table[:, step] = fresh_block_dyn(step, np.arange(R), R_s)
    return table
