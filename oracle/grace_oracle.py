"""Plain, slow, fp64 CPU oracle of one wide-beam decode step's attention.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import, call or time this module.  It
shares no code with the HIP path: no kernels, headers, helpers or tables.

What is computed (GRACE, arXiv 2608.00938):

* Cross-attention in the beam-as-query layout (Sec. 5.1, App. B).  The M beams
  of request b are the query sequence of one attention call against that
  request's encoder K/V, per head: ``O = softmax(scale * Q_bh K_bh^T) V_bh``.
  The layout change is exact: the result equals M independent one-query
  attentions (App. B).
* Paged beam rearrangement (Sec. 3.3, Sec. 5.3).  A block holds one generated
  token's k/v of one beam row across all heads; the block table row of new beam
  i copies its parent's ids for positions ``j < t``, ``P_new[i, j] = P[p_i, j]``,
  and position t gets a fresh block holding the current token.
* Short-prefix self-attention (Sec. 5.2, Sec. 5.3).  Beam row r at step t
  attends over the t+1 blocks ``P_t[r, 0..t]`` (its prefix 0..t, no other mask).

Readings where the paper is silent (each is listed with its reason in the
design notes): softmax scale is an explicit argument (default 1/sqrt(d));
prefix length at step t is t+1; parents are request-local; the beam width is
B*M rows at every step, step 0 included, and parents are ignored at step 0; the
fresh block of (step t, row r) is ``t*R + r``, i.e. slab t row r of a pool laid
out ``[T_max, R, H, d]``; an empty encoder sequence (L_b = 0) attends to nothing
and yields a zero output row.

Everything is float64; inputs (bf16 or fp32) are upcast exactly.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "softmax", "attend", "cross_attn_request", "cross_attn", "fresh_block",
    "kv_append_table", "kv_append", "self_attn_step", "table_rows", "self_attn_rows",
]


def _f64(x) -> np.ndarray:
    """Exact upcast to float64 (accepts numpy arrays or CPU torch tensors)."""
    if hasattr(x, "detach"):
        x = x.detach().cpu().float().numpy()   # bf16 -> fp32 is exact
    return np.asarray(x, dtype=np.float64)


def softmax(S: np.ndarray) -> np.ndarray:
    """Row softmax over the last axis, shifted by the row maximum before exp."""
    mu = S.max(axis=-1, keepdims=True)
    E = np.exp(S - mu)
    return E / E.sum(axis=-1, keepdims=True)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float,
           return_probs: bool = False):
    """Scaled dot-product attention of queries q [n, d] over keys K [L, d], values V [L, d].

    This is the SDPA call the beam-as-query layout feeds (Sec. 5.1):
    ``softmax(scale * q K^T) V``.  With L = 0 the output is zero (reading above).
    """
    n, d = q.shape
    if K.shape[0] == 0:
        out = np.zeros((n, V.shape[1]))
        return (out, np.zeros((n, 0))) if return_probs else out
    S = scale * (q @ K.T)
    P = softmax(S)
    out = P @ V
    return (out, P) if return_probs else out


def cross_attn_request(q_rows, K_b, V_b, scale: float, return_probs: bool = False):
    """Cross-attention of one request's beam queries against its shared encoder K/V.

    q_rows: [n, H, d] beam queries of request b (any subset of its M beams);
    K_b, V_b: [L_b, H, d].  Per head h, the beams form the query sequence of a
    single attention call over ``K_b[:, h]`` and ``V_b[:, h]`` (Sec. 5.1, App. B).
    Returns [n, H, d] (and probabilities [n, H, L_b] if asked).
    """
    q_rows, K_b, V_b = _f64(q_rows), _f64(K_b), _f64(V_b)
    n, H, d = q_rows.shape
    out = np.empty((n, H, V_b.shape[2]))
    probs = np.empty((n, H, K_b.shape[0]))
    for h in range(H):
        o, p = attend(q_rows[:, h, :], K_b[:, h, :], V_b[:, h, :], scale, return_probs=True)
        out[:, h, :] = o
        probs[:, h, :] = p
    return (out, probs) if return_probs else out


def cross_attn(q, enc_k, enc_v, enc_off, M: int, scale: float, return_probs: bool = False):
    """Cross-attention of all beam rows, beam-as-query per request (Sec. 5.1, App. B).

    q: [B*M, H, d] with row r = b*M + m (request-major, App. B);
    enc_k, enc_v: packed [sum L, H, d]; enc_off: [B+1] offsets (request b owns
    rows ``enc_off[b]:enc_off[b+1]``).  Returns out [B*M, H, d] and, if asked,
    a list of per-request probabilities [M, H, L_b].
    """
    q, enc_k, enc_v = _f64(q), _f64(enc_k), _f64(enc_v)
    off = np.asarray(enc_off, dtype=np.int64)
    B = off.shape[0] - 1
    assert q.shape[0] == B * M
    out = np.empty((B * M, q.shape[1], enc_v.shape[2]))
    probs = []
    for b in range(B):
        rows = slice(b * M, (b + 1) * M)
        kv = slice(off[b], off[b + 1])
        o, p = cross_attn_request(q[rows], enc_k[kv], enc_v[kv], scale, return_probs=True)
        out[rows] = o
        probs.append(p)
    return (out, probs) if return_probs else out


def fresh_block(step: int, r, R: int):
    """Physical id of the fresh block that holds row r's token of step ``step``."""
    return step * R + np.asarray(r, dtype=np.int64)


def kv_append_table(table_prev, parents, B: int, M: int, step: int) -> np.ndarray:
    """Block table after paged beam rearrangement at ``step`` (Sec. 3.3, Sec. 5.3).

    table_prev: [B*M, >= step] ids for positions 0..step-1 (ignored at step 0);
    parents: [B*M] request-local parent beam of each new row (ignored at step 0).
    Row i = b*M + m copies its parent's prefix ids, ``P_new[i, j] = P[b*M + p_i, j]``
    for j < step, and takes the fresh block of (step, i) at position ``step``.
    Returns int64 [B*M, step + 1].
    """
    R = B * M
    table = np.empty((R, step + 1), dtype=np.int64)
    if step > 0:
        prev = np.asarray(table_prev, dtype=np.int64)
        par = np.asarray(parents, dtype=np.int64)
        parent_row = (np.arange(R) // M) * M + par
        table[:, :step] = prev[parent_row, :step]
    table[:, step] = fresh_block(step, np.arange(R), R)
    return table


def kv_append(k_pool, v_pool, table_prev, parents, k_new, v_new, B: int, M: int, step: int):
    """Full paged update: the new table plus pools whose slab ``step`` holds k_new/v_new.

    Pools are [T_max, B*M, H, d]; block id ``t*R + r`` is slab t row r.
    Returns (k_pool', v_pool', table [B*M, step+1]) without modifying the inputs.
    """
    kp, vp = np.array(_f64(k_pool)), np.array(_f64(v_pool))
    kp[step] = _f64(k_new)
    vp[step] = _f64(v_new)
    return kp, vp, kv_append_table(table_prev, parents, B, M, step)


def self_attn_rows(q_rows, k_prefix, v_prefix, scale: float, return_probs: bool = False):
    """Self-attention of each row's query over its own gathered prefix.

    q_rows: [n, H, d]; k_prefix, v_prefix: [n, T, H, d] (T = step + 1 tokens in
    prefix order).  No mask: the prefix is all a row sees (Sec. 5.2).
    Returns [n, H, d] (and probabilities [n, H, T] if asked).
    """
    q_rows, k_prefix, v_prefix = _f64(q_rows), _f64(k_prefix), _f64(v_prefix)
    n, H, d = q_rows.shape
    out = np.empty((n, H, v_prefix.shape[3]))
    probs = np.empty((n, H, k_prefix.shape[1]))
    for h in range(H):
        # one single-query attention per row, evaluated for all rows at once
        S = scale * np.einsum("nd,ntd->nt", q_rows[:, h, :], k_prefix[:, :, h, :])
        P = softmax(S)
        out[:, h, :] = np.einsum("nt,ntd->nd", P, v_prefix[:, :, h, :])
        probs[:, h, :] = P
    return (out, probs) if return_probs else out


def self_attn_step(q, k_pool, v_pool, table, step: int, scale: float, return_probs: bool = False):
    """Paged self-attention at ``step`` (Sec. 5.2, Sec. 5.3).

    q: [R, H, d]; pools [T_max, R, H, d]; table: [R, >= step+1] block ids.
    Row r gathers blocks ``table[r, 0..step]`` in prefix order and attends over them.
    """
    q, kp, vp = _f64(q), _f64(k_pool), _f64(v_pool)
    T_max, R, H, d = kp.shape
    kflat = kp.reshape(T_max * R, H, d)
    vflat = vp.reshape(T_max * R, H, vp.shape[3])
    ids = np.asarray(table, dtype=np.int64)[:, :step + 1]
    return self_attn_rows(q, kflat[ids], vflat[ids], scale, return_probs=return_probs)


def table_rows(rows, step: int, parents_by_step, B: int, M: int) -> np.ndarray:
    """Block-table rows ``P_step[rows, 0..step]`` from the parents alone.

    Unrolls the paged update rule over steps for a subset of rows: position
    ``step`` of row r is its fresh block; walking back, the row that owns
    position j-1's entry is the parent (mapped to a global row) of the row that
    owns position j.  ``parents_by_step[s]`` is the [B*M] request-local parent
    array of step s (entry 0 unused).  Returns int64 [len(rows), step + 1].
    """
    R = B * M
    cur = np.asarray(rows, dtype=np.int64).copy()
    out = np.empty((cur.shape[0], step + 1), dtype=np.int64)
    for j in range(step, -1, -1):
        out[:, j] = fresh_block(j, cur, R)
        if j > 0:
            par = np.asarray(parents_by_step[j], dtype=np.int64)
            cur = (cur // M) * M + par[cur]
    return out
