"""Plain CPU oracle of the decode-time constraint filter (CD + GTM) and the trie step.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import, call or time this module.  It
shares no code with the HIP path.

What is computed (GRACE, arXiv 2608.00938, Sec. 4, Sec. 5.4 and App. A):

* Constrained decoding.  A beam sits at trie node p (its SID prefix).  Token v
  is admissible only if p||v is a prefix of a valid SID, i.e. v labels one of
  p's child entries in the CSR index (node offsets -> child-entry range).
* Target matching.  The child entry names a bitmask matcher row and a Bloom
  matcher row (deduplicated tables).  The bitmask test passes when every bit
  of the request's bitmask is present in the node matcher:
  ``(matcher & user) == user`` over all packed words (Sec. 4.2).  The Bloom
  test passes when at least one of the request's location filters is
  contained in the node matcher: ``(loc & matcher) == loc`` (Sec. 4.3).  The
  token survives when both pass.
* Trie step.  A selected (parent beam, token) moves the new beam to the child
  node reached by that token.

Readings where the paper is silent (also listed in the design notes):

* The request's location list may be empty; then the Bloom test is an ANY
  over nothing and fails, so no token survives (the lookup's any() reading).
* A beam whose node id is negative or not a node is dead: it has no children.
* Matcher ids or tokens out of range make that child entry fail.
* Within a node's child range, tokens are unique and ascending; a selected
  token that is not a child (a filtered candidate kept as a dead beam) leads to
  node -1.
* The filter is returned as packed uint32 words, 32 tokens per word, bit
  v % 32 of word v // 32 set = token v allowed (the beam score update's input).
"""
from __future__ import annotations

import numpy as np

__all__ = ["bitmask_pass", "bloom_pass", "gtm_mask", "pack_mask", "trie_advance"]


def bitmask_pass(matcher_words, user_words) -> bool:
    """Every user attribute bit is present in the node matcher (Sec. 4.2)."""
    m = np.asarray(matcher_words, dtype=np.uint64)
    u = np.asarray(user_words, dtype=np.uint64)
    return bool(np.all((m & u) == u))


def bloom_pass(matcher_words, user_locations) -> bool:
    """Some user location's filter is contained in the node matcher (Sec. 4.3)."""
    m = np.asarray(matcher_words, dtype=np.uint64)
    for loc in user_locations:
        q = np.asarray(loc, dtype=np.uint64)
        if np.all((q & m) == q):
            return True
    return False


def gtm_mask(index: dict, user: dict, node_ids, B: int, M: int) -> np.ndarray:
    """Allowed-token matrix bool [B*M, V] of the beams at ``node_ids`` (row b*M + m).

    index: node_offsets [N+1], tokens [E], bitmask_index [E], bloom_index [E],
    bitmask_table [rows, W_bm], bloom_table [rows, W_bl] (uint64), vocab V.
    user: bitmask [B, W_bm], bloom [B, L_max, W_bl] (uint64), n_loc [B].
    """
    V = int(index["vocab"])
    off = np.asarray(index["node_offsets"], dtype=np.int64)
    tok = np.asarray(index["tokens"], dtype=np.int64)
    bmi = np.asarray(index["bitmask_index"], dtype=np.int64)
    bli = np.asarray(index["bloom_index"], dtype=np.int64)
    bmt, blt = index["bitmask_table"], index["bloom_table"]
    n_nodes = off.shape[0] - 1
    nodes = np.asarray(node_ids, dtype=np.int64)
    allowed = np.zeros((B * M, V), dtype=bool)
    for r in range(B * M):
        p = nodes[r]
        if p < 0 or p >= n_nodes:
            continue                                  # dead beam: no children
        b = r // M
        u = user["bitmask"][b]
        locs = user["bloom"][b][: int(user["n_loc"][b])]
        for e in range(off[p], off[p + 1]):           # the node's child entries
            v = tok[e]
            if not (0 <= v < V):
                continue
            if not (0 <= bmi[e] < bmt.shape[0]) or not (0 <= bli[e] < blt.shape[0]):
                continue
            if bitmask_pass(bmt[bmi[e]], u) and bloom_pass(blt[bli[e]], locs):
                allowed[r, v] = True
    return allowed


def pack_mask(allowed) -> np.ndarray:
    """uint32 words [R, ceil(V/32)] of a bool [R, V] filter (bit v % 32 of word v // 32)."""
    a = np.asarray(allowed, dtype=bool)
    R, V = a.shape
    W = (V + 31) // 32
    out = np.zeros((R, W), dtype=np.uint64)
    for v in range(V):
        out[:, v // 32] |= a[:, v].astype(np.uint64) << np.uint64(v % 32)
    return out.astype(np.uint32)


def trie_advance(index: dict, node_prev, parents, tokens, B: int, M_prev: int, k: int) -> np.ndarray:
    """Node of each new beam: the child of its parent's node reached by its token.

    node_prev [B*M_prev]; parents, tokens [B*k] (request-local parents).
    Returns int64 [B*k]; -1 for dead parents or tokens that are not children.
    """
    off = np.asarray(index["node_offsets"], dtype=np.int64)
    tok = np.asarray(index["tokens"], dtype=np.int64)
    child = np.asarray(index["child_nodes"], dtype=np.int64)
    n_nodes = off.shape[0] - 1
    prev = np.asarray(node_prev, dtype=np.int64)
    par = np.asarray(parents, dtype=np.int64)
    tk = np.asarray(tokens, dtype=np.int64)
    out = np.full(B * k, -1, dtype=np.int64)
    for i in range(B * k):
        b = i // k
        p = prev[b * M_prev + par[i]]
        if p < 0 or p >= n_nodes:
            continue
        rng = np.arange(off[p], off[p + 1])
        hit = rng[tok[rng] == tk[i]]
        if hit.size:
            out[i] = child[hit[0]]
    return out
