"""Pins of the beam-step oracle (score update, top-k, dynamic-width tables).

Each pin is independent of the oracle's code path: pure-Python brute force with
``math`` and ``sorted``, closed forms, invariants, and small examples worked by
hand.  A slip in the oracle (log-softmax without the max shift or the log-sum,
wrong tie-break, NaN/-0 order, parent/token decode swapped, parent row taken
with the wrong width) fails at least one of them.
"""
import math

import numpy as np
import pytest

from oracle import beam_oracle as BO


def _py_key(score, idx):
    """Python sort key of the reading's order: NaN last, score descending, index ascending."""
    if math.isnan(score):
        return (1, 0.0, idx)
    return (0, -score, idx)


def _py_topk(scores, k):
    order = sorted(range(len(scores)), key=lambda i: _py_key(float(scores[i]), i))
    return order[:k]


def test_log_softmax_closed_forms():
    V = 7
    assert np.allclose(BO.log_softmax(np.zeros((1, V))), -math.log(V), atol=1e-15, rtol=0)
    a, b = 1.25, -3.5
    got = BO.log_softmax(np.array([[a, b]]))[0]
    # log(e^a / (e^a + e^b)) = -log1p(e^(b-a))
    assert got[0] == pytest.approx(-math.log1p(math.exp(b - a)), abs=1e-15)
    assert got[1] == pytest.approx(-math.log1p(math.exp(a - b)), abs=1e-15)


def test_log_softmax_invariants():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 33)) * 4
    ls = BO.log_softmax(x)
    assert np.allclose(np.exp(ls).sum(axis=1), 1.0, atol=1e-14)
    assert np.allclose(BO.log_softmax(x + 1000.0), ls, atol=1e-12)   # shift invariance
    assert np.all(ls <= 0)
    # huge logits: the max shift keeps it finite
    assert np.isfinite(BO.log_softmax(np.array([[1e4, 0.0, -1e4]]))).all()


def test_candidate_scores_brute_force():
    rng = np.random.default_rng(1)
    R, V = 3, 5
    logits = rng.standard_normal((R, V))
    prev = np.array([-1.5, 0.0, -7.25])
    allowed = rng.random((R, V)) < 0.6
    got = BO.candidate_scores(logits, prev, allowed)
    for r in range(R):
        z = sum(math.exp(x) for x in logits[r])
        for v in range(V):
            want = prev[r] + logits[r, v] - math.log(z) if allowed[r, v] else -math.inf
            if allowed[r, v]:
                assert got[r, v] == pytest.approx(want, abs=1e-13)
            else:
                assert got[r, v] == -math.inf


def test_unpack_mask_bit_order():
    bits = np.array([[0b101, 0x80000000]], dtype=np.uint32)
    m = BO.unpack_mask(bits, 64)
    assert m[0, 0] and not m[0, 1] and m[0, 2] and m[0, 63]
    assert m.sum() == 3


def test_topk_matches_python_sort_with_ties_and_specials():
    rng = np.random.default_rng(2)
    for trial in range(20):
        n = int(rng.integers(1, 300))
        s = rng.choice(np.array([-1.0, -0.5, 0.0, -0.0, -np.inf, np.nan, 2.0, -3.25], dtype=np.float32),
                       size=n)
        s = np.where(rng.random(n) < 0.5, s, rng.standard_normal(n).astype(np.float32))
        k = int(rng.integers(1, n + 1))
        idx, sc = BO.topk_select(s, k)
        want = _py_topk(s.tolist(), k)
        assert idx.tolist() == want
        assert np.array_equal(sc, s[want], equal_nan=True)


def test_topk_zero_signs_tie_and_nan_last():
    s = np.array([np.nan, -0.0, 0.0, -np.inf, -0.0], dtype=np.float32)
    idx, _ = BO.topk_select(s, 5)
    assert idx.tolist() == [1, 2, 4, 3, 0]


def test_beam_topk_hand_example():
    # B=1, M=2, V=3; flat index m*V + v
    cand = np.array([[-1.0, -0.5, -3.0],
                     [-0.2, -np.inf, -0.5]])
    parents, tokens, scores = BO.beam_topk(cand, B=1, M=2, V=3, k=4)
    assert parents.tolist() == [[1, 0, 1, 0]]
    assert tokens.tolist() == [[0, 1, 2, 0]]
    assert scores.tolist() == [[-0.2, -0.5, -0.5, -1.0]]


def test_beam_topk_fewer_finite_than_k_gives_dead_beams():
    cand = np.full((2, 4), -np.inf)
    cand[1, 2] = -3.0
    parents, tokens, scores = BO.beam_topk(cand, B=1, M=2, V=4, k=3)
    assert parents.tolist() == [[1, 0, 0]] and tokens.tolist() == [[2, 0, 1]]
    assert scores[0, 0] == -3.0 and np.all(np.isneginf(scores[0, 1:]))


def test_first_step_topk_is_logit_order():
    """M_1 = 1: log-softmax is monotone, so the k best tokens are the k largest logits."""
    rng = np.random.default_rng(3)
    V, k = 64, 10
    logits = rng.standard_normal((1, V))
    cand = BO.candidate_scores(logits, np.array([0.0]))
    parents, tokens, _ = BO.beam_topk(cand, B=1, M=1, V=V, k=k)
    assert np.all(parents == 0)
    assert tokens[0].tolist() == sorted(range(V), key=lambda v: -logits[0, v])[:k]


def test_dynamic_table_hand_example():
    # B=2, widths 2 -> 3, step 1, slab row stride 8
    table_prev = np.zeros((4, 4), dtype=np.int64)
    table_prev[:, 0] = [0, 1, 2, 3]            # fresh blocks of step 0
    parents = np.array([1, 0, 1, 0, 0, 1])
    t = BO.kv_append_table_dyn(table_prev, parents, B=2, M_prev=2, M_cur=3, step=1, R_s=8)
    assert t[:, 0].tolist() == [1, 0, 1, 2, 2, 3]
    assert t[:, 1].tolist() == [8, 9, 10, 11, 12, 13]


def test_dynamic_table_step0_ignores_parents():
    t = BO.kv_append_table_dyn(None, None, B=3, M_prev=1, M_cur=1, step=0, R_s=5)
    assert t.tolist() == [[0], [1], [2]]
