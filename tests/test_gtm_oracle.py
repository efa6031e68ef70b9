"""Pins of the CD+GTM oracle (constraint filter and trie step).

Independent of the oracle's code path: the paper's printed toy example
(``tests/golden/gtm_toy_bitmask.txt``), closed Bloom-containment cases, a trie
rebuilt from the SID list with Python sets, ad-level brute force (the node test
must never reject a child that holds an eligible ad: the union test is
conservative, Sec. 4.2-4.3), and exactness where a node holds a single ad.
"""
import os

import numpy as np
import pytest

from oracle import gtm_oracle as GO
from paper_2608_00938_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits(s):
    """'110 11' -> packed uint64 word, first character = bit 0."""
    w = 0
    for i, ch in enumerate(s.replace(" ", "")):
        w |= (ch == "1") << i
    return np.array([w], dtype=np.uint64)


def _golden():
    vals = {}
    for ln in open(os.path.join(GOLDEN, "gtm_toy_bitmask.txt")):
        if "=" in ln and not ln.startswith("#"):
            k, v = ln.split("=")
            vals[k.strip()] = v.strip()
    return vals


def test_paper_toy_bitmask_example():
    g = _golden()
    ad1, ad2, node, user = (_bits(g[k]) for k in ("ad_us_18_24", "ad_ca_25_34", "node_union", "user_us_30"))
    assert np.array_equal(ad1 | ad2, node)
    assert GO.bitmask_pass(node, user) == bool(int(g["node_passes"]))
    assert GO.bitmask_pass(ad1, user) == bool(int(g["ad_us_18_24_passes"]))
    assert GO.bitmask_pass(ad2, user) == bool(int(g["ad_ca_25_34_passes"]))
    # a UK user fails the node: country 001 does not meet 110
    assert not GO.bitmask_pass(node, _bits("001 01"))


def test_toy_index_through_gtm_mask():
    g = _golden()
    node = _bits(g["node_union"])
    index = {"vocab": 4, "node_offsets": np.array([0, 2, 2, 2]), "child_nodes": np.array([1, 2]),
             "tokens": np.array([0, 3], dtype=np.int16), "bitmask_index": np.array([0, 1]),
             "bloom_index": np.array([0, 0]),
             "bitmask_table": np.array([[node[0]], [_bits("001 11")[0]]], dtype=np.uint64),
             "bloom_table": np.array([[np.uint64(0xFFFFFFFFFFFFFFFF)]], dtype=np.uint64)}
    user = {"bitmask": np.array([[_bits(g["user_us_30"])[0]]], dtype=np.uint64),
            "bloom": np.array([[[np.uint64(1)]]], dtype=np.uint64), "n_loc": np.array([1])}
    allowed = GO.gtm_mask(index, user, [0], B=1, M=1)
    assert allowed.tolist() == [[True, False, False, False]]
    assert GO.pack_mask(allowed).tolist() == [[1]]
    # no locations: the Bloom test is an ANY over nothing
    user0 = dict(user, n_loc=np.array([0]))
    assert not GO.gtm_mask(index, user0, [0], 1, 1).any()
    # a dead beam has no children
    assert not GO.gtm_mask(index, user, [-1], 1, 1).any()


def test_bloom_containment_cases():
    loc_a = np.array([0b1011, 0], dtype=np.uint64)
    loc_b = np.array([0, 0b11 << 60], dtype=np.uint64)
    matcher = loc_a | np.array([0b10000, 1], dtype=np.uint64)
    assert GO.bloom_pass(matcher, [loc_a])
    assert not GO.bloom_pass(matcher, [loc_b])
    assert GO.bloom_pass(matcher, [loc_b, loc_a])      # ANY of many
    assert not GO.bloom_pass(matcher, [])
    partial = np.array([0b0011, 0], dtype=np.uint64)    # misses one bit of loc_a
    assert not GO.bloom_pass(partial, [loc_a])


def test_pack_mask_bit_order():
    a = np.zeros((1, 70), dtype=bool)
    a[0, [0, 31, 32, 69]] = True
    assert GO.pack_mask(a).tolist() == [[1 | (1 << 31), 1, 1 << 5]]


@pytest.fixture(scope="module")
def small():
    return W.gtm_index(3, 3000), W.gtm_users(3, 3, L_max=8)


def _prefix_children(sids):
    """prefix tuple -> set of next tokens, from the SID list (Python sets)."""
    ch = {}
    for s in sids.tolist():
        for l in range(len(s)):
            ch.setdefault(tuple(s[:l]), set()).add(s[l])
    return ch


def _node_prefixes(index):
    """node id -> prefix tuple, walking the CSR from the root."""
    off, tok, child = index["node_offsets"], index["tokens"], index["child_nodes"]
    pre = {0: ()}
    stack = [0]
    while stack:
        p = stack.pop()
        for e in range(off[p], off[p + 1]):
            pre[int(child[e])] = pre[p] + (int(tok[e]),)
            stack.append(int(child[e]))
    return pre


def test_constrained_decoding_equals_trie_children(small):
    index, users = small
    ones = dict(index, bitmask_table=np.full_like(index["bitmask_table"], 0xFFFFFFFFFFFFFFFF),
                bloom_table=np.full_like(index["bloom_table"], 0xFFFFFFFFFFFFFFFF))
    ch = _prefix_children(index["sids"])
    pre = _node_prefixes(index)
    rng = np.random.default_rng(0)
    nodes = rng.choice(list(pre.keys()), size=3 * 40)
    allowed = GO.gtm_mask(ones, users, nodes, B=3, M=40)
    for r, n in enumerate(nodes):
        want = ch.get(pre[int(n)], set())
        assert set(np.nonzero(allowed[r])[0].tolist()) == want


def _ad_eligible(index, users, b, ads):
    u = users["bitmask"][b]
    locs = users["bloom"][b][: users["n_loc"][b]]
    return [GO.bitmask_pass(index["ad_bitmask"][a], u) and GO.bloom_pass(index["ad_bloom"][a], locs)
            for a in ads]


def test_union_test_is_conservative_and_exact_for_single_ads(small):
    """No child holding an eligible ad is filtered (Sec. 4.2-4.3); where the child
    subtree holds exactly one ad, the node test is the ad test."""
    index, users = small
    pre = _node_prefixes(index)
    sid_of = {tuple(s): i for i, s in enumerate(index["sids"].tolist())}
    ads_of_sid = {}
    for a, s in enumerate(index["ad_sid"].tolist()):
        ads_of_sid.setdefault(s, []).append(a)
    ads_under = {}
    for s, i in sid_of.items():
        for l in range(len(s) + 1):
            ads_under.setdefault(s[:l], []).extend(ads_of_sid[i])
    rng = np.random.default_rng(1)
    nodes = rng.choice(list(pre.keys()), size=3 * 60)
    allowed = GO.gtm_mask(index, users, nodes, B=3, M=60)
    checked = exact = 0
    for r, n in enumerate(nodes):
        b = r // 60
        p = pre[int(n)]
        for v in range(index["vocab"]):
            ads = ads_under.get(p + (v,))
            if not ads:
                assert not allowed[r, v]
                continue
            elig = _ad_eligible(index, users, b, ads)
            if any(elig):
                assert allowed[r, v]
                checked += 1
            if len(ads) == 1:
                assert allowed[r, v] == elig[0]
                exact += 1
    assert checked > 0 and exact > 0


def test_trie_advance_matches_prefix_walk(small):
    index, _ = small
    pre = _node_prefixes(index)
    node_of = {v: k for k, v in pre.items()}
    ch = _prefix_children(index["sids"])
    rng = np.random.default_rng(2)
    B, M, k = 2, 30, 25
    prev = rng.choice(list(pre.keys()), size=B * M)
    parents = rng.integers(0, M, size=B * k)
    tokens = np.empty(B * k, dtype=np.int64)
    for i in range(B * k):
        p = pre[int(prev[(i // k) * M + parents[i]])]
        kids = sorted(ch.get(p, []))
        tokens[i] = kids[rng.integers(0, len(kids))] if kids and rng.random() < 0.8 else 511
    prev[0] = -1
    got = GO.trie_advance(index, prev, parents, tokens, B, M, k)
    for i in range(B * k):
        pn = int(prev[(i // k) * M + parents[i]])
        want = node_of.get(pre[pn] + (int(tokens[i]),), -1) if pn >= 0 else -1
        assert got[i] == want
