"""Parity of the CD+GTM constraint filter and the trie step with the oracle,
through the C ABI on the GPU.  Both are integer/bit work: compared bit-exactly.
The index is synthetic (the paper's 30M-SID index and targeting data are not
public); its form follows Sec. 4.4 and App. A."""
import sys

import numpy as np
import pytest
import torch

from oracle import beam_oracle as BO
from oracle import gtm_oracle as GO
from paper_2608_00938_amd import grace as G
from paper_2608_00938_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def small():
    return W.gtm_index(3, 3000), W.gtm_users(3, 3, L_max=8)


@pytest.fixture(scope="module")
def medium():
    return W.gtm_index(4, 100_000), W.gtm_users(4, 8, L_max=64)


def _mask_np(t):
    return t.cpu().numpy().view(np.uint32)


def test_gtm_mask_full_parity_small(gpu, small):
    ix, us = small
    gi, gu = G.GtmIndex(ix, gpu), G.GtmUsers(us, gpu)
    B, M = 3, 40
    rng = np.random.default_rng(0)
    nodes = np.concatenate([W.gtm_beam_nodes(5, ix, 1, M, level) for level in range(3)])
    nodes = rng.permutation(nodes)[:B * M].astype(np.int32)
    nodes[:3] = [-1, 0, 0]                  # a dead beam and the root twice
    err = torch.zeros(1, dtype=torch.int32, device=gpu)
    got = G.grace_gtm_mask(gi, gu, torch.from_numpy(nodes).to(gpu), B, M, err_flag=err)
    torch.cuda.synchronize()
    want = GO.pack_mask(GO.gtm_mask(ix, us, nodes, B, M))
    assert np.array_equal(_mask_np(got), want)
    assert int(err.item()) == 0
    _log(f"  allowed tokens per beam: mean {np.unpackbits(want.view(np.uint8)).sum() / (B * M):.1f}")


@pytest.mark.parametrize("level", [1, 2, 3])
def test_gtm_mask_sampled_parity_medium(gpu, medium, level):
    ix, us = medium
    gi, gu = G.GtmIndex(ix, gpu), G.GtmUsers(us, gpu)
    B, M = 8, 512
    nodes = W.gtm_beam_nodes(6, ix, B, M, level)
    _log(f"[gtm] level {level}: {B}x{M} beams, {ix['num_nodes']} nodes")
    got = _mask_np(G.grace_gtm_mask(gi, gu, torch.from_numpy(nodes).to(gpu), B, M))
    rows = np.random.default_rng(level).choice(B * M, size=96, replace=False)
    for r in rows:
        b = r // M
        sub = {"bitmask": us["bitmask"][b:b + 1], "bloom": us["bloom"][b:b + 1],
               "n_loc": us["n_loc"][b:b + 1]}
        want = GO.pack_mask(GO.gtm_mask(ix, sub, nodes[r:r + 1], 1, 1))[0]
        assert np.array_equal(got[r], want), f"row {r}"


def test_gtm_mask_flags_bad_index_data(gpu, small):
    ix, us = small
    bad = dict(ix)
    bad["tokens"] = ix["tokens"].copy()
    bad["bitmask_index"] = ix["bitmask_index"].copy()
    e0 = ix["node_offsets"][0]
    bad["tokens"][e0] = 600                  # token past the vocabulary
    bad["bitmask_index"][e0 + 1] = 10 ** 7   # matcher row past the table
    gi, gu = G.GtmIndex(bad, gpu), G.GtmUsers(us, gpu)
    err = torch.zeros(1, dtype=torch.int32, device=gpu)
    nodes = torch.tensor([0, -1, 0], dtype=torch.int32, device=gpu)
    got = _mask_np(G.grace_gtm_mask(gi, gu, nodes, 3, 1, err_flag=err))
    torch.cuda.synchronize()
    assert int(err.item()) == 1
    want = GO.pack_mask(GO.gtm_mask(bad, us, nodes.cpu().numpy(), 3, 1))
    assert np.array_equal(got, want)
    err.zero_()
    G.grace_gtm_mask(gi, gu, torch.tensor([ix["num_nodes"]], dtype=torch.int32, device=gpu), 1, 1,
                     err_flag=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 1


def test_trie_advance_parity(gpu, medium):
    ix, _ = medium
    gi = G.GtmIndex(ix, gpu)
    B, Mp, k = 4, 64, 50
    rng = np.random.default_rng(3)
    prev = W.gtm_beam_nodes(7, ix, B, Mp, 2)
    prev[5] = -1
    parents = rng.integers(0, Mp, size=B * k).astype(np.int32)
    off, tok = ix["node_offsets"], ix["tokens"]
    tokens = np.empty(B * k, dtype=np.int32)
    for i in range(B * k):
        p = prev[(i // k) * Mp + parents[i]]
        kids = tok[off[p]:off[p + 1]] if p >= 0 else []
        tokens[i] = rng.choice(kids) if len(kids) and rng.random() < 0.85 else 511
    got = G.grace_trie_advance(gi, torch.from_numpy(prev).to(gpu), torch.from_numpy(parents).to(gpu),
                               torch.from_numpy(tokens).to(gpu), B, Mp, k).cpu().numpy()
    want = GO.trie_advance(ix, prev, parents, tokens, B, Mp, k)
    assert np.array_equal(got, want)
    assert (want == -1).any() and (want >= 0).any()


def test_filter_scores_topk_advance_chain(gpu, medium):
    """Filter -> score update -> top-k -> trie step on the GPU: every finite
    selected candidate is an allowed child and moves to a real node; dead picks
    (score -inf) are the only ones that may lead nowhere."""
    ix, us = medium
    gi, gu = G.GtmIndex(ix, gpu), G.GtmUsers(us, gpu)
    B, M, V, k = 8, 256, ix["vocab"], 256
    nodes = torch.from_numpy(W.gtm_beam_nodes(8, ix, B, M, 2)).to(gpu)
    mask = G.grace_gtm_mask(gi, gu, nodes, B, M)
    logits = W.beam_logits(8, 2, B * M, V, "bf16", gpu)
    prev = torch.from_numpy(W.beam_prev_scores(8, 2, B * M)).to(gpu)
    cand, rmax = G.grace_beam_scores(logits, prev, mask)
    par, tok, sc = G.grace_beam_topk(cand, B, M, k, row_max=rmax)
    nxt = G.grace_trie_advance(gi, nodes, par.view(-1), tok.view(-1), B, M, k)
    torch.cuda.synchronize()
    sc, nxt = sc.view(-1).cpu().numpy(), nxt.cpu().numpy()
    assert np.all(nxt[np.isfinite(sc)] >= 0)
    allowed = BO.unpack_mask(_mask_np(mask), V)
    par, tok = par.view(-1).cpu().numpy(), tok.view(-1).cpu().numpy()
    rows = (np.arange(B * k) // k) * M + par
    assert np.all(allowed[rows[np.isfinite(sc)], tok[np.isfinite(sc)]])
    assert np.all(~allowed[rows[~np.isfinite(sc)], tok[~np.isfinite(sc)]])
