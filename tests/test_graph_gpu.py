"""A whole decode loop (layers x steps of cross-attention and fused paged
self-attention, then score update and top-k feeding the next step's parents)
recorded as one HIP graph.

The graph is replayed several times with eager library work, host
synchronisations and overwritten outputs in between; every replay must
reproduce every output of the eager run exactly.  After a replay, every output
of every layer and step is also checked against the oracle, fed with the
parents the loop itself chose on the GPU: attention outputs within 2e-2, block
tables (the last two steps': the two tables alternate), filter words and trie
nodes bit-exact, and each step's selection a
valid top-k of the fp64 candidate scores (scores within 1e-4).
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import beam_oracle as BO
from oracle import gtm_oracle as GO
from paper_2608_00938_amd import decode as D
from paper_2608_00938_amd import grace as G
from paper_2608_00938_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _make_loop(dev, B=2, widths=(1, 8, 16, 16), H=2, d=64, V=64, layers=2, L=24, seed=31,
               gtm=None):
    wl = W.custom(dtype="bf16", B=B, M=max(widths), H=H, d=d, steps=len(widths), L=L)
    inp = W.DecodeInputs(wl, seed, dev)
    ek, ev = inp.enc_kv
    off = inp.offsets_tensor()
    step_inputs = []
    for l in range(layers):
        per = []
        for t, M in enumerate(widths):
            g = lambda tag: W.normal((B * M, H, d), seed + 100 * l, tag, t, wl, dev)  # noqa: E731
            per.append(dict(q_cross=g("q_cross"), q_self=g("q_self"), k_new=g("k_new"),
                            v_new=g("v_new")))
        step_inputs.append(per)
    logits = [W.beam_logits(seed, t, B * M, V, "bf16", dev) for t, M in enumerate(widths)]
    masks = [torch.from_numpy(W.beam_mask(seed, t, B * M, V, keep=0.7).view(np.int32)).to(dev)
             for t, M in enumerate(widths)]
    loop = D.DecodeLoop(B, widths, H, d, V, layers, ek, ev, off, step_inputs, logits, masks,
                        gtm=gtm)
    return loop, inp


def _gtm(dev, B, seed=41):
    ix = W.gtm_index(seed, 20000)
    return ix, (G.GtmIndex(ix, dev), G.GtmUsers(_users(B, seed), dev))


def _users(B, seed=41):
    return W.gtm_users(seed, B, L_max=16)


def _snapshot(loop):
    outs = []
    for l in range(loop.layers):
        outs += [x.clone() for x in loop.x_cross[l]] + [x.clone() for x in loop.x_self[l]]
    outs += [x.clone() for x in loop.parents + loop.tokens + loop.scores]
    if loop.gtm is not None:
        outs += [x.clone() for x in loop.masks + loop.nodes[1:]]
    return outs + [x.clone() for x in _written_slabs(loop)]


def _written_slabs(loop):
    """The pool rows the loop writes: slab t, rows 0 .. B*M_t - 1 (the rest is padding)."""
    out = []
    for c in loop.caches:
        for t, M in enumerate(loop.widths):
            out += [c.k_pool[t, :loop.B * M], c.v_pool[t, :loop.B * M]]
    return out


def _current(loop):
    outs = []
    for l in range(loop.layers):
        outs += list(loop.x_cross[l]) + list(loop.x_self[l])
    outs += list(loop.parents + loop.tokens + loop.scores)
    if loop.gtm is not None:
        outs += list(loop.masks + loop.nodes[1:])
    return outs + _written_slabs(loop)


@pytest.mark.parametrize("with_gtm", [False, True], ids=["given_masks", "cd_gtm"])
def test_decode_loop_graph_replays_match_eager(gpu, with_gtm):
    gtm = _gtm(gpu, 2)[1] if with_gtm else None
    loop, _ = _make_loop(gpu, V=512 if with_gtm else 64, gtm=gtm)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        loop.run()
    stream.synchronize()
    ref = _snapshot(loop)
    _log(f"[graph] eager loop done; {len(ref)} outputs")
    graph = loop.capture(stream)
    other, _ = _make_loop(gpu, seed=77)          # unrelated eager work between replays
    for rep in range(3):
        for x in _current(loop):
            x.fill_(-1) if x.dtype in (torch.int32,) else x.fill_(float("nan"))
        with torch.cuda.stream(stream):
            other.run()
        torch.cuda.synchronize()
        graph.launch(stream)
        stream.synchronize()
        for i, (a, b) in enumerate(zip(_current(loop), ref)):
            same = torch.equal(a.view(torch.uint8) if a.dtype != torch.int32 else a,
                               b.view(torch.uint8) if b.dtype != torch.int32 else b)
            assert same, f"replay {rep}: output {i} differs"
        _log(f"  replay {rep}: all outputs identical to the eager run")
    graph.destroy()


def test_decode_loop_wiring(gpu):
    """Step 0 cross-attention matches the oracle; every row's table starts with
    its request's step-0 block (M_0 = 1 beam per request: every beam descends
    from it), checked on the last step's table."""
    loop, inp = _make_loop(gpu)
    loop.run()
    torch.cuda.synchronize()
    f = lambda t: t.float().cpu().numpy().astype(np.float64)  # noqa: E731
    q = loop.inputs[0][0]["q_cross"]
    ref = oracle.cross_attn(f(q), f(loop.enc_k), f(loop.enc_v), inp.offsets, loop.widths[0],
                            1 / math.sqrt(loop.d))
    assert np.max(np.abs(f(loop.x_cross[0][0]) - ref)) <= 2e-2
    assert int(loop.parents[0].max()) == 0 and int(loop.parents[0].min()) == 0
    t = loop.T - 1
    Mt = loop.widths[t]
    for c in loop.caches:
        tab = c.table(t)[:loop.B * Mt].cpu().numpy()
        assert tab[:, 0].tolist() == [r // Mt for r in range(loop.B * Mt)]
        assert tab[:, t].tolist() == [t * c.B * c.M + r for r in range(loop.B * Mt)]
    for c in loop.caches:
        assert int(c.err_flag.item()) == 0


def test_graph_capture_on_null_stream_is_refused(gpu):
    with pytest.raises(G.GraceError):
        G.capture(lambda: None, torch.cuda.default_stream())


def test_decode_loop_with_filter_follows_the_trie(gpu):
    """With the CD+GTM filter in the loop, every finite beam's token sequence is a
    prefix of a valid SID (its node is real), and its trie node is the walk of
    its tokens (reconstructed from parents on the host)."""
    B = 2
    ix, gtm = _gtm(gpu, B)
    loop, _ = _make_loop(gpu, V=512, gtm=gtm)
    loop.run()
    torch.cuda.synchronize()
    assert int(loop.gtm_err.item()) == 0
    off, tok, child = ix["node_offsets"], ix["tokens"], ix["child_nodes"]
    T = loop.T
    par = [p.cpu().numpy() for p in loop.parents]
    toks = [t.cpu().numpy() for t in loop.tokens]
    sc = loop.scores[-1].cpu().numpy()
    node_last = loop.nodes[T].cpu().numpy().reshape(B, -1)
    for b in range(B):
        for j in range(sc.shape[1]):
            if not np.isfinite(sc[b, j]):
                continue
            seq, jj = [], j
            for t in range(T - 1, -1, -1):          # walk back through the parents
                seq.append(int(toks[t][b, jj]))
                jj = int(par[t][b, jj])
            seq.reverse()
            node = 0
            for v in seq:                            # walk down the trie
                rng = range(off[node], off[node + 1])
                hit = [e for e in rng if tok[e] == v]
                assert hit, (b, j, seq)
                node = int(child[hit[0]])
            assert node == node_last[b, j]


def _f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _check_topk(cand, par, tok, sc, B, M, V, k, eps=1e-4):
    """The GPU's selection is a top-k of the fp64 candidates up to the scores'
    error: k distinct candidates, each within eps of the k-th best score or
    above it, every candidate clearly above the k-th taken, the reported
    scores those of the selected candidates (-inf exactly), best first."""
    for b in range(B):
        s = cand[b * M:(b + 1) * M].reshape(-1)
        kth = np.sort(s)[::-1][k - 1]
        sel = par[b].astype(np.int64) * V + tok[b]
        assert np.all((par[b] >= 0) & (par[b] < M)) and np.all((tok[b] >= 0) & (tok[b] < V))
        assert len(set(sel.tolist())) == k
        assert np.all(s[sel] >= kth - eps)
        clearly = np.nonzero(s > kth + eps)[0]
        assert set(clearly.tolist()) <= set(sel.tolist())
        ref = s[sel]
        fin = np.isfinite(ref)
        assert np.array_equal(np.isneginf(sc[b]), np.isneginf(ref))
        assert np.all(np.abs(sc[b][fin] - ref[fin]) <= eps)
        assert np.all(np.diff(sc[b][fin]) <= 0) and np.all(fin[:fin.sum()])


@pytest.mark.parametrize("with_gtm", [False, True], ids=["given_masks", "cd_gtm"])
def test_decode_loop_matches_oracle(gpu, with_gtm):
    """The replayed loop at widths (1, 8, 16, 16), two layers, against the
    oracle at every layer and step."""
    B = 2
    ix = us = None
    gtm = None
    if with_gtm:
        ix, gtm = _gtm(gpu, B)
        us = _users(B)
    loop, inp = _make_loop(gpu, V=512 if with_gtm else 64, gtm=gtm)
    stream = torch.cuda.Stream()
    graph = loop.capture(stream)
    graph.launch(stream)
    stream.synchronize()
    graph.destroy()
    _log(f"[graph oracle] widths {loop.widths} layers {loop.layers} gtm={with_gtm}")
    B, V, H, d, T = loop.B, loop.V, loop.H, loop.d, loop.T
    R_s = B * max(loop.widths)
    scale = 1.0 / math.sqrt(d)
    ek, ev = _f64(loop.enc_k), _f64(loop.enc_v)
    par = [p.cpu().numpy() for p in loop.parents]
    tok = [x.cpu().numpy() for x in loop.tokens]
    sc = [x.cpu().numpy().astype(np.float64) for x in loop.scores]
    tables = [None] * loop.layers
    pools = [(np.zeros((T, R_s, H, d)), np.zeros((T, R_s, H, d))) for _ in range(loop.layers)]
    worst_c = worst_s = 0.0
    for t, M in enumerate(loop.widths):
        M_prev = loop.widths[t - 1] if t > 0 else 1
        R = B * M
        par_t = par[t - 1].reshape(-1) if t > 0 else None
        for l in range(loop.layers):
            x = loop.inputs[l][t]
            ref = oracle.cross_attn(_f64(x["q_cross"]), ek, ev, inp.offsets, M, scale)
            err = float(np.max(np.abs(_f64(loop.x_cross[l][t]) - ref)))
            assert err <= 2e-2, (l, t, "cross", err)
            worst_c = max(worst_c, err)
            tnew = BO.kv_append_table_dyn(tables[l], par_t, B, M_prev, M, t, R_s)
            if t >= T - 2:   # the two tables alternate: the last two steps' survive the loop
                got = loop.caches[l].table(t)[:R, :t + 1].cpu().numpy()
                assert np.array_equal(got, tnew), (l, t, "table")
            full = np.zeros((R, T), dtype=np.int64)
            full[:, :t + 1] = tnew
            tables[l] = full
            kp, vp = pools[l]
            kp[t, :R] = _f64(x["k_new"])
            vp[t, :R] = _f64(x["v_new"])
            ref = oracle.self_attn_step(_f64(x["q_self"]), kp, vp, full, t, scale)
            err = float(np.max(np.abs(_f64(loop.x_self[l][t]) - ref)))
            assert err <= 2e-2, (l, t, "self", err)
            worst_s = max(worst_s, err)
        # the filter of this step's beams
        if with_gtm:
            nodes = loop.nodes[t].cpu().numpy()
            allowed = GO.gtm_mask(ix, us, nodes, B, M)
            words = loop.masks[t].cpu().numpy().view(np.uint32)
            assert np.array_equal(words, GO.pack_mask(allowed)), (t, "mask")
        else:
            allowed = BO.unpack_mask(loop.masks[t].cpu().numpy().view(np.uint32), V)
        prev = np.zeros(R) if t == 0 else sc[t - 1].reshape(-1)
        cand = BO.candidate_scores(_f64(loop.logits[t]), prev, allowed)
        _check_topk(cand, par[t], tok[t], sc[t], B, M, V, loop.k_out[t])
        if with_gtm:
            nxt = GO.trie_advance(ix, loop.nodes[t].cpu().numpy(), par[t].reshape(-1),
                                  tok[t].reshape(-1), B, M, loop.k_out[t])
            assert np.array_equal(loop.nodes[t + 1].cpu().numpy(), nxt), (t, "trie")
        _log(f"  step {t} (M {M_prev}->{M}): attention, tables, filter and top-k match")
    _log(f"  worst cross err {worst_c:.3e}, worst self err {worst_s:.3e}")
    for c in loop.caches:
        assert int(c.err_flag.item()) == 0
    if with_gtm:
        assert int(loop.gtm_err.item()) == 0
