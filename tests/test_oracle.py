"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each pin is independent of the oracle's own code path: pure-Python brute force
(scalar loops with ``math.exp``), a library routine on a differently laid out
problem (torch's float64 SDPA), closed forms, invariants and the paper's own
printed worked example and table.  A plausible slip in the oracle (dropped
scale, transposed operand, swapped K/V, wrong parent row, off-by-one prefix,
no max shift, wrong request offsets) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2608_00938_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL = 1e-12


def _rand(rng, *shape):
    return rng.standard_normal(shape)


# ----------------------------------------------------------------------------
# pure-Python brute force
# ----------------------------------------------------------------------------

def _bf_attend(q, keys, vals, scale):
    """One query (list) over lists of keys/values, scalar loops, math.exp."""
    if not keys:
        return [0.0] * len(q)
    s = [scale * sum(qi * ki for qi, ki in zip(q, k)) for k in keys]
    mx = max(s)
    e = [math.exp(x - mx) for x in s]
    z = sum(e)
    return [sum(e[j] / z * vals[j][c] for j in range(len(keys))) for c in range(len(vals[0]))]


def _bf_cross_unshared(q, enc_k, enc_v, off, M, scale):
    """The layout before the reshape (Sec. 5.1): every beam row gets its own copy of
    its request's K/V, [B*M, H, L, d], and runs a one-query attention."""
    R, H, d = q.shape
    out = np.zeros((R, H, enc_v.shape[2]))
    for r in range(R):
        b = r // M
        kcopy = [enc_k[j].tolist() for j in range(off[b], off[b + 1])]   # per-beam copy
        vcopy = [enc_v[j].tolist() for j in range(off[b], off[b + 1])]
        for h in range(H):
            out[r, h] = _bf_attend(q[r, h].tolist(), [k[h] for k in kcopy],
                                   [v[h] for v in vcopy], scale)
    return out


def _bf_full_history(qs, ks, vs, parents, B, M, scale):
    """Dense rearrangement (Sec. 3.3): each new beam row copies its parent's whole
    token history, then appends its own token; attention over the history."""
    R = B * M
    hist = [[(ks[0][r], vs[0][r])] for r in range(R)]
    outs = []
    for t in range(len(qs)):
        if t > 0:
            hist = [list(hist[(r // M) * M + int(parents[t][r])]) + [(ks[t][r], vs[t][r])]
                    for r in range(R)]
        H = qs[t].shape[1]
        o = np.zeros_like(qs[t])
        for r in range(R):
            for h in range(H):
                o[r, h] = _bf_attend(qs[t][r, h].tolist(), [kk[h].tolist() for kk, _ in hist[r]],
                                     [vv[h].tolist() for _, vv in hist[r]], scale)
        outs.append(o)
    return outs


def _paged_decode(qs, ks, vs, parents, B, M, scale, T_max=None):
    """Run the oracle's paged path over all steps; returns outputs, tables, pools."""
    T = len(qs)
    T_max = T_max or T
    R, H, d = qs[0].shape
    kp = np.zeros((T_max, R, H, d))
    vp = np.zeros((T_max, R, H, d))
    table = np.zeros((R, T_max), dtype=np.int64)
    outs, tables = [], []
    for t in range(T):
        kp, vp, tnew = oracle.kv_append(kp, vp, table, parents[t], ks[t], vs[t], B, M, t)
        table = np.zeros((R, T_max), dtype=np.int64)
        table[:, :t + 1] = tnew
        outs.append(oracle.self_attn_step(qs[t], kp, vp, table, t, scale))
        tables.append(tnew)
    return outs, tables, kp, vp


def _decode_inputs(rng, B, M, H, d, T):
    qs = [_rand(rng, B * M, H, d) for _ in range(T)]
    ks = [_rand(rng, B * M, H, d) for _ in range(T)]
    vs = [_rand(rng, B * M, H, d) for _ in range(T)]
    parents = [None] + [rng.integers(0, M, size=B * M) for _ in range(1, T)]
    return qs, ks, vs, parents


# ----------------------------------------------------------------------------
# cross-attention pins
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_c1_shared_equals_unshared_bruteforce(seed):
    """App. B: the beam-as-query layout is layout-only; ragged requests included."""
    rng = np.random.default_rng(seed)
    B, M, H, d = 3, 5, 2, 8
    lens = [1, 7, 4]
    off = np.concatenate([[0], np.cumsum(lens)])
    q = _rand(rng, B * M, H, d)
    k = _rand(rng, off[-1], H, d)
    v = _rand(rng, off[-1], H, d)
    scale = 1 / math.sqrt(d)
    got = oracle.cross_attn(q, k, v, off, M, scale)
    ref = _bf_cross_unshared(q, k, v, off, M, scale)
    assert np.max(np.abs(got - ref)) <= TOL


@pytest.mark.parametrize("d,scale", [(32, None), (64, 0.3), (16, 2.0)])
def test_c2_matches_torch_sdpa_on_paper_view(d, scale):
    """The paper's view/permute to [B, H, M, d] followed by SDPA (Sec. 5.1), in float64."""
    rng = np.random.default_rng(d)
    B, M, H, L = 2, 6, 3, 9
    q = _rand(rng, B * M, H, d)
    k = _rand(rng, B * L, H, d)
    v = _rand(rng, B * L, H, d)
    off = np.arange(B + 1) * L
    sc = 1 / math.sqrt(d) if scale is None else scale
    got = oracle.cross_attn(q, k, v, off, M, sc)
    tq = torch.from_numpy(q).view(B, M, H, 1, d).permute(0, 2, 1, 3, 4).reshape(B, H, M, d)
    tk = torch.from_numpy(k).view(B, L, H, d).permute(0, 2, 1, 3)
    tv = torch.from_numpy(v).view(B, L, H, d).permute(0, 2, 1, 3)
    x = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=sc)
    X = x.reshape(B, H, M, 1, d).permute(0, 2, 1, 3, 4).reshape(B * M, H, d).numpy()
    assert np.max(np.abs(got - X)) <= TOL


def test_c3_closed_forms():
    rng = np.random.default_rng(7)
    H, d, M = 2, 8, 4
    # one encoder token: every beam reads that token's value exactly
    q = _rand(rng, M, H, d)
    k1 = _rand(rng, 1, H, d)
    v1 = _rand(rng, 1, H, d)
    out = oracle.cross_attn(q, k1, v1, [0, 1], M, 0.5)
    assert np.array_equal(out, np.broadcast_to(v1, out.shape))
    # zero query, or all keys identical: uniform weights, output = mean value
    L = 6
    k = _rand(rng, L, H, d)
    v = _rand(rng, L, H, d)
    out = oracle.cross_attn(np.zeros((M, H, d)), k, v, [0, L], M, 1.0)
    assert np.max(np.abs(out - v.mean(axis=0))) <= TOL
    ksame = np.broadcast_to(k[:1], k.shape).copy()
    out = oracle.cross_attn(q, ksame, v, [0, L], M, 0.7)
    assert np.max(np.abs(out - v.mean(axis=0))) <= TOL
    # a query far along one key of an orthogonal set selects that key's value;
    # scores ~1e4 also check the max shift (exp would overflow without it)
    kk = np.zeros((L, H, d))
    for j in range(L):
        kk[j, :, j] = 1.0
    qq = np.zeros((M, H, d))
    qq[:, :, 3] = 1e4
    out = oracle.cross_attn(qq, kk, v, [0, L], M, 1.0)
    assert np.all(np.isfinite(out))
    assert np.max(np.abs(out - v[3])) <= TOL
    # empty encoder sequence attends to nothing: zero rows
    out = oracle.cross_attn(q, np.zeros((0, H, d)), np.zeros((0, H, d)), [0, 0], M, 1.0)
    assert np.array_equal(out, np.zeros_like(out))


def test_c4_softmax_rows_are_distributions():
    rng = np.random.default_rng(11)
    B, M, H, d = 2, 7, 3, 16
    off = [0, 5, 13]
    _, probs = oracle.cross_attn(_rand(rng, B * M, H, d), _rand(rng, 13, H, d),
                                 _rand(rng, 13, H, d), off, M, 0.25, return_probs=True)
    for p in probs:
        assert np.all(p >= 0)
        assert np.max(np.abs(p.sum(axis=-1) - 1)) <= TOL


def test_c5_equivariance_and_ragged_concatenation():
    rng = np.random.default_rng(5)
    B, M, H, d = 3, 6, 2, 8
    lens = [3, 9, 1]
    off = np.concatenate([[0], np.cumsum(lens)])
    q = _rand(rng, B * M, H, d)
    k = _rand(rng, off[-1], H, d)
    v = _rand(rng, off[-1], H, d)
    full = oracle.cross_attn(q, k, v, off, M, 0.4)
    # permuting the beams of a request permutes its output rows
    perm = np.concatenate([b * M + rng.permutation(M) for b in range(B)])
    assert np.max(np.abs(oracle.cross_attn(q[perm], k, v, off, M, 0.4) - full[perm])) <= TOL
    # a ragged batch equals its requests run one at a time
    for b in range(B):
        one = oracle.cross_attn(q[b * M:(b + 1) * M], k[off[b]:off[b + 1]], v[off[b]:off[b + 1]],
                                [0, lens[b]], M, 0.4)
        assert np.array_equal(one, full[b * M:(b + 1) * M])


# ----------------------------------------------------------------------------
# self-attention pins
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("seed,B,M,T", [(0, 2, 3, 4), (1, 1, 5, 5), (2, 3, 2, 3)])
def test_s1_paged_equals_full_history(seed, B, M, T):
    """Sec. 3.3 / Sec. 5.3: copying block ids equals copying the parent's KV bytes."""
    rng = np.random.default_rng(seed)
    H, d = 2, 4
    qs, ks, vs, parents = _decode_inputs(rng, B, M, H, d, T)
    paged, tables, _, _ = _paged_decode(qs, ks, vs, parents, B, M, 0.5)
    dense = _bf_full_history(qs, ks, vs, parents, B, M, 0.5)
    for t in range(T):
        assert np.max(np.abs(paged[t] - dense[t])) <= TOL
        # the row-subset recursion reproduces the full tables
        rows = np.arange(B * M)
        assert np.array_equal(oracle.table_rows(rows, t, parents, B, M), tables[t])


def test_s1_parents_are_request_local():
    """Parent p of row b*M+m names beam p of the same request (App. B: no mixing)."""
    B, M = 3, 4
    prev = np.arange(B * M)[:, None] * 10 + np.arange(2)[None, :]
    par = np.array([3, 0, 0, 1] * B)
    t = oracle.kv_append_table(prev, par, B, M, 2)
    for r in range(B * M):
        src = (r // M) * M + par[r]
        assert list(t[r, :2]) == list(prev[src, :2])
        assert t[r, 2] == 2 * B * M + r


def test_s2_first_step_returns_v_new():
    rng = np.random.default_rng(3)
    q, k, v = _rand(rng, 6, 2, 8), _rand(rng, 6, 2, 8), _rand(rng, 6, 2, 8)
    outs, _, _, _ = _paged_decode([q], [k], [v], [None], 2, 3, 0.9)
    assert np.array_equal(outs[0], v)


def test_s3_identity_parents_is_plain_decode_attention():
    """With every beam its own parent, the paged cache is an ordinary per-row KV cache."""
    rng = np.random.default_rng(4)
    B, M, H, d, T = 2, 3, 2, 8, 4
    qs, ks, vs, _ = _decode_inputs(rng, B, M, H, d, T)
    parents = [None] + [np.tile(np.arange(M), B) for _ in range(1, T)]
    paged, _, _, _ = _paged_decode(qs, ks, vs, parents, B, M, 0.35)
    for t in range(T):
        K = torch.from_numpy(np.stack(ks[:t + 1], axis=2)).permute(0, 1, 2, 3)   # [R, H, t+1, d]
        V = torch.from_numpy(np.stack(vs[:t + 1], axis=2))
        Q = torch.from_numpy(qs[t])[:, :, None, :]
        x = torch.nn.functional.scaled_dot_product_attention(Q, K, V, scale=0.35)[:, :, 0, :]
        assert np.max(np.abs(paged[t] - x.numpy())) <= TOL


def test_s4_common_parent_shares_blocks():
    rng = np.random.default_rng(8)
    B, M, H, d, T = 1, 4, 2, 4, 3
    qs, ks, vs, _ = _decode_inputs(rng, B, M, H, d, T)
    parents = [None] + [np.full(M, 2) for _ in range(1, T)]
    for t in range(1, T):   # rows 0 and 1 get identical query and new token
        qs[t][1], ks[t][1], vs[t][1] = qs[t][0], ks[t][0], vs[t][0]
    outs, tables, _, _ = _paged_decode(qs, ks, vs, parents, B, M, 0.5)
    for t in range(1, T):
        assert np.all(tables[t][:, :t] == tables[t][0, :t])
        assert np.array_equal(outs[t][0], outs[t][1])


def _mask_from_golden():
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "block_diag_mask_g4_t3.txt"))
            if ln.strip() and not ln.startswith("#")]
    return np.array(rows, dtype=np.int64)


def _coalesced_tile(q_rows, k_pref, v_pref, scale, mask):
    """Sec. 5.2's coalesced tile: G queries against all G*T keys, block-diagonal -inf mask."""
    G, T = k_pref.shape[0], k_pref.shape[1]
    out = np.empty_like(q_rows)
    for h in range(q_rows.shape[1]):
        Kall = k_pref[:, :, h, :].reshape(G * T, -1)
        Vall = v_pref[:, :, h, :].reshape(G * T, -1)
        S = scale * q_rows[:, h, :] @ Kall.T
        S = np.where(mask == 1, S, -np.inf)
        E = np.exp(S - S.max(axis=1, keepdims=True))
        out[:, h, :] = (E / E.sum(axis=1, keepdims=True)) @ Vall
    return out


def test_s5_paper_worked_mask():
    """The printed G=4, T=3 mask is block-diagonal, and the masked coalesced tile
    equals four independent 1x3 attentions."""
    mask = _mask_from_golden()
    assert mask.shape == (4, 12)
    assert np.array_equal(mask, np.kron(np.eye(4, dtype=np.int64), np.ones((1, 3), dtype=np.int64)))
    rng = np.random.default_rng(9)
    H, d = 2, 8
    q, kp, vp = _rand(rng, 4, H, d), _rand(rng, 4, 3, H, d), _rand(rng, 4, 3, H, d)
    ref = oracle.self_attn_rows(q, kp, vp, 0.6)
    assert np.max(np.abs(_coalesced_tile(q, kp, vp, 0.6, mask) - ref)) <= TOL


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_s5_coalesced_tiles_any_group(G):
    rng = np.random.default_rng(G)
    B, M, H, d, T = 2, 4, 2, 8, 3
    qs, ks, vs, parents = _decode_inputs(rng, B, M, H, d, T)
    paged, tables, kp, vp = _paged_decode(qs, ks, vs, parents, B, M, 0.45)
    t = T - 1
    R = B * M
    kflat, vflat = kp.reshape(-1, H, d), vp.reshape(-1, H, d)
    mask = np.kron(np.eye(G, dtype=np.int64), np.ones((1, t + 1), dtype=np.int64))
    for g0 in range(0, R, G):
        ids = tables[t][g0:g0 + G]
        got = _coalesced_tile(qs[t][g0:g0 + G], kflat[ids], vflat[ids], 0.45, mask)
        assert np.max(np.abs(got - paged[t][g0:g0 + G])) <= TOL


def test_s6_block_relabelling_invariance():
    rng = np.random.default_rng(10)
    B, M, H, d, T = 2, 3, 2, 4, 3
    qs, ks, vs, parents = _decode_inputs(rng, B, M, H, d, T)
    outs, tables, kp, vp = _paged_decode(qs, ks, vs, parents, B, M, 0.5)
    t = T - 1
    nblk = kp.shape[0] * kp.shape[1]
    pi = rng.permutation(nblk)              # physical block i moves to pi[i]
    kflat = np.empty((nblk, H, d))
    vflat = np.empty((nblk, H, d))
    kflat[pi] = kp.reshape(nblk, H, d)
    vflat[pi] = vp.reshape(nblk, H, d)
    table = pi[tables[t]]
    got = oracle.self_attn_step(qs[t], kflat.reshape(kp.shape), vflat.reshape(vp.shape),
                                table, t, 0.5)
    assert np.array_equal(got, outs[t])


def test_s7_printed_tflops_fix_prefix_length():
    """The paper's TFLOP/s row at t=3 is 4*R*H*d*(keys attended)/latency only when
    the prefix holds t+1 tokens; the oracle attends exactly that many."""
    lines = [ln.split() for ln in open(os.path.join(GOLDEN, "self_attn_microbench_t3.txt"))
             if ln.strip() and not ln.startswith("#")]
    R, H, d, t = (int(x) for x in lines[0])
    rng = np.random.default_rng(0)
    Bs, Ms = 1, 2
    qs, ks, vs, parents = _decode_inputs(rng, Bs, Ms, 1, 4, t + 1)
    _, _, kp, vp = _paged_decode(qs, ks, vs, parents, Bs, Ms, 1.0)
    table = oracle.table_rows(np.arange(Bs * Ms), t, parents, Bs, Ms)
    _, probs = oracle.self_attn_step(qs[t], kp, vp, table, t, 1.0, return_probs=True)
    n_keys = probs.shape[-1]
    assert n_keys == t + 1
    for name, ms, tflops in lines[1:]:
        ms, tflops = float(ms), float(tflops)
        model = 4.0 * R * H * d * n_keys / (ms * 1e-3) / 1e12
        assert abs(model - tflops) / tflops < 0.011, name
        wrong = 4.0 * R * H * d * t / (ms * 1e-3) / 1e12
        assert abs(wrong - tflops) / tflops > 0.2, name


def test_self_attn_probs_are_distributions():
    rng = np.random.default_rng(12)
    q, kp, vp = _rand(rng, 5, 3, 8), _rand(rng, 5, 4, 3, 8), _rand(rng, 5, 4, 3, 8)
    _, p = oracle.self_attn_rows(q, kp, vp, 0.3, return_probs=True)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(axis=-1) - 1)) <= TOL


def test_oracle_on_generated_tiny_workload():
    """End to end on the tiny fp32 workload: paged path equals the dense brute force
    on the generated (seeded) inputs, and cross-attention equals the unshared form."""
    wl = W.WORKLOADS["tiny_fp32"]
    inp = W.DecodeInputs(wl, seed=0, device="cpu")
    ek, ev = inp.enc_kv
    scale = 1 / math.sqrt(wl.d)
    q = inp.step_tensor("q_cross", 0).double().numpy()
    got = oracle.cross_attn(q, ek, ev, inp.offsets, wl.M, scale)
    ref = _bf_cross_unshared(q, ek.double().numpy(), ev.double().numpy(), inp.offsets, wl.M, scale)
    assert np.max(np.abs(got - ref)) <= TOL
    T = wl.steps
    qs = [inp.step_tensor("q_self", t).double().numpy() for t in range(T)]
    ks = [inp.step_tensor("k_new", t).double().numpy() for t in range(T)]
    vs = [inp.step_tensor("v_new", t).double().numpy() for t in range(T)]
    parents = [inp.parents(t) for t in range(T)]
    paged, _, _, _ = _paged_decode(qs, ks, vs, parents, wl.B, wl.M, scale)
    dense = _bf_full_history(qs, ks, vs, parents, wl.B, wl.M, scale)
    for t in range(T):
        assert np.max(np.abs(paged[t] - dense[t])) <= TOL
