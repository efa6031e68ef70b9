"""Parity of the beam-step entry points and of the dynamic-width fused step with
the oracle, through the C ABI on the GPU.

Score update: max abs error <= 1e-4 (fp32 arithmetic on scores of magnitude
<= ~60), the filter pattern (-inf entries) bit-exact.  Top-k: bit-exact
(parents, tokens and scores) on seeded fp32 candidate arrays of every
structure the selection has a separate path for.  Dynamic-width fused step:
tables and pools bit-exact, attention within 2e-2 (bf16) / 1e-5 (fp32).
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import beam_oracle as BO
from paper_2608_00938_amd import grace as G
from paper_2608_00938_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _mask_tensor(mask, dev):
    return None if mask is None else torch.from_numpy(np.ascontiguousarray(mask).view(np.int32)).to(dev)


@pytest.mark.parametrize("R,V", [(37, 512), (5, 33), (1, 1), (64, 1000)])
@pytest.mark.parametrize("masked", [False, True], ids=["all", "filtered"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_beam_scores_parity(gpu, dtype, masked, R, V):
    _log(f"[beam scores] {dtype} masked={masked} R={R} V={V}")
    logits = W.beam_logits(3, 2, R, V, dtype, gpu)
    prev = W.beam_prev_scores(3, 2, R)
    mask = W.beam_mask(3, 2, R, V) if masked else None
    cand, rmax = G.grace_beam_scores(logits, torch.from_numpy(prev).to(gpu), _mask_tensor(mask, gpu))
    torch.cuda.synchronize()
    allowed = None if mask is None else BO.unpack_mask(mask, V)
    ref = BO.candidate_scores(logits.float().cpu().numpy(), prev, allowed)
    got = cand.cpu().numpy().astype(np.float64)
    assert np.array_equal(np.isneginf(got), np.isneginf(ref))
    fin = np.isfinite(ref)
    err = float(np.max(np.abs(got[fin] - ref[fin]))) if fin.any() else 0.0
    _log(f"  max|err| = {err:.3e}")
    assert err <= 1e-4
    ref_max = ref.max(axis=1)
    gmax = rmax.cpu().numpy().astype(np.float64)
    assert np.array_equal(np.isneginf(gmax), np.isneginf(ref_max))
    f = np.isfinite(ref_max)
    assert np.all(np.abs(gmax[f] - ref_max[f]) <= 1e-4)


def _topk_case(gpu, cand, B, M, V, k, row_max=None):
    par, tok, sc = G.grace_beam_topk(torch.from_numpy(cand).to(gpu), B, M, k,
                                     row_max=None if row_max is None else
                                     torch.from_numpy(row_max).to(gpu))
    torch.cuda.synchronize()
    rp, rt, rs = BO.beam_topk(cand, B, M, V, k)
    assert np.array_equal(par.cpu().numpy(), rp), "parents"
    assert np.array_equal(tok.cpu().numpy(), rt), "tokens"
    assert np.array_equal(sc.cpu().numpy().view(np.uint32), rs.view(np.uint32)), "scores (bitwise)"


TOPK_SHAPES = [(3, 37, 64, 50), (2, 16, 600, 4096), (4, 200, 100, 1), (1, 3, 5, 15), (2, 64, 512, 777),
               (2, 131, 257, 2000)]   # the last: M*V not a multiple of 4, over two slices


@pytest.mark.parametrize("shape", TOPK_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("kind", ["normal", "ties", "equal", "sparse", "wide", "special"])
def test_beam_topk_bit_exact(gpu, kind, shape):
    B, M, V, k = shape
    k = min(k, M * V)
    _log(f"[beam topk] kind={kind} B={B} M={M} V={V} k={k}")
    cand = W.candidate_array(5, B, M, V, kind)
    _topk_case(gpu, cand, B, M, V, k)


@pytest.mark.parametrize("hint", ["true", "low", "high"])
def test_beam_topk_row_max_hint_does_not_change_result(gpu, hint):
    B, M, V, k = 3, 128, 512, 1000
    cand = W.candidate_array(6, B, M, V, "normal")
    true_max = cand.max(axis=1)
    row_max = {"true": true_max, "low": true_max - 500.0, "high": true_max + 70.0}[hint]
    _log(f"[beam topk hint] {hint}")
    _topk_case(gpu, cand, B, M, V, k, row_max=row_max.astype(np.float32))


def test_beam_topk_sampled_bin_too_low_falls_back(gpu):
    """The k best are not spread like the rest: in each request only the first
    32 candidates (a chunk that the kernel's sixteenth-sample always holds) score
    high, so the sampled bin has too few candidates above it (32 < k) and the
    full histogram path must take over.  The result must not change."""
    B, M, V, k = 2, 64, 512, 64
    rng = np.random.default_rng(11)
    cand = (-20.0 - rng.random((B * M, V))).astype(np.float32)
    for b in range(B):
        cand[b * M, :32] = (-rng.random(32)).astype(np.float32)
    _log(f"[beam topk sample miss] B={B} M={M} V={V} k={k}")
    _topk_case(gpu, cand, B, M, V, k)


def test_beam_topk_large_fast_path(gpu):
    """The paper's widths: 1024 beams x 512 tokens per request, k = 1024."""
    B, M, V, k = 8, 1024, 512, 1024
    _log(f"[beam topk large] B={B} M={M} V={V} k={k}")
    cand = W.candidate_array(7, B, M, V, "normal")
    _topk_case(gpu, cand, B, M, V, k)


def test_beam_scores_then_topk_is_a_valid_topk(gpu):
    """GPU scores feed GPU top-k; the selection must be a top-k of the fp64
    scores up to the scores' error: every selected candidate is within eps of
    the oracle's k-th score or above, every candidate clearly above it is taken."""
    B, M, V, k, eps = 4, 96, 512, 512, 1e-4
    R = B * M
    logits = W.beam_logits(8, 2, R, V, "bf16", gpu)
    prev = W.beam_prev_scores(8, 2, R)
    mask = W.beam_mask(8, 2, R, V, keep=0.5)
    cand, rmax = G.grace_beam_scores(logits, torch.from_numpy(prev).to(gpu), _mask_tensor(mask, gpu))
    par, tok, _ = G.grace_beam_topk(cand, B, M, k, row_max=rmax)
    torch.cuda.synchronize()
    ref = BO.candidate_scores(logits.float().cpu().numpy(), prev, BO.unpack_mask(mask, V))
    par, tok = par.cpu().numpy(), tok.cpu().numpy()
    for b in range(B):
        s = ref[b * M:(b + 1) * M].reshape(-1)
        kth = np.sort(s)[::-1][k - 1]
        sel = par[b].astype(np.int64) * V + tok[b]
        assert len(set(sel.tolist())) == k
        assert np.all(s[sel] >= kth - eps)
        clearly = np.nonzero(s > kth + eps)[0]
        assert set(clearly.tolist()) <= set(sel.tolist())


STEP_CASES = [
    dict(dtype="bf16", B=3, M=128, V=512, k=300, mask=True),    # 8-token-run score kernel
    dict(dtype="f32", B=2, M=40, V=100, k=50, mask=True),       # generic score kernel (V % 8 != 0)
    dict(dtype="bf16", B=2, M=16, V=600, k=4096, mask=False),   # two runs per lane, k = max
    dict(dtype="bf16", B=2, M=3, V=5, k=15, mask=False),        # k = M*V
    dict(dtype="bf16", B=8, M=1024, V=512, k=1024, mask=True),  # the paper's widths: sampled path
    dict(dtype="bf16", B=2, M=32, V=512, k=100, mask=False, equal=True),   # all equal: radix path
]


@pytest.mark.parametrize("i", range(len(STEP_CASES)))
def test_beam_step_equals_scores_then_topk(gpu, i):
    """grace_beam_step recomputes each candidate from the logits instead of
    reading a written array; its outputs must equal grace_beam_scores followed
    by grace_beam_topk bit for bit."""
    c = STEP_CASES[i]
    B, M, V, k = c["B"], c["M"], c["V"], c["k"]
    R = B * M
    _log(f"[beam step] {c}")
    if c.get("equal"):
        logits = torch.full((R, V), 0.5, device=gpu).to(W.TORCH_DTYPES[c["dtype"]])
        prev = torch.full((R,), -3.0, device=gpu)
    else:
        logits = W.beam_logits(9 + i, 2, R, V, c["dtype"], gpu)
        prev = torch.from_numpy(W.beam_prev_scores(9 + i, 2, R)).to(gpu)
    mask = _mask_tensor(W.beam_mask(9 + i, 2, R, V, keep=0.6), gpu) if c["mask"] else None
    cand, rmax = G.grace_beam_scores(logits, prev, mask)
    p1, t1, s1 = G.grace_beam_topk(cand, B, M, k, row_max=rmax)
    p2, t2, s2 = G.grace_beam_step(logits, prev, B, M, k, mask=mask)
    torch.cuda.synchronize()
    assert torch.equal(p1, p2), "parents"
    assert torch.equal(t1, t2), "tokens"
    assert torch.equal(s1.view(torch.int32), s2.view(torch.int32)), "scores (bitwise)"


DYN = [
    dict(dtype="bf16", B=3, H=2, d=64, widths=(1, 5, 12, 12)),
    dict(dtype="f32", B=2, H=3, d=32, widths=(1, 4, 9, 7, 9)),
    dict(dtype="bf16", B=2, H=8, d=128, widths=(1, 8, 16, 16)),   # 2 KiB rows: wave-uniform path
]


@pytest.mark.parametrize("cfg", DYN, ids=["bf16_d64", "f32_d32", "bf16_d128"])
def test_fused_dyn_parity(gpu, cfg):
    B, H, d, widths = cfg["B"], cfg["H"], cfg["d"], cfg["widths"]
    T = len(widths)
    Mmax = max(widths)
    R_s = B * Mmax
    wl = W.custom(dtype=cfg["dtype"], B=B, M=Mmax, H=H, d=d, steps=T, L=4)
    tol = 2e-2 if cfg["dtype"] == "bf16" else 1e-5
    scale = 1.0 / math.sqrt(d)
    _log(f"[fused dyn] {cfg}")
    cache = G.KVCache(B, Mmax, H, d, T, wl.torch_dtype, gpu)
    kp = np.zeros((T, R_s, H, d))
    vp = np.zeros_like(kp)
    table = None
    news = []
    for t, Mc in enumerate(widths):
        R = B * Mc
        Mp = widths[t - 1] if t > 0 else 1
        gen = lambda tag: W.normal((R, H, d), 21, tag, t, wl, gpu)  # noqa: E731
        q, kn, vn = gen("q_self"), gen("k_new"), gen("v_new")
        par_np = W.dyn_parents(21, t, B, Mp, Mc) if t > 0 else None
        par = None if par_np is None else torch.from_numpy(par_np).to(gpu)
        out = cache.append_attend_dyn(t, q, kn, vn, par, Mp, Mc, scale)
        torch.cuda.synchronize()
        tnew = BO.kv_append_table_dyn(table, par_np, B, Mp, Mc, t, R_s)
        kp[t, :R] = kn.float().cpu().numpy()
        vp[t, :R] = vn.float().cpu().numpy()
        full = np.zeros((R, T), dtype=np.int64)
        full[:, :t + 1] = tnew
        ref = oracle.self_attn_step(q.float().cpu().numpy(), kp, vp, full, t, scale)
        got_table = cache.table(t)[:R, :t + 1].cpu().numpy()
        assert np.array_equal(got_table, tnew), f"table t={t}"
        err = float(np.max(np.abs(out.float().cpu().numpy() - ref)))
        _log(f"  t={t} widths {Mp}->{Mc}: max|err| = {err:.3e}")
        assert err <= tol
        assert torch.equal(cache.k_pool[t, :R], kn) and torch.equal(cache.v_pool[t, :R], vn)
        table = full
        news.append((kn, vn))
    assert int(cache.err_flag.item()) == 0


def test_fused_dyn_out_of_range_parent(gpu):
    B, H, d = 2, 2, 64
    wl = W.custom(dtype="bf16", B=B, M=6, H=H, d=d, steps=2, L=4)
    cache = G.KVCache(B, 6, H, d, 2, wl.torch_dtype, gpu)
    gen = lambda R, tag, t: W.normal((R, H, d), 22, tag, t, wl, gpu)  # noqa: E731
    cache.append_attend_dyn(0, gen(2 * B, "q_self", 0), gen(2 * B, "k_new", 0),
                            gen(2 * B, "v_new", 0), None, 1, 2)
    par = torch.tensor([0, 1, 2, 1, 5, 0], dtype=torch.int32, device=gpu)   # M_prev = 2
    cache.append_attend_dyn(1, gen(3 * B, "q_self", 1), gen(3 * B, "k_new", 1),
                            gen(3 * B, "v_new", 1), par, 2, 3)
    torch.cuda.synchronize()
    assert int(cache.err_flag.item()) == 1
    tab = cache.table(1)[:3 * B, 0].cpu().numpy()
    # row 2 (parent 2 -> clamped to 1) and row 4 (parent 5 -> 1) of request 1
    assert tab.tolist() == [0, 1, 1, 3, 3, 2]
